// Layer-sweep map kernel for bf16 caches with head dimension 128 and k <= 4.
//
// Each source row (layer, head, K|V, token) is an input of about L_t*k/L_s
// target layers.  This kernel makes one XCD run every target layer of a
// (head, K|V) over the same token tiles at the same time, so a source row is
// fetched from HBM once and then served to all its users from that XCD's L2.
//
// Grid: one workgroup per CU (256), 4 waves, one wave per SIMD with the whole
// register file.  Workgroup b runs on XCD b % 8 and takes slot j = b / 8 of
// it.  A unit of work is (layer group, head, K|V); XCD x takes units x, x+8,
// ...  Within a unit, slot j owns a pair of target layers and a token part.
// Per unit, each wave keeps its slice of one target layer's map in registers:
//   wave w: layer slot w / 2 of the pair, output half w % 2, i.e. the output
//   channels 32*(w%2) .. +31 and 64 + 32*(w%2) .. +31 (whole RoPE planes of
//   either layout), held as 4 blocks x 4k steps of v_mfma_f32_16x16x32_bf16
//   A-fragments (W^T rows, 256 VGPRs at k = 4).
//
// The token part is swept in 32-token tiles.  The workgroup stages the tile's
// rows of the (at most 2k) distinct source layers its two target layers
// select into LDS, stripping the source RoPE from keys on the way (Sec. 3.3)
// and rounding once to bf16.  Then every wave contracts the tile with its
// register-resident map (Eq. ridge_kv, C^T = W^T X^T, fp32 accumulation),
// adds the bias, applies the target RoPE in registers and stores.  Source rows
// are loaded two tiles ahead into one of two register sets; while tile i is
// multiplied, the rows of tile i+1 are stripped and written to the other LDS
// buffer between the matrix instructions, so the vector ALU work runs in the
// shadow of the matrix core.  One barrier per tile hands the buffers over.
//
// LDS tile layout: [source slot u][token r][16 chunks of 8 channels], chunk q
// of row r stored at position q ^ (r & 15), so the 16 tokens of an MFMA
// B-fragment read fall on distinct banks.  The map image is the one the
// W-stationary kernel uses (packed once per call): row rho = 16b + 4c + r of
// a task holds output channel 32*(b/2) + 8c + 4*(b%2) + r, and reduction
// chunk 4z + c of step z holds input features 32z + 8c .. 32z + 8c + 7.
#include "kvx_bf16.h"
#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int D = 128;
constexpr int HALF = 64;
constexpr int MT = 16;    // tokens per tile (one MFMA token block)
// LDS tile layout (bf16 elements): token rows padded to 272 bytes, so that the
// 16 tokens of a B-fragment read, for any chunk, fall on 16 distinct groups
// of four banks, and a fragment's address moves by a constant from one
// reduction step to the next; source slots padded by 32 bytes, so that the
// two slot halves written by one 16-lane group use complementary banks.
constexpr int RS = D + 8;            // row stride
constexpr int SS = MT * RS + 16;     // slot stride
constexpr int NT = 256;   // threads per workgroup

// LDS fragment reads are issued from inline assembly so that the compiler,
// short of registers, cannot sink them next to their use: the MFMA loop keeps
// two steps of reads in flight.  Such a read is unknown to the compiler's
// wait-count bookkeeping, so each result is tied to an explicit wait on the
// LDS counter (lds_wait) before it is used; LDS operations complete in order.
__device__ __forceinline__ u32x4_t lds_read_b128(const uint16_t* p) {
  u32x4_t v;
  const uint32_t addr = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

// Wait until at most N LDS operations are outstanding; a and b are live
// through the wait so no use of them can be scheduled above it.
template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t& a) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(a) : "n"(N));
}

// The same wait with a count known only after unrolling.
__device__ __forceinline__ void lds_wait_n(int n, u32x4_t& a) {
  switch (n) {
    case 0: lds_wait<0>(a); break;
    case 1: lds_wait<1>(a); break;
    case 2: lds_wait<2>(a); break;
    case 3: lds_wait<3>(a); break;
    case 4: lds_wait<4>(a); break;
    case 5: lds_wait<5>(a); break;
    case 6: lds_wait<6>(a); break;
    case 7: lds_wait<7>(a); break;
    default: lds_wait<8>(a); break;
  }
}

// LDS write from inline assembly, so that it keeps its place among the
// fragment reads (the wait counts above count it).
__device__ __forceinline__ void lds_write_b128(uint16_t* p, const u32x4_t& v) {
  const uint32_t addr = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)p;
  asm volatile("ds_write_b128 %0, %1" : : "v"(addr), "v"(v) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const uint16_t* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Read / write at a constant byte offset from an LDS address.
template <int OFF>
__device__ __forceinline__ u32x4_t lds_read_off(uint32_t addr) {
  u32x4_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
  return v;
}
template <int OFF>
__device__ __forceinline__ void lds_write_off(uint32_t addr, const u32x4_t& v) {
  asm volatile("ds_write_b128 %0, %1 offset:%2" : : "v"(addr), "v"(v), "n"(OFF) : "memory");
}
__device__ __forceinline__ u32x4_t lds_read_step(uint32_t addr, int s) {
  switch (s) {
    case 0: return lds_read_off<0>(addr);
    case 1: return lds_read_off<64>(addr);
    case 2: return lds_read_off<128>(addr);
    default: return lds_read_off<192>(addr);
  }
}

// All LDS operations issued so far have completed.
__device__ __forceinline__ void lds_drain() { asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory"); }

// The map fragments live in accumulation registers (AGPRs) and feed the
// matrix instruction's A operand from there, which the compiler's own
// lowering does not do (it would copy them into VGPRs before every use).
// acc = A * B + acc, and acc = A * B.
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc) : "a"(w), "v"(x));
}
__device__ __forceinline__ void mfma_first(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(acc) : "a"(w), "v"(x));
}

// Results of matrix instructions issued from inline assembly are invisible
// to the compiler's hazard tracking: 24 wait states before any vector
// instruction reads them (more than a 16x16x32 instruction needs).
__device__ __forceinline__ void mfma_drain(f32x4_t (&acc)[4]) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
               : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]));
}

// Everything the units of one workgroup share.
struct SweepCtx {
  int tid, lane, wave, c, row, sl, o, sr, sq, sh;
  int64_t T, t_begin, t_end;
  int n_tiles;
};

// One unit (layer group, head, K|V) of one workgroup: stage the maps, then
// sweep the token part.  KV is 0 for keys (strip and re-apply RoPE), 1 for
// values.  NS register sets hold source rows of the next NS tiles in flight.
template <int K, int STYLE, bool SLOTS, int KV, int NS>
__device__ __forceinline__ void sweep_unit(const MapArgs& a, const SweepCtx& q, uint16_t* X,
                                           float (*Bs)[D], int h, int ll0, bool has1) {
  constexpr int KD = K * D;
  constexpr int U = 2 * K;          // source slots
  constexpr int UH = K;             // slots per staging thread (half of them)
  constexpr int XBUF = U * SS;
  constexpr int Z = 4 * K;          // reduction steps
  const int c = q.c, row = q.row, sl = q.sl, o = q.o, sr = q.sr, sq = q.sq, sh = q.sh;
  const bool mine = sl == 0 || has1;   // this wave has a layer to write
  const int64_t T = q.T, t_begin = q.t_begin, t_end = q.t_end;
  const int n_tiles = q.n_tiles;

  // Distinct source layers of the pair, and each block's slot among them.
  int srcs[U];
  int umap[2][K];
  int nU = 0;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int i = 0; i < K; ++i) {
      umap[s][i] = 0;
      if (s == 1 && !has1) continue;
      const int v = a.idx[(ll0 + s) * K + i];
      int pos = -1;
#pragma unroll
      for (int w = 0; w < U; ++w)
        if (pos < 0 && w < nU && srcs[w] == v) pos = w;
      if (pos < 0) {
#pragma unroll
        for (int w = 0; w < U; ++w)
          if (w == nU) srcs[w] = v;
        pos = nU++;
      }
      umap[s][i] = pos;
    }
  }
#pragma unroll
  for (int w = 0; w < U; ++w)
    if (w >= nU) srcs[w] = srcs[0];
  int um[K];
#pragma unroll
  for (int i = 0; i < K; ++i) um[i] = sl ? umap[1][i] : umap[0][i];

  // this thread's staging slots: UH * sh .. UH * sh + UH - 1
  const char* Xrow[UH];
#pragma unroll
  for (int j = 0; j < UH; ++j) {
    const int s0 = sh ? srcs[UH + j] : srcs[j];
    Xrow[j] = reinterpret_cast<const char*>(a.src) + (((int64_t)s0 * 2 + KV) * a.H + h) * T * (D * 2);
  }
  const uint32_t* cs_s = reinterpret_cast<const uint32_t*>(a.cs16);
  const uint32_t* cs_t = reinterpret_cast<const uint32_t*>(a.cs16_tgt);

  // ---- this wave's map slice: 4 output blocks x Z reduction steps.  A wave
  // without a layer multiplies with the pair's first map and stores nothing.
  u32x4_t wf[4][Z];
  {
    const int l = a.l0 + ll0 + (mine ? sl : 0);
    const uint16_t* img = reinterpret_cast<const uint16_t*>(a.wpack) +
                          (((int64_t)l * a.H + h) * 2 + KV) * (int64_t)D * KD;
#pragma unroll
    for (int lb = 0; lb < 4; ++lb) {
      const int b = 4 * (lb >> 1) + 2 * o + (lb & 1);
      const uint16_t* r0 = img + (int64_t)(16 * b + row) * KD;
#pragma unroll
      for (int z = 0; z < Z; ++z)
        wf[lb][z] = *reinterpret_cast<const u32x4_t*>(r0 + 8 * ((4 * z + c) ^ row));
    }
  }
  __syncthreads();   // the previous unit's last tile and bias are no longer read
  {
    const int s = q.tid >> 7, n = q.tid & 127;
    const uint16_t* bias = reinterpret_cast<const uint16_t*>(KV ? a.bv : a.bk);
    const bool ok = bias != nullptr && (s == 0 || has1);
    Bs[s][n] = ok ? lo_bf16(bias[((int64_t)(a.l0 + ll0 + s) * a.H + h) * D + n]) : 0.0f;
  }

  // ---- staging: thread (token sr, channel group sq, slot half sh) loads
  // channels 8sq.. and 64+8sq.. of its token for UH slots.  Loads are
  // unconditional (unused slots repeat slot 0, tokens past the end repeat
  // the last row) so the memory counter retires them in order.  Register set
  // j % 2 holds tile j: each slot is reloaded with tile j + 2 as soon as it
  // has been written to LDS during tile j - 1, so its loads have two tiles
  // to arrive.
  u32x4_t ra[NS][UH], rb[NS][UH];
  uint32_t csx[NS][8];
  auto clamp_row = [&](int64_t tt) __attribute__((always_inline)) -> int64_t {
    return tt + sr < t_end ? tt + sr : t_end - 1;
  };
  auto stage_load_cs = [&](int set, int64_t tt) __attribute__((always_inline)) {
    if (KV == 0) {
      const uint32_t* pc = cs_s + clamp_row(tt) * HALF;
      const u32x4_t c0 = *reinterpret_cast<const u32x4_t*>(pc + (STYLE == 0 ? 8 * sq : 4 * sq));
      const u32x4_t c1 = *reinterpret_cast<const u32x4_t*>(pc + (STYLE == 0 ? 8 * sq + 4 : 32 + 4 * sq));
      unpack4(c0, csx[set]);
      unpack4(c1, csx[set] + 4);
    }
  };
  auto stage_load_slot = [&](int set, int j, int64_t tt) __attribute__((always_inline)) {
    const uint32_t off = (uint32_t)(clamp_row(tt) * (D * 2)) + 16u * sq;
    ra[set][j] = *reinterpret_cast<const u32x4_t*>(Xrow[j] + off);
    rb[set][j] = *reinterpret_cast<const u32x4_t*>(Xrow[j] + off + HALF * 2);
  };
  // coefficients first: the memory counter retires in order, so waiting for
  // them does not also wait for the rows that follow
  auto stage_load = [&](int set, int64_t tt) __attribute__((always_inline)) {
    stage_load_cs(set, tt);
#pragma unroll
    for (int j = 0; j < UH; ++j) stage_load_slot(set, j, tt);
  };
  // LDS address of this thread's row of staging slot j in buffer buf; chunk
  // sq at +0, chunk 8 + sq at +128 bytes.
  auto stage_addr = [&](int buf, int j) __attribute__((always_inline)) -> uint32_t {
    return lds_addr(X + buf * XBUF + (UH * sh + j) * SS + sr * RS + 8 * sq);
  };
  // Strip (keys) and write slot j of a register set into an LDS buffer.
  auto stage_store = [&](int set, int buf, int j) __attribute__((always_inline)) {
    if (KV == 0) {
      if (STYLE == 0) {
        strip_halfsplit(ra[set][j], rb[set][j], csx[set]);
      } else {
        strip_interleaved(ra[set][j], csx[set]);
        strip_interleaved(rb[set][j], csx[set] + 4);
      }
    }
    const uint32_t ad = stage_addr(buf, j);
    lds_write_off<0>(ad, ra[set][j]);
    lds_write_off<128>(ad, rb[set][j]);
  };
  // The same work cut in four, one part per MFMA step of a slot's window:
  // part w strips word w of both chunks (keys); part 3 also writes the slot.
  // Empty asm statements pin each part's inputs and results to its step, so
  // the compiler can neither hoist nor gather the vector work of a slot.
  auto stage_part = [&](int set, int buf, int j, int w, int64_t tt_reload) __attribute__((always_inline)) {
    if (KV == 0) {
      uint32_t a0 = ra[set][j][w], b0 = rb[set][j][w];
      asm volatile("" : "+v"(a0), "+v"(b0));   // inputs taken here, not earlier
      if (STYLE == 0) {
        float u0 = lo_bf16(a0), u1 = hi_bf16(a0);
        float v0 = lo_bf16(b0), v1 = hi_bf16(b0);
        strip(u0, v0, csx[set][2 * w]);
        strip(u1, v1, csx[set][2 * w + 1]);
        a0 = pack2(u0, u1);
        b0 = pack2(v0, v1);
      } else {
        float u = lo_bf16(a0), v = hi_bf16(a0);
        strip(u, v, csx[set][w]);
        a0 = pack2(u, v);
        u = lo_bf16(b0), v = hi_bf16(b0);
        strip(u, v, csx[set][4 + w]);
        b0 = pack2(u, v);
      }
      asm volatile("" : "+v"(a0), "+v"(b0));
      ra[set][j][w] = a0;
      rb[set][j][w] = b0;
    }
    if (w == 3) {
      const uint32_t ad = stage_addr(buf, j);
      lds_write_off<0>(ad, ra[set][j]);
      lds_write_off<128>(ad, rb[set][j]);
      // the slot's registers are free: rows of the set's next tile; after the
      // last slot, the set's coefficients too
      stage_load_slot(set, j, tt_reload);
      if (j == UH - 1) stage_load_cs(set, tt_reload);
    }
  };

  stage_load(0, t_begin);
  stage_load(1, t_begin + MT);
#pragma unroll
  for (int j = 0; j < UH; ++j) stage_store(0, 0, j);
  stage_load(0, t_begin + 2 * MT);
  lds_drain();
  __syncthreads();

  // Tile it (LDS buffer it % 2): register set (it + 1) % 2 holds the rows of
  // tile it+1, which are stripped into the other buffer between the matrix
  // instructions, each slot then taking the rows of tile it+3.
  auto tile = [&](int it, int r) __attribute__((always_inline)) {
    const int par = r & 1;
    const int st_set = (r + 1) & 1;
    const int64_t tt = t_begin + (int64_t)it * MT;
    // target RoPE coefficients and destination row of this lane's token; a
    // token past the end is clamped to the last row of the part, so its lane
    // computes exactly that row's output and stores the same bytes
    uint32_t ct[8];
    const int64_t tl = tt + row;
    const int64_t tc = tl < t_end ? tl : t_end - 1;
    const int64_t orow = SLOTS ? (int64_t)a.slots[tc] : tc;
    if (KV == 0) {
      const uint32_t* pc = cs_t + tc * HALF;
      const u32x4_t c0 = *reinterpret_cast<const u32x4_t*>(pc + (STYLE == 0 ? 32 * o + 8 * c : 16 * o + 4 * c));
      const u32x4_t c1 = *reinterpret_cast<const u32x4_t*>(pc + (STYLE == 0 ? 32 * o + 8 * c + 4 : 32 + 16 * o + 4 * c));
      unpack4(c0, ct);
      unpack4(c1, ct + 4);
    }

    // ---- contraction, B-fragment reads PF steps ahead of the MFMAs
    const uint16_t* xrow = X + par * XBUF + row * RS + 8 * c;
    auto xfrag = [&](int z) __attribute__((always_inline)) -> u32x4_t {
      return lds_read_step(lds_addr(xrow + um[z / 4] * SS), z % 4);
    };
    constexpr int PF = 3;
    f32x4_t acc[4];
    u32x4_t xf[PF + 1];
#pragma unroll
    for (int z = 0; z < PF && z < Z; ++z) xf[z] = xfrag(z);
    // Step z issues, in this order: its wait, the read for step z + PF, its
    // MFMAs and, at the last step of each slot's window, two staging writes.
    // LDS operations complete in order, so the wait before step z allows the
    // reads for the later steps already issued plus the staging writes
    // issued since the read for step z.
    constexpr int SE = Z / UH;   // steps per staging slot (4)
    static_assert(SE == 4, "one staging slot per four reduction steps");
#pragma unroll
    for (int z = 0; z < Z; ++z) {
      int pending = (Z - 1 - z < PF - 1) ? Z - 1 - z : PF - 1;
#pragma unroll
      for (int s2 = 0; s2 < Z; ++s2)
        if (s2 < z && s2 >= z - PF && s2 % SE == SE - 1) pending += 2;
      lds_wait_n(pending, xf[z % (PF + 1)]);
      if (z + PF < Z) xf[(z + PF) % (PF + 1)] = xfrag(z + PF);
#pragma unroll
      for (int lb = 0; lb < 4; ++lb) {
        if (z == 0)
          mfma_first(acc[lb], wf[lb][z], xf[z % (PF + 1)]);
        else
          mfma_acc(acc[lb], wf[lb][z], xf[z % (PF + 1)]);
      }
      // the next tile's rows: one staging slot every SE steps
      stage_part(st_set, par ^ 1, z / SE, z % SE, tt + 3 * MT);
    }
    mfma_drain(acc);

    // ---- epilogue: y[x][e] is output channel 64x + 32o + 8c + e
    if (mine) {
      float y[2][8];
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const float4 b0 = *reinterpret_cast<const float4*>(&Bs[sl][64 * x + 32 * o + 8 * c]);
        const float4 b1 = *reinterpret_cast<const float4*>(&Bs[sl][64 * x + 32 * o + 8 * c + 4]);
        y[x][0] = acc[2 * x][0] + b0.x;
        y[x][1] = acc[2 * x][1] + b0.y;
        y[x][2] = acc[2 * x][2] + b0.z;
        y[x][3] = acc[2 * x][3] + b0.w;
        y[x][4] = acc[2 * x + 1][0] + b1.x;
        y[x][5] = acc[2 * x + 1][1] + b1.y;
        y[x][6] = acc[2 * x + 1][2] + b1.z;
        y[x][7] = acc[2 * x + 1][3] + b1.w;
      }
      if (KV == 0) {
        if (STYLE == 0) {
#pragma unroll
          for (int e = 0; e < 8; ++e) rot_fwd16(y[0][e], y[1][e], ct[e]);
        } else {
#pragma unroll
          for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int e = 0; e < 8; e += 2) rot_fwd16(y[x][e], y[x][e + 1], ct[4 * x + e / 2]);
        }
      }
      const bool store = !SLOTS || (orow >= 0 && orow < a.tgt_rows);
      if (store) {
        uint16_t* dst = reinterpret_cast<uint16_t*>(a.tgt) +
                        ((((int64_t)(a.l0 + ll0 + sl) * 2 + KV) * a.H + h) * a.tgt_rows + orow) * D +
                        32 * o + 8 * c;
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          u32x4_t v;
          v[0] = pack2(y[x][0], y[x][1]);
          v[1] = pack2(y[x][2], y[x][3]);
          v[2] = pack2(y[x][4], y[x][5]);
          v[3] = pack2(y[x][6], y[x][7]);
          *reinterpret_cast<u32x4_t*>(dst + 64 * x) = v;
        }
      }
    }
    lds_drain();   // the staging writes (not tracked by the compiler) are done
    __syncthreads();
  };

  // Two tiles per trip, so that register sets and LDS buffers are indexed
  // with constants.  All of them run even past the end: a
  // conditional tile would merge the register sets and make the compiler copy
  // (and so wait for) every staging load right after issuing it.  A phantom
  // tile's tokens are all clamped to the last row, whose bytes it stores again.
  static_assert(NS == 2, "the tile loop is written for two register sets");
  for (int it = 0; it < n_tiles; it += 2) {
    tile(it, 0);
    tile(it + 1, 1);
  }
}

template <int K, int STYLE, bool SLOTS>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void map_sweep_kernel(const MapArgs a, const SweepPlan p) {
  constexpr int XBUF = 2 * K * SS;
  __shared__ __attribute__((aligned(16))) uint16_t X[2 * XBUF];
  __shared__ __attribute__((aligned(16))) float Bs[2][D];

  SweepCtx q;
  q.tid = threadIdx.x;
  q.lane = q.tid & 63;
  q.wave = q.tid >> 6;
  q.c = q.lane >> 4;       // reduction chunk of an MFMA fragment
  q.row = q.lane & 15;     // token (B, D) or map row (A) within a block
  q.sl = q.wave >> 1;      // layer slot of the pair
  q.o = q.wave & 1;        // output half
  q.sr = q.tid >> 4;       // staging: token of the tile
  q.sq = (q.tid >> 1) & 7; // staging: 8-channel group (and its partner +64)
  q.sh = q.tid & 1;        // staging: slot half

  const int slot = blockIdx.x >> 3;   // CU slot within the XCD (0 .. 31)
  q.T = a.T;

  // Unit u -> (group, K|V, head).  Within a group, keys cost more vector work
  // than values (two rotations), so when the units of one kind divide evenly
  // over the eight XCDs every XCD takes both kinds.
  for (int unit = blockIdx.x & 7; unit < p.n_units; unit += 8) {
    const int g = unit / (2 * a.H);
    const int rem = unit % (2 * a.H);
    int kv, h;
    if (a.H % 8 == 0) {
      kv = (rem >> 3) & 1;
      h = (rem & 7) | ((rem >> 4) << 3);
    } else {
      kv = rem & 1;
      h = rem >> 1;
    }
    int g0, g_n;
    if (g < p.full_groups) {
      g0 = 64 * g;
      g_n = 64;
    } else {
      g0 = 64 * p.full_groups;
      g_n = 0;
      for (int r = 0; r < p.n_rest; ++r) {
        if (r == g - p.full_groups) g_n = p.rest_len[r];
        else if (r < g - p.full_groups) g0 += p.rest_len[r];
      }
    }
    // this CU's layer pair and token part (pairs * parts = 32)
    const int pairs = (g_n + 1) / 2;
    const int parts = 32 / pairs;
    const int pair = slot % pairs;
    const int part = slot / pairs;
    const int64_t per = (q.T + parts - 1) / parts;
    const int64_t part_len = (per + MT - 1) / MT * MT;
    q.t_begin = (int64_t)part * part_len;
    if (part >= parts || q.t_begin >= q.T) continue;   // same decision in every thread
    q.t_end = q.t_begin + part_len < q.T ? q.t_begin + part_len : q.T;
    q.n_tiles = (int)((q.t_end - q.t_begin + MT - 1) / MT);
    const int ll0 = g0 + 2 * pair;          // first layer of the pair, relative to l0
    const bool has1 = 2 * pair + 1 < g_n;
    if (kv == 0)
      sweep_unit<K, STYLE, SLOTS, 0, 2>(a, q, X, Bs, h, ll0, has1);
    else
      sweep_unit<K, STYLE, SLOTS, 1, 2>(a, q, X, Bs, h, ll0, has1);
  }
}

template <int K, int STYLE>
hipError_t launch_sk(const MapArgs& a, const SweepPlan& p, hipStream_t stream) {
  if (a.slots != nullptr)
    hipLaunchKernelGGL((map_sweep_kernel<K, STYLE, true>), dim3(256), dim3(NT), 0, stream, a, p);
  else
    hipLaunchKernelGGL((map_sweep_kernel<K, STYLE, false>), dim3(256), dim3(NT), 0, stream, a, p);
  return hipGetLastError();
}

template <int K>
hipError_t launch_sstyle(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  return style == 0 ? launch_sk<K, 0>(a, p, stream) : launch_sk<K, 1>(a, p, stream);
}

}  // namespace

SweepPlan plan_sweep(int nl, int H, int64_t /*T*/) {
  SweepPlan p{};
  p.full_groups = nl / 64;
  int r = nl % 64;
  for (int bit = 32; bit >= 1; bit >>= 1)
    if (r & bit) p.rest_len[p.n_rest++] = bit;
  p.n_groups = p.full_groups + p.n_rest;
  p.n_units = p.n_groups * H * 2;
  return p;
}

hipError_t launch_map_sweep(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  if (a.T == 0 || a.nl == 0) return hipSuccess;
  switch (a.k) {
    case 1: return launch_sstyle<1>(a, p, style, stream);
    case 2: return launch_sstyle<2>(a, p, style, stream);
    case 3: return launch_sstyle<3>(a, p, style, stream);
    case 4: return launch_sstyle<4>(a, p, style, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kvx
