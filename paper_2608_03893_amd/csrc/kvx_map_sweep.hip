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
constexpr int NT = 256;   // threads per workgroup

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

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

// The map fragments live in accumulation registers (AGPRs) and feed the
// matrix instruction's A operand from there, which the compiler's own
// lowering does not do (it would copy them into VGPRs before every use).
// acc = A * B + acc, and acc = A * B.
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc) : "a"(w), "v"(x));
}
__device__ __forceinline__ void mfma_first(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(acc) : "a"(w), "v"(x));
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
  constexpr int XBUF = U * MT * D;
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
  // the last row) so the memory counter retires them in order.
  uint4 ra[NS][UH], rb[NS][UH];
  uint32_t csx[NS][8];
  auto stage_load = [&](int set, int64_t tt) __attribute__((always_inline)) {
    const int64_t t = tt + sr < t_end ? tt + sr : t_end - 1;
    const uint32_t off = (uint32_t)(t * (D * 2)) + 16u * sq;
#pragma unroll
    for (int j = 0; j < UH; ++j) {
      ra[set][j] = *reinterpret_cast<const uint4*>(Xrow[j] + off);
      rb[set][j] = *reinterpret_cast<const uint4*>(Xrow[j] + off + HALF * 2);
    }
    if (KV == 0) {
      const uint32_t* pc = cs_s + t * HALF;
      const uint4 c0 = *reinterpret_cast<const uint4*>(pc + (STYLE == 0 ? 8 * sq : 4 * sq));
      const uint4 c1 = *reinterpret_cast<const uint4*>(pc + (STYLE == 0 ? 8 * sq + 4 : 32 + 4 * sq));
      unpack4(c0, csx[set]);
      unpack4(c1, csx[set] + 4);
    }
  };
  // Strip (keys) and write slot j of a register set into an LDS buffer.
  // Chunk q of token r of slot u sits at position q ^ r ^ (8 if u >= UH): the
  // two slot halves of a 16-lane group then write complementary bank halves.
  auto stage_store = [&](int set, int buf, int j) __attribute__((always_inline)) {
    uint16_t* xb = X + buf * XBUF + (UH * sh + j) * (MT * D) + sr * D;
    const int sw = (sr & 15) ^ (8 * sh);
    if (KV == 0) {
      if (STYLE == 0) {
        strip_halfsplit(ra[set][j], rb[set][j], csx[set]);
      } else {
        strip_interleaved(ra[set][j], csx[set]);
        strip_interleaved(rb[set][j], csx[set] + 4);
      }
    }
    *reinterpret_cast<uint4*>(xb + 8 * (sq ^ sw)) = ra[set][j];
    *reinterpret_cast<uint4*>(xb + 8 * ((8 + sq) ^ sw)) = rb[set][j];
  };

#pragma unroll
  for (int s = 0; s < NS; ++s) stage_load(s, t_begin + (int64_t)s * MT);
#pragma unroll
  for (int j = 0; j < UH; ++j) stage_store(0, 0, j);
  __syncthreads();

  // Tile it (LDS buffer it % 2, register set it % NS):  multiply it while the
  // rows of tile it+1 (set (it+1) % NS) are stripped into the other buffer;
  // then set it % NS takes the loads of tile it+NS.
  auto tile = [&](int it, int cur) __attribute__((always_inline)) {
    const int par = it & 1;
    const int nxt = cur + 1 < NS ? cur + 1 : 0;
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
      const uint4 c0 = *reinterpret_cast<const uint4*>(pc + (STYLE == 0 ? 32 * o + 8 * c : 16 * o + 4 * c));
      const uint4 c1 = *reinterpret_cast<const uint4*>(pc + (STYLE == 0 ? 32 * o + 8 * c + 4 : 32 + 16 * o + 4 * c));
      unpack4(c0, ct);
      unpack4(c1, ct + 4);
    }

    // ---- contraction, B-fragment reads two steps ahead
    const uint16_t* xcur = X + par * XBUF;
    auto xfrag = [&](int z) __attribute__((always_inline)) -> u32x4_t {
      const int u = um[z / 4];
      const uint16_t* xs = xcur + u * (MT * D);
      return lds_read_b128(xs + row * D + 8 * ((4 * (z % 4) + c) ^ row ^ (u >= UH ? 8 : 0)));
    };
    // B-fragment reads run PF steps ahead of the MFMAs (ring of PF + 1)
    constexpr int PF = 3;
    f32x4_t acc[4];
    u32x4_t xf[PF + 1];
#pragma unroll
    for (int z = 0; z < PF && z < Z; ++z) xf[z] = xfrag(z);
#pragma unroll
    for (int z = 0; z < Z; ++z) {
      // reads issued after step z's: min(PF - 1, Z - 1 - z)
      if (Z - 1 - z >= PF - 1)
        lds_wait<PF - 1>(xf[z % (PF + 1)]);
      else if (Z - 1 - z == 1)
        lds_wait<1>(xf[z % (PF + 1)]);
      else
        lds_wait<0>(xf[z % (PF + 1)]);
      if (z + PF < Z) xf[(z + PF) % (PF + 1)] = xfrag(z + PF);
#pragma unroll
      for (int lb = 0; lb < 4; ++lb) {
        if (z == 0)
          mfma_first(acc[lb], wf[lb][z], xf[z % (PF + 1)]);
        else
          mfma_acc(acc[lb], wf[lb][z], xf[z % (PF + 1)]);
      }
      // the next tile's rows: one staging slot every Z / UH steps
      if (z % (Z / UH) == 0) stage_store(nxt, par ^ 1, z / (Z / UH));
    }
    mfma_drain(acc);
    stage_load(cur, tt + (int64_t)NS * MT);

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
          uint4 v;
          v.x = pack2(y[x][0], y[x][1]);
          v.y = pack2(y[x][2], y[x][3]);
          v.z = pack2(y[x][4], y[x][5]);
          v.w = pack2(y[x][6], y[x][7]);
          *reinterpret_cast<uint4*>(dst + 64 * x) = v;
        }
      }
    }
    __syncthreads();
  };

  // two tiles per trip, so that register sets and LDS buffers are indexed
  // with constants
  static_assert(NS == 2, "the tile loop is written for two register sets");
  for (int it = 0; it < n_tiles; it += 2) {
    tile(it, 0);
    if (it + 1 < n_tiles) tile(it + 1, 1);
  }
}

template <int K, int STYLE, bool SLOTS>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void map_sweep_kernel(const MapArgs a, const SweepPlan p) {
  constexpr int XBUF = 2 * K * MT * D;
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

  const int slot = blockIdx.x >> 3;
  const int pair = slot % p.pairs;
  const int part = slot / p.pairs;
  if (part >= p.parts) return;
  q.T = a.T;
  q.t_begin = (int64_t)part * p.part_len;
  if (q.t_begin >= q.T) return;
  q.t_end = q.t_begin + p.part_len < q.T ? q.t_begin + p.part_len : q.T;
  q.n_tiles = (int)((q.t_end - q.t_begin + MT - 1) / MT);

  // Unit u -> (K|V, head, group).  Keys cost more vector work than values
  // (two rotations), so when the units of one kind divide evenly over the
  // eight XCDs every XCD alternates between them.
  const int per_kind = p.n_units / 2;
  for (int unit = blockIdx.x & 7; unit < p.n_units; unit += 8) {
    int kv, rest;
    if (per_kind % 8 == 0) {
      kv = (unit >> 3) & 1;
      rest = (unit & 7) | ((unit >> 4) << 3);
    } else {
      kv = unit & 1;
      rest = unit >> 1;
    }
    const int h = rest % a.H;
    const int g = rest / a.H;
    const int g0 = g * p.group_len;
    const int g_n = a.nl - g0 < p.group_len ? a.nl - g0 : p.group_len;
    if (2 * pair >= g_n) continue;          // same decision in every thread
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

SweepPlan plan_sweep(int nl, int H, int64_t T) {
  SweepPlan p{};
  const int groups = (nl + 63) / 64;
  p.groups = groups;
  p.group_len = (nl + groups - 1) / groups;
  p.pairs = (p.group_len + 1) / 2;
  p.parts = 32 / p.pairs;
  const int64_t per = (T + p.parts - 1) / p.parts;
  p.part_len = (int32_t)((per + MT - 1) / MT * MT);
  p.n_units = groups * H * 2;
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
