// Pipelined layer-sweep map kernel for bf16 caches with head dimension 128 and
// k <= 4.
//
// The work decomposition is the layer sweep's: one workgroup per CU, 4 waves
// (one per SIMD, all 512 registers), a unit of work is (layer group, head,
// K|V), workgroup b runs on XCD b % 8 and takes CU slot b / 8 of it, and in a
// unit CU slot j owns a pair of target layers and a token part, so that one
// XCD sweeps every target layer of a (head, K|V) over the same tokens at the
// same time and each source row comes from HBM once.  Each wave keeps its
// slice of one target layer's map in AGPRs (4 output blocks x 4k steps of
// v_mfma_f32_16x16x32_bf16 A-fragments).
//
// What differs is how a 16-token tile reaches the matrix cores (Eq. ridge_kv
// and Sec. 3.3 define the arithmetic):
//  * Source rows go from memory straight into LDS (buffer loads with the LDS
//    flag), three tiles ahead, into a ring of four stages.  No register holds
//    a row in flight, and the only wait on them is at the end of a tile.
//  * Keys are stripped of the source RoPE in place in LDS, one tile ahead of
//    their use, by all 256 threads; the vector work is issued between the
//    matrix instructions, at most four instructions after each.
//  * The bias enters as the accumulator's initial value.
//  * The target RoPE, the rounding to bf16 and the stores of tile i run at the
//    start of tile i+1, while its first operand reads are in flight, from a
//    second accumulator set.
//  * Every memory instruction is a buffer instruction whose range is one
//    (layer, K|V, head) plane, so rows past the end of the cache read as zero
//    and rows outside the target are dropped by the hardware.
//
// LDS stage layout: 2k source slots, slot 2i + s holding block i of layer s of
// the pair (a pair with one layer repeats its rows), each 16 token rows of
// 256 bytes, chunk q (8 channels) of token r stored at chunk position q ^ r;
// slots are 4224 bytes apart, so that odd slots sit 128 bytes off the bank
// pattern of even ones.  After the slots, the tile's (cos, sin) fp16 pairs of
// the source RoPE, [16 tokens][64 planes].
#include "kvx_bf16.h"
#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int D = 128;
constexpr int MT = 16;                   // tokens per tile
constexpr int NT = 256;                  // threads per workgroup
constexpr int ROWB = D * 2;              // bytes per token row
constexpr int SLOTB = MT * ROWB + 128;   // slot stride in LDS
constexpr int CSB = MT * 256;            // coefficient block of a stage
constexpr int NSTAGE = 4;
constexpr int PF = 3;                    // operand reads issued ahead of their step

template <int K>
struct Geo {
  static constexpr int NSLOT = 2 * K;
  static constexpr int CS_OFF = NSLOT * SLOTB;
  static constexpr int STAGE = CS_OFF + CSB;
  static constexpr int LDS = NSTAGE * STAGE;
  static constexpr int Z = 4 * K;        // reduction steps per tile
};
static_assert(Geo<4>::LDS <= 160 * 1024, "four stages fit the LDS of a CU");

typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Buffer resource over [base, base + bytes): raw addressing, range-checked
// (reads outside return zero, writes outside are dropped).
__device__ __forceinline__ i32x4_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  i32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// 16 bytes per lane from buffer r at voff + soff into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory");
}

// Register loads and stores through buffer r.  Issued from inline assembly so
// that every memory instruction keeps its place: the waits below count them.
__device__ __forceinline__ void vload16(u32x4_t& v, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("buffer_load_dwordx4 %0, %1, %2, %3 offen" : "=v"(v) : "v"(voff), "s"(r), "s"(soff) : "memory");
}
__device__ __forceinline__ void vload4(uint32_t& v, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("buffer_load_dword %0, %1, %2, %3 offen" : "=v"(v) : "v"(voff), "s"(r), "s"(soff) : "memory");
}
template <int OFF>
__device__ __forceinline__ void vstore16(const u32x4_t& v, uint32_t voff, const i32x4_t& r) {
  asm volatile("buffer_store_dwordx4 %0, %1, %2, 0 offen offset:%3"
               :
               : "v"(v), "v"(voff), "s"(r), "n"(OFF)
               : "memory");
}

// Wait until at most N vector memory operations are outstanding (they retire
// in order); x is live through the wait so no use is scheduled above it.
template <int N>
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory"); }
template <int N, typename T>
__device__ __forceinline__ void vm_wait(T& x) { asm volatile("s_waitcnt vmcnt(%1)" : "+v"(x) : "n"(N) : "memory"); }

template <int OFF>
__device__ __forceinline__ void lds_read(u32x4_t& v, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
}
template <int OFF>
__device__ __forceinline__ void lds_write(uint32_t addr, const u32x4_t& v) {
  asm volatile("ds_write_b128 %0, %1 offset:%2" : : "v"(addr), "v"(v), "n"(OFF) : "memory");
}
template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t& a) { asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(a) : "n"(N)); }
template <int N>
__device__ __forceinline__ void lds_wait2(u32x4_t& a, u32x4_t& b) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "n"(N));
}
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
    case 8: lds_wait<8>(a); break;
    case 9: lds_wait<9>(a); break;
    case 10: lds_wait<10>(a); break;
    case 11: lds_wait<11>(a); break;
    case 12: lds_wait<12>(a); break;
    case 13: lds_wait<13>(a); break;
    case 14: lds_wait<14>(a); break;
    default: lds_wait<15>(a); break;
  }
}
__device__ __forceinline__ void lds_drain() { asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory"); }

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// acc = A * B + acc, and acc = A * B + C with A (the map) in AGPRs.
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc) : "a"(w), "v"(x));
}
__device__ __forceinline__ void mfma_init(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x,
                                          const f32x4_t& c) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %3" : "=&v"(acc) : "a"(w), "v"(x), "v"(c));
}

// Pin values to a point of the instruction stream (between two matrix
// instructions): they are produced before it and consumed after it.
template <typename A>
__device__ __forceinline__ void pin(A& a) { asm volatile("" : "+v"(a)); }
template <typename A, typename B>
__device__ __forceinline__ void pin(A& a, B& b) { asm volatile("" : "+v"(a), "+v"(b)); }
template <typename A, typename B, typename C, typename E>
__device__ __forceinline__ void pin(A& a, B& b, C& c, E& e) {
  asm volatile("" : "+v"(a), "+v"(b), "+v"(c), "+v"(e));
}

// ---- LDS operations of one tile, in issue order (for the wait counts).
// Tile start: [keys: 2 coefficient reads, 2 reads of strip item 0] then the
// operand reads of steps 0 .. PF-1.  Step z: [keys, z % 4 == 1: 2 reads of
// strip item z/4 + 1] [operand read of step z + PF] ... [keys, z % 4 == 3: 2
// writes of strip item z/4].  pend(z) = operations issued after the operand
// read of step z when step z begins; LDS operations complete in order.
template <int K, bool KEYS>
struct LdsSched {
  static constexpr int Z = 4 * K;
  static constexpr int ops_before_step(int z) {   // operations issued before step z begins
    int n = KEYS ? 4 : 0;
    n += PF < Z ? PF : Z;
    for (int s = 0; s < z; ++s) {
      if (KEYS && s % 4 == 1 && s / 4 + 1 < K) n += 2;
      if (s + PF < Z) n += 1;
      if (KEYS && s % 4 == 3) n += 2;
    }
    return n;
  }
  static constexpr int frag_index(int z) {        // position of step z's operand read (1-based)
    if (z < PF) return (KEYS ? 4 : 0) + z + 1;
    const int s = z - PF;                          // issued during step s
    int n = ops_before_step(s);
    if (KEYS && s % 4 == 1 && s / 4 + 1 < K) n += 2;
    return n + 1;
  }
  static constexpr int pend(int z) { return ops_before_step(z) - frag_index(z); }
};

struct PipeCtx {
  int tid, lane, wave, c, row, sl, o, sr, sg, sh;
  int64_t t_begin, t_end;
  int n_tiles;
};

// One unit (layer group, head, K|V) of one workgroup.  KV is 0 for keys.
template <int K, int STYLE, bool SLOTS, int KV>
__device__ __forceinline__ void pipe_unit(const MapArgs& a, uint32_t lds0, const PipeCtx& q, int h,
                                          int ll0, bool has1) {
  using G = Geo<K>;
  constexpr int Z = G::Z;
  constexpr int NSLOT = G::NSLOT;
  constexpr bool KEYS = KV == 0;
  constexpr int N_DMA = NSLOT + (KEYS ? 1 : 0);      // buffer-to-LDS loads per wave per tile
  constexpr int N_CTL = (KEYS ? 2 : 0) + (SLOTS ? 1 : 0);   // register loads per tile
  // vector memory operations per tile, in order: [N_CTL register loads]
  // [N_DMA loads into LDS] [2 stores of the previous tile]
  constexpr int WAIT_DMA = 4 + N_CTL + N_DMA;        // DMA of tile i+2, at the end of tile i
  constexpr int WAIT_CTL = 2 * N_DMA + 2 + N_CTL;    // loads of tile i-1, at the start of tile i
  using S = LdsSched<K, KEYS>;

  const int c = q.c, row = q.row, sl = q.sl, o = q.o, wave = q.wave;
  const bool mine = sl == 0 || has1;
  const int T = a.T;
  const int64_t t_begin = q.t_begin, t_end = q.t_end;
  const int n_tiles = q.n_tiles;
  const uint32_t plane_bytes = (uint32_t)T * ROWB;

  // ---- buffers: the source plane of each slot, the RoPE tables, the target plane
  i32x4_t rs_src[NSLOT];
#pragma unroll
  for (int u = 0; u < NSLOT; ++u) {
    const int s = (u & 1) && has1 ? 1 : 0;
    const int sidx = a.idx[(ll0 + s) * K + (u >> 1)];
    rs_src[u] = make_rsrc(static_cast<const char*>(a.src) +
                              (((int64_t)sidx * 2 + KV) * a.H + h) * (int64_t)plane_bytes,
                          plane_bytes);
  }
  const i32x4_t rs_cs = make_rsrc(a.cs16, plane_bytes);
  const i32x4_t rs_ct = make_rsrc(a.cs16_tgt, plane_bytes);
  const i32x4_t rs_slot = make_rsrc(a.slots, (uint32_t)T * 4u);
  const uint32_t out_bytes = (uint32_t)a.tgt_rows * ROWB;
  const i32x4_t rs_out = make_rsrc(static_cast<char*>(a.tgt) +
                                       (((int64_t)(a.l0 + ll0 + (mine ? sl : 0)) * 2 + KV) * a.H + h) *
                                           (int64_t)out_bytes,
                                   out_bytes);

  // ---- this wave's map slice in AGPRs, and its bias as the accumulator's start
  u32x4_t wf[4][Z];
  f32x4_t bias[4];
  {
    const int l = a.l0 + ll0 + (mine ? sl : 0);
    const uint16_t* img = reinterpret_cast<const uint16_t*>(a.wpack) +
                          (((int64_t)l * a.H + h) * 2 + KV) * (int64_t)D * (K * D);
#pragma unroll
    for (int lb = 0; lb < 4; ++lb) {
      const int b = 4 * (lb >> 1) + 2 * o + (lb & 1);
      const uint16_t* r0 = img + (int64_t)(16 * b + row) * (K * D);
#pragma unroll
      for (int z = 0; z < Z; ++z)
        wf[lb][z] = *reinterpret_cast<const u32x4_t*>(r0 + 8 * ((4 * z + c) ^ row));
    }
    // accumulator element i of block lb is output channel
    // 64 (lb / 2) + 32 o + 8 c + 4 (lb % 2) + i: 8 contiguous channels per lb / 2
    const uint16_t* bp = reinterpret_cast<const uint16_t*>(KV ? a.bv : a.bk);
    u32x4_t bw[2] = {{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
    if (bp != nullptr) {
#pragma unroll
      for (int x = 0; x < 2; ++x)
        bw[x] = *reinterpret_cast<const u32x4_t*>(bp + ((int64_t)l * a.H + h) * D + 64 * x + 32 * o + 8 * c);
    }
#pragma unroll
    for (int lb = 0; lb < 4; ++lb)
#pragma unroll
      for (int i = 0; i < 4; i += 2) {
        const uint32_t wd = bw[lb >> 1][2 * (lb & 1) + i / 2];
        bias[lb][i] = lo_bf16(wd);
        bias[lb][i + 1] = hi_bf16(wd);
      }
  }
  // The map and bias loads are the compiler's own: wait for them here, with a
  // wait it knows of, so that it inserts none inside the tile loop.
  __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0)

  // ---- per-lane offsets that do not change from tile to tile
  // DMA: wave w loads tokens 4w .. 4w+3 of every slot; lane -> (token tr, position lane & 15)
  const int tr = 4 * wave + (q.lane >> 4);
  const uint32_t vo_row = (uint32_t)(tr * ROWB + 16 * ((q.lane & 15) ^ tr));
  const uint32_t vo_cs = (uint32_t)(tr * 256 + 16 * (q.lane & 15));
  // operand fragments: token row, chunk 4s + c at position (4s + c) ^ row
  uint32_t fpos[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) fpos[s] = (uint32_t)(row * ROWB + 16 * ((4 * s + c) ^ row) + sl * SLOTB);
  // strip pass: thread (token sr, chunk pair sg / sg + 8, slot parity sh)
  const uint32_t sposx = (uint32_t)(q.sh * SLOTB + q.sr * ROWB + 16 * (q.sg ^ q.sr));
  const uint32_t sposy = (uint32_t)(q.sh * SLOTB + q.sr * ROWB + 16 * ((q.sg + 8) ^ q.sr));
  const uint32_t scs = (uint32_t)(G::CS_OFF + q.sr * 256 + (STYLE == 0 ? 32 * q.sg : 16 * q.sg));
  // target coefficients of this lane's output planes, and its output columns
  const uint32_t vo_ct = (uint32_t)(row * 256 + (STYLE == 0 ? 4 * (32 * o + 8 * c) : 2 * (32 * o + 8 * c)));
  const uint32_t colb = (uint32_t)(2 * (32 * o + 8 * c));

  auto tile_soff = [&](int j) __attribute__((always_inline)) -> uint32_t {
    return (uint32_t)((t_begin + (int64_t)MT * j) * ROWB);
  };
  // Loads of tile j into stage st (the tile may lie past the end: rows past
  // the plane read as zero, and nothing of them is stored).
  auto dma_tile = [&](int st, int j) __attribute__((always_inline)) {
    const uint32_t so = tile_soff(j);
    const uint32_t base = lds0 + (uint32_t)(st * G::STAGE + wave * 1024);
#pragma unroll
    for (int u = 0; u < NSLOT; ++u) dma16(base + u * SLOTB, vo_row, rs_src[u], so);
    if (KEYS) dma16(base + G::CS_OFF, vo_cs, rs_cs, so);
  };
  // Register loads of tile j: target coefficients (keys) and slot of the row.
  u32x4_t ct[2][2];
  uint32_t slotv[2];
  auto ctl_tile = [&](int p, int j) __attribute__((always_inline)) {
    if (KEYS) {
      const uint32_t so = tile_soff(j);
      vload16(ct[p][0], vo_ct, rs_ct, so);
      vload16(ct[p][1], vo_ct + (STYLE == 0 ? 16u : 128u), rs_ct, so);
    }
    if (SLOTS) vload4(slotv[p], (uint32_t)(row * 4), rs_slot, (uint32_t)((t_begin + (int64_t)MT * j) * 4));
  };
  // Store address of this lane's row of tile j: outside the target when the
  // token is past the part or its slot is outside the pool.
  auto out_voff = [&](int p, int j) __attribute__((always_inline)) -> uint32_t {
    const int64_t tl = t_begin + (int64_t)MT * j + row;
    int64_t orow = SLOTS ? (int64_t)(int32_t)slotv[p] : tl;
    const bool ok = mine && j >= 0 && tl < t_end && orow >= 0 && orow < a.tgt_rows;
    return ok ? (uint32_t)orow * ROWB + colb : 0xffffff00u;
  };

  // ---- epilogue of tile j from accumulator set p: target RoPE (keys),
  // rounding to bf16, two 16-byte stores (64 contiguous bytes per 4 lanes).
  f32x4_t acc[2][4];
  auto epilogue = [&](int p, int j) __attribute__((always_inline)) {
    float y[2][8];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        y[x][i] = acc[p][2 * x][i];
        y[x][4 + i] = acc[p][2 * x + 1][i];
      }
    if (KEYS) {
      uint32_t cw[8];
      unpack4(ct[p][0], cw);
      unpack4(ct[p][1], cw + 4);
      if (STYLE == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) rot_fwd16(y[0][e], y[1][e], cw[e]);
      } else {
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int e = 0; e < 8; e += 2) rot_fwd16(y[x][e], y[x][e + 1], cw[4 * x + e / 2]);
      }
    }
    const uint32_t vo = out_voff(p, j);
    u32x4_t v0, v1;
    v0[0] = pack2(y[0][0], y[0][1]);
    v0[1] = pack2(y[0][2], y[0][3]);
    v0[2] = pack2(y[0][4], y[0][5]);
    v0[3] = pack2(y[0][6], y[0][7]);
    v1[0] = pack2(y[1][0], y[1][1]);
    v1[1] = pack2(y[1][2], y[1][3]);
    v1[2] = pack2(y[1][4], y[1][5]);
    v1[3] = pack2(y[1][6], y[1][7]);
    vstore16<0>(v0, vo, rs_out);
    vstore16<128>(v1, vo, rs_out);
  };

  // ---- strip pass (keys): item jj = slot 2 jj + sh of the thread's token
  // and chunk pair, x = chunk sg (first channels), y = chunk sg + 8.
  u32x4_t sx[2], sy[2], scw[2];
  auto strip_read = [&](uint32_t bx, uint32_t by, int jj) __attribute__((always_inline)) {
    switch (jj) {
      case 0: lds_read<0>(sx[0], bx); lds_read<0>(sy[0], by); break;
      case 1: lds_read<2 * SLOTB>(sx[1], bx); lds_read<2 * SLOTB>(sy[1], by); break;
      case 2: lds_read<4 * SLOTB>(sx[0], bx); lds_read<4 * SLOTB>(sy[0], by); break;
      default: lds_read<6 * SLOTB>(sx[1], bx); lds_read<6 * SLOTB>(sy[1], by); break;
    }
  };
  auto strip_write = [&](uint32_t bx, uint32_t by, int jj) __attribute__((always_inline)) {
    switch (jj) {
      case 0: lds_write<0>(bx, sx[0]); lds_write<0>(by, sy[0]); break;
      case 1: lds_write<2 * SLOTB>(bx, sx[1]); lds_write<2 * SLOTB>(by, sy[1]); break;
      case 2: lds_write<4 * SLOTB>(bx, sx[0]); lds_write<4 * SLOTB>(by, sy[0]); break;
      default: lds_write<6 * SLOTB>(bx, sx[1]); lds_write<6 * SLOTB>(by, sy[1]); break;
    }
  };
  auto strip_coef_read = [&](uint32_t cbase) __attribute__((always_inline)) {
    lds_read<0>(scw[0], cbase);
    lds_read<(STYLE == 0 ? 16 : 128)>(scw[1], cbase);
  };
  // word w of item set p, in four parts (one after each matrix instruction)
  float su0, su1, sv0, sv1;
  auto strip_part = [&](int p, int w, int part) __attribute__((always_inline)) {
    if (part == 0) {
      uint32_t xa = sx[p][w], ya = sy[p][w];
      pin(xa, ya);
      su0 = lo_bf16(xa);
      su1 = hi_bf16(xa);
      sv0 = lo_bf16(ya);
      sv1 = hi_bf16(ya);
      pin(su0, su1, sv0, sv1);
    } else if (part == 1) {
      if (STYLE == 0) strip(su0, sv0, scw[w >> 1][2 * (w & 1)]);
      else strip(su0, su1, scw[0][w]);
      pin(su0, su1, sv0, sv1);
    } else if (part == 2) {
      if (STYLE == 0) strip(su1, sv1, scw[w >> 1][2 * (w & 1) + 1]);
      else strip(sv0, sv1, scw[1][w]);
      pin(su0, su1, sv0, sv1);
    } else {
      uint32_t xa = pack2(su0, su1), ya = pack2(sv0, sv1);
      pin(xa, ya);
      sx[p][w] = xa;
      sy[p][w] = ya;
    }
  };

  // ---- pipeline prologue: tiles 0..2 in flight, the register loads and
  // stores that the steady state expects before them
  const uint32_t vo_none = 0xffffff00u;
  {
    u32x4_t zero4 = {0u, 0u, 0u, 0u};
    dma_tile(0, 0);
    ctl_tile(0, 0);
    dma_tile(1, 1);
    vstore16<0>(zero4, vo_none, rs_out);
    vstore16<128>(zero4, vo_none, rs_out);
    ctl_tile(1, 0);
    dma_tile(2, 2);
    vstore16<0>(zero4, vo_none, rs_out);
    vstore16<128>(zero4, vo_none, rs_out);
    vm_wait<WAIT_DMA>();                       // tiles 0 and 1 are in LDS
    // The first register loads above only keep the counts of the steady
    // state; their values are never used.  The hardware still writes them:
    // keep the registers reserved until the wait has seen them land.
    if (KEYS) pin(ct[0][0], ct[0][1]);
    if (SLOTS) pin(slotv[0]);
  }
  __syncthreads();
  if (KEYS) {
    // strip stage 0 before the first tile
    const uint32_t bx = lds0 + sposx, by = lds0 + sposy;
    strip_coef_read(lds0 + scs);
#pragma unroll
    for (int jj = 0; jj < K; ++jj) {
      const int p = jj & 1;
      strip_read(bx, by, jj);
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(sx[p]), "+v"(sy[p]), "+v"(scw[0]), "+v"(scw[1]));
      uint32_t cw[8];
      unpack4(scw[0], cw);
      unpack4(scw[1], cw + 4);
      if (STYLE == 0) {
        strip_halfsplit(sx[p], sy[p], cw);
      } else {
        strip_interleaved(sx[p], cw);
        strip_interleaved(sy[p], cw + 4);
      }
      strip_write(bx, by, jj);
    }
    lds_drain();
    __syncthreads();
  }
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int lb = 0; lb < 4; ++lb) acc[p][lb] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  // ---- tile i in stage ST = i % 4 with accumulator set P = i % 2.  On entry
  // (after a barrier): stage ST holds tile i ready for the matrix cores, stage
  // ST+1 holds tile i+1 as loaded, stage ST+2 is being loaded, stage ST+3 is free.
  auto tile = [&](auto stc, int i) __attribute__((always_inline)) {
    constexpr int ST = decltype(stc)::value;
    constexpr int P = ST & 1;
    constexpr int ST1 = (ST + 1) % NSTAGE;
    constexpr int ST3 = (ST + 3) % NSTAGE;
    const uint32_t sbx = lds0 + ST1 * G::STAGE + sposx;       // strip pass on tile i+1
    const uint32_t sby = lds0 + ST1 * G::STAGE + sposy;
    uint32_t fa[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) fa[s] = lds0 + ST * G::STAGE + fpos[s];
    // LDS: strip coefficients and item 0 of tile i+1, operand reads of steps 0..PF-1
    if (KEYS) {
      strip_coef_read(lds0 + ST1 * G::STAGE + scs);
      strip_read(sbx, sby, 0);
    }
    u32x4_t xf[PF + 1];
    auto frag_read = [&](int z) __attribute__((always_inline)) {
      u32x4_t& d = xf[z % (PF + 1)];
      switch (z / 4) {
        case 0: lds_read<0>(d, fa[z % 4]); break;
        case 1: lds_read<2 * SLOTB>(d, fa[z % 4]); break;
        case 2: lds_read<4 * SLOTB>(d, fa[z % 4]); break;
        default: lds_read<6 * SLOTB>(d, fa[z % 4]); break;
      }
    };
#pragma unroll
    for (int z = 0; z < PF && z < Z; ++z) frag_read(z);
    // memory: register loads of tile i, then tile i+3 into the free stage
    ctl_tile(P, i);
    dma_tile(ST3, i + 3);
    // epilogue of tile i-1 (for tile 0: a tile before the part, nothing stored)
    if (KEYS) {
      vm_wait<WAIT_CTL>(ct[P ^ 1][1]);
      pin(ct[P ^ 1][0]);
    } else if (SLOTS) {
      vm_wait<WAIT_CTL>(slotv[P ^ 1]);
    }
    if (KEYS && SLOTS) pin(slotv[P ^ 1]);
    epilogue(P ^ 1, i - 1);

    // contraction: step z waits for its operand, issues the read for step
    // z + PF, then four matrix instructions with the strip pass between them
#pragma unroll
    for (int z = 0; z < Z; ++z) {
      lds_wait_n(S::pend(z), xf[z % (PF + 1)]);
      const int jj = z / 4, w = z % 4, p = jj & 1;
      if (KEYS && w == 0) pin(sx[p], sy[p], scw[0], scw[1]);   // item jj and coefficients arrived
      if (KEYS && w == 1 && jj + 1 < K) strip_read(sbx, sby, jj + 1);
      if (z + PF < Z) frag_read(z + PF);
      const u32x4_t& x = xf[z % (PF + 1)];
#pragma unroll
      for (int lb = 0; lb < 4; ++lb) {
        if (z == 0) mfma_init(acc[P][lb], wf[lb][z], x, bias[lb]);
        else mfma_acc(acc[P][lb], wf[lb][z], x);
        if (KEYS) strip_part(p, w, lb);
      }
      if (KEYS && w == 3) strip_write(sbx, sby, jj);
    }
    // tile i+2 is in LDS (this wave's part), the strip writes are done
    vm_wait<WAIT_DMA>();
    lds_drain();
    __syncthreads();
  };

  // Epilogue of the last tile: its register loads were followed by one
  // tile's loads into LDS and two stores.
  auto final_epilogue = [&](int p, int j) __attribute__((always_inline)) {
    vm_wait<0>();
    if (KEYS) pin(ct[p][0], ct[p][1]);
    if (SLOTS) pin(slotv[p]);
    epilogue(p, j);
  };

  // Four tiles per trip, so that stages and accumulator sets are constants.
  for (int i0 = 0; i0 < n_tiles; i0 += 4) {
    tile(std::integral_constant<int, 0>{}, i0);
    if (i0 + 1 >= n_tiles) { final_epilogue(0, i0); break; }
    tile(std::integral_constant<int, 1>{}, i0 + 1);
    if (i0 + 2 >= n_tiles) { final_epilogue(1, i0 + 1); break; }
    tile(std::integral_constant<int, 2>{}, i0 + 2);
    if (i0 + 3 >= n_tiles) { final_epilogue(0, i0 + 2); break; }
    tile(std::integral_constant<int, 3>{}, i0 + 3);
    if (i0 + 4 >= n_tiles) { final_epilogue(1, i0 + 3); break; }
  }
  // everything this unit issued has landed before the next one reuses LDS
  vm_wait<0>();
  __syncthreads();
}

template <int K, int STYLE, bool SLOTS>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void map_pipe_kernel(const MapArgs a, const SweepPlan p) {
  __shared__ __attribute__((aligned(16))) char smem[Geo<K>::LDS];
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_u32(smem));

  PipeCtx q;
  q.tid = threadIdx.x;
  q.lane = q.tid & 63;
  q.wave = __builtin_amdgcn_readfirstlane(q.tid >> 6);
  q.c = q.lane >> 4;        // reduction chunk of an MFMA fragment
  q.row = q.lane & 15;      // token (B, D) or map row (A) within a block
  q.sl = q.wave >> 1;       // layer slot of the pair
  q.o = q.wave & 1;         // output half
  q.sr = q.tid >> 4;        // strip pass: token of the tile
  q.sg = (q.tid >> 1) & 7;  // strip pass: chunk pair sg, sg + 8
  q.sh = q.tid & 1;         // strip pass: slot parity (layer of the pair)

  const int slot = blockIdx.x >> 3;   // CU slot within the XCD (0 .. 31)
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
    const int pairs = (g_n + 1) / 2;
    const int parts = 32 / pairs;
    const int pair = slot % pairs;
    const int part = slot / pairs;
    const int64_t per = ((int64_t)a.T + parts - 1) / parts;
    const int64_t part_len = (per + MT - 1) / MT * MT;
    q.t_begin = (int64_t)part * part_len;
    if (part >= parts || q.t_begin >= a.T) continue;   // same decision in every thread
    q.t_end = q.t_begin + part_len < a.T ? q.t_begin + part_len : a.T;
    q.n_tiles = (int)((q.t_end - q.t_begin + MT - 1) / MT);
    const int ll0 = g0 + 2 * pair;
    const bool has1 = 2 * pair + 1 < g_n;
    if (kv == 0)
      pipe_unit<K, STYLE, SLOTS, 0>(a, lds0, q, h, ll0, has1);
    else
      pipe_unit<K, STYLE, SLOTS, 1>(a, lds0, q, h, ll0, has1);
  }
}

template <int K, int STYLE>
hipError_t launch_pk(const MapArgs& a, const SweepPlan& p, hipStream_t stream) {
  if (a.slots != nullptr)
    hipLaunchKernelGGL((map_pipe_kernel<K, STYLE, true>), dim3(256), dim3(NT), 0, stream, a, p);
  else
    hipLaunchKernelGGL((map_pipe_kernel<K, STYLE, false>), dim3(256), dim3(NT), 0, stream, a, p);
  return hipGetLastError();
}

template <int K>
hipError_t launch_pstyle(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  return style == 0 ? launch_pk<K, 0>(a, p, stream) : launch_pk<K, 1>(a, p, stream);
}

}  // namespace

bool map_pipe_supported(int64_t T, int64_t tgt_rows) {
  // byte offsets within a plane, and of the tiles loaded ahead past its end,
  // must fit the 32-bit buffer offsets
  return T >= 1 && (T + 64) * ROWB < 0xffffff00LL && tgt_rows * ROWB < 0xffffff00LL;
}

hipError_t launch_map_pipe(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  if (a.T == 0 || a.nl == 0) return hipSuccess;
  switch (a.k) {
    case 1: return launch_pstyle<1>(a, p, style, stream);
    case 2: return launch_pstyle<2>(a, p, style, stream);
    case 3: return launch_pstyle<3>(a, p, style, stream);
    case 4: return launch_pstyle<4>(a, p, style, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kvx
