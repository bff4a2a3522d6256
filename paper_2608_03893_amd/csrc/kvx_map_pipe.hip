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
#include "kvx_asm.h"
#include "kvx_bf16.h"
#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int D = 128;
constexpr int MT = 16;                   // tokens per tile
constexpr int NT = 256;                  // threads per workgroup
constexpr int ROWB = D * 2;              // bytes per token row
constexpr int SLOTB = MT * ROWB;         // slot stride in LDS
constexpr int CSB = MT * 256;            // coefficient block of a stage
constexpr int NSTAGE = 4;
constexpr int PF = 3;                    // operand reads issued ahead of their step

// Stage layouts.  Key units: 2k slots, the source and (TGT) target RoPE
// coefficients, (SLOTS) the slot indices; four stages.  Value units need no
// coefficients: 2k slots and the slot indices, in as many stages (up to
// five) as fit, so that their loads have a tile longer to arrive.
template <int K, bool SLOTS, bool TGT>
struct Geo {
  static constexpr int NSLOT = 2 * K;
  static constexpr int CS_OFF = NSLOT * SLOTB;             // source RoPE (cos, sin)
  static constexpr int CT_OFF = CS_OFF + CSB;              // target RoPE (cos, sin), TGT
  static constexpr int SL_OFF = CS_OFF + (TGT ? 2 : 1) * CSB;   // slot indices, 256 B per wave
  static constexpr int STAGE = SL_OFF + (SLOTS ? 1024 : 0);
  static constexpr int VSL_OFF = NSLOT * SLOTB;
  static constexpr int VSTAGE = VSL_OFF + (SLOTS ? 1024 : 0);
  static constexpr int NV = 5 * VSTAGE <= 160 * 1024 ? 5 : NSTAGE;
  static constexpr int LDS = NSTAGE * STAGE > NV * VSTAGE ? NSTAGE * STAGE : NV * VSTAGE;
  static constexpr int Z = 4 * K;        // reduction steps per tile
  static constexpr bool fits = LDS <= 160 * 1024;
};
static_assert(Geo<4, false, true>::fits && Geo<4, true, false>::fits && Geo<3, true, true>::fits,
              "stages fit the LDS of a CU");

// ---- LDS operations of one tile, in issue order (for the wait counts).
// Tile start: [keys: 2 coefficient reads, 2 reads of strip item 0] then the
// operand reads of steps 0 .. PF-1.  Step z: [keys, z % 4 == 1: 2 reads of
// strip item z/4 + 1] [operand read of step z + PF] ... [keys, z % 4 == 3: 2
// writes of strip item z/4] [z == Z - 3: the E reads of the epilogue's
// inputs].  pend(z) = operations issued after the operand read of step z when
// step z begins; LDS operations complete in order.  PRE: the operand reads of
// steps 0 .. PF-1 were issued (and completed) before the tile's barrier.
template <int K, bool KEYS, int E, bool PRE>
struct LdsSched {
  static constexpr int Z = 4 * K;
  static constexpr int ops_before_step(int z) {   // operations issued before step z begins
    int n = KEYS ? 4 : 0;
    n += PRE ? 0 : (PF < Z ? PF : Z);
    for (int s = 0; s < z; ++s) {
      if (KEYS && s % 4 == 1 && s / 4 + 1 < K) n += 2;
      if (s + PF < Z) n += 1;
      if (KEYS && s % 4 == 3) n += 2;
      if (s == Z - 3) n += E;
    }
    return n;
  }
  static constexpr int frag_index(int z) {        // position of step z's operand read (1-based)
    if (z < PF) return PRE ? 0 : (KEYS ? 4 : 0) + z + 1;
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
// TGT: the target RoPE differs from the source RoPE (its coefficients get a
// block of their own in each stage).
template <int K, int STYLE, bool SLOTS, bool TGT, int KV>
__device__ __forceinline__ void pipe_unit(const MapArgs& a, uint32_t lds0, const PipeCtx& q, int h,
                                          int ll0, bool has1) {
  using G = Geo<K, SLOTS, TGT>;
  constexpr int Z = G::Z;
  constexpr int NSLOT = G::NSLOT;
  constexpr bool KEYS = KV == 0;
  // buffer-to-LDS loads per wave per tile: its 4 rows of every slot, of the
  // source (keys) and target (keys, TGT) coefficients, and the tile's slot
  // indices (SLOTS)
  constexpr int N_DMA = NSLOT + (KEYS ? 1 : 0) + (KEYS && TGT ? 1 : 0) + (SLOTS ? 1 : 0);
  constexpr int NS = KEYS ? NSTAGE : G::NV;            // stages of the ring
  constexpr int SB = KEYS ? G::STAGE : G::VSTAGE;      // bytes per stage
  constexpr int SLOFF = KEYS ? G::SL_OFF : G::VSL_OFF;  // slot indices in a stage
  // at the end of tile i the loads of tile i+2 must have landed; those of
  // tiles i+3 .. i+NS-1 are the only loads into LDS issued after them
  constexpr int WAIT_DMA = (NS - 3) * N_DMA;
  // Values have no strip pass: the stage of tile i+1 is complete when tile i
  // begins, so tile i+1's first operand reads are issued before the barrier
  // that ends tile i.
  constexpr bool PRE = !KEYS;
  using S = LdsSched<K, KEYS, (KEYS ? 2 : 0) + (SLOTS ? 1 : 0), PRE>;
  // the tile's N_DMA buffer loads, then the two stores of the previous tile,
  // spread evenly over its reduction steps
  constexpr int N_VM = N_DMA + 2;
  static_assert(Z >= 4, "at least four reduction steps");

  const int c = q.c, row = q.row, sl = q.sl, o = q.o, wave = q.wave;
  const bool mine = sl == 0 || has1;
  const int T = a.T;
  const int64_t t_begin = q.t_begin, t_end = q.t_end;
  const int n_tiles = q.n_tiles;
  const uint32_t plane_bytes = (uint32_t)T * ROWB;

  // ---- buffers: the source plane of each slot, the RoPE tables, the slot
  // indices, the target plane
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
  // DMA: wave w loads tokens 4w .. 4w+3 of every slot; lane -> (token tr,
  // position lane & 15), which holds chunk position ^ tr ^ 8 (slot parity)
  const int tr = 4 * wave + (q.lane >> 4);
  uint32_t vo_row[2];
#pragma unroll
  for (int par = 0; par < 2; ++par)
    vo_row[par] = (uint32_t)(tr * ROWB + 16 * ((q.lane & 15) ^ tr ^ (8 * par)));
  const uint32_t vo_cs = vo_row[0];   // coefficient rows: position ^ tr as well
  const uint32_t vo_slot = (uint32_t)(4 * (q.lane & 15));
  // operand fragments: token row, chunk 4s + c of the wave's layer sl
  uint32_t fpos[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    fpos[s] = (uint32_t)(sl * SLOTB + row * ROWB + 16 * ((4 * s + c) ^ row ^ (8 * sl)));
  // strip pass: thread (token sr, chunk pair sg / sg + 8, slot parity sh)
  const uint32_t sposx = (uint32_t)(q.sh * SLOTB + q.sr * ROWB + 16 * (q.sg ^ q.sr ^ (8 * q.sh)));
  // coefficient rows: 16-byte piece q of token r at position q ^ r.  The
  // strip pass needs the planes of chunks sg and sg + 8 of its token; the
  // epilogue the planes of its 16 output channels.
  const int sq0 = STYLE == 0 ? 2 * q.sg : q.sg, sq1 = STYLE == 0 ? 2 * q.sg + 1 : 8 + q.sg;
  const uint32_t scs0 = (uint32_t)(G::CS_OFF + q.sr * 256 + 16 * (sq0 ^ q.sr));
  constexpr uint32_t SX1 = STYLE == 0 ? 16u : 128u;   // second piece: position bit 0 or 3 flipped
  (void)sq1;
  const int eq0 = STYLE == 0 ? 8 * o + 2 * c : 4 * o + c;
  const int eq1 = STYLE == 0 ? 8 * o + 2 * c + 1 : 8 + 4 * o + c;
  const uint32_t vct0 = (uint32_t)((TGT ? G::CT_OFF : G::CS_OFF) + row * 256 + 16 * (eq0 ^ row));
  (void)eq1;
  const uint32_t colb = (uint32_t)(2 * (32 * o + 8 * c));

  auto tile_soff = [&](int j) __attribute__((always_inline)) -> uint32_t {
    return (uint32_t)((t_begin + (int64_t)MT * j) * ROWB);
  };
  // Load m of tile j into stage st (the tile may lie past the end: rows past
  // the plane read as zero, and nothing of them is stored).
  auto dma_one = [&](int st, int j, int m) __attribute__((always_inline)) {
    const uint32_t so = __builtin_amdgcn_readfirstlane(tile_soff(j));
    const uint32_t base = lds0 + (uint32_t)(st * SB + wave * 1024);
    if (m < NSLOT) {
      dma16(base + m * SLOTB, vo_row[m & 1], rs_src[m], so);
    } else if (KEYS && m == NSLOT) {
      dma16(base + G::CS_OFF, vo_cs, rs_cs, so);
    } else if (KEYS && TGT && m == NSLOT + 1) {
      dma16(base + G::CT_OFF, vo_cs, rs_ct, so);
    } else {
      dma4(lds0 + (uint32_t)(st * SB + SLOFF + wave * 256), vo_slot, rs_slot,
           __builtin_amdgcn_readfirstlane((uint32_t)((t_begin + (int64_t)MT * j) * 4)));
    }
  };
  auto dma_tile = [&](int st, int j) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < N_DMA; ++m) dma_one(st, j, m);
  };

  // ---- epilogue of tile j from accumulator set p: target RoPE (keys),
  // rounding to bf16, two 16-byte stores (64 contiguous bytes per 4 lanes).
  // ct and slotv were read from the tile's stage at its end.
  f32x4_t acc[2][4];
  u32x4_t ct[2] = {{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
  uint32_t slotv = 0;
  u32x4_t ev[2];
  uint32_t eo = 0;
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
      unpack4(ct[0], cw);
      unpack4(ct[1], cw + 4);
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
    // store address of this lane's row: outside the target when the token is
    // past the part or its slot is outside the pool
    const int64_t tl = t_begin + (int64_t)MT * j + row;
    const int64_t orow = SLOTS ? (int64_t)(int32_t)slotv : tl;
    const bool ok = mine && j >= 0 && tl < t_end && orow >= 0 && orow < a.tgt_rows;
    eo = ok ? (uint32_t)orow * ROWB + colb : 0xffffff00u;
    u32x4_t& v0 = ev[0];
    u32x4_t& v1 = ev[1];
    v0[0] = pack2(y[0][0], y[0][1]);
    v0[1] = pack2(y[0][2], y[0][3]);
    v0[2] = pack2(y[0][4], y[0][5]);
    v0[3] = pack2(y[0][6], y[0][7]);
    v1[0] = pack2(y[1][0], y[1][1]);
    v1[1] = pack2(y[1][2], y[1][3]);
    v1[2] = pack2(y[1][4], y[1][5]);
    v1[3] = pack2(y[1][6], y[1][7]);
  };
  auto epilogue_store = [&](int x) __attribute__((always_inline)) {
    if (x == 0) vstore16<0>(ev[0], eo, rs_out);
    else vstore16<128>(ev[1], eo, rs_out);
  };
  // After tile j's contraction, while its stage is intact: the coefficients
  // and the slot of this lane's row, for the epilogue of tile j.
  auto epilogue_reads = [&](int st) __attribute__((always_inline)) {
    const uint32_t base = lds0 + (uint32_t)(st * SB);
    if (KEYS) {
      lds_read<0>(ct[0], base + vct0);
      lds_read<0>(ct[1], (base + vct0) ^ SX1);
    }
    if (SLOTS) lds_read_b32(slotv, lds0 + (uint32_t)(st * SB + SLOFF + row * 4));
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
  auto strip_coef_read = [&](uint32_t sbase) __attribute__((always_inline)) {
    lds_read<0>(scw[0], sbase + scs0);
    lds_read<0>(scw[1], (sbase + scs0) ^ SX1);
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

  // ---- pipeline prologue: tiles 0 .. NS-2 in flight; stage 0 stripped
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) dma_tile(j, j);
  vm_wait<WAIT_DMA>();                         // tiles 0 and 1 are in LDS
  __syncthreads();
  if (KEYS) {
    const uint32_t bx = lds0 + sposx, by = bx ^ 128u;   // chunk sg + 8: position bit 3 flipped
    strip_coef_read(lds0);
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

  // operand fragment of step z of the tile whose stage addresses are fa
  u32x4_t xf[PF + 1];
  auto frag_read = [&](const uint32_t (&fa)[4], int z) __attribute__((always_inline)) {
    u32x4_t& d = xf[z % (PF + 1)];
    switch (z / 4) {
      case 0: lds_read<0>(d, fa[z % 4]); break;
      case 1: lds_read<2 * SLOTB>(d, fa[z % 4]); break;
      case 2: lds_read<4 * SLOTB>(d, fa[z % 4]); break;
      default: lds_read<6 * SLOTB>(d, fa[z % 4]); break;
    }
  };
  auto pre_reads = [&](int st) __attribute__((always_inline)) {
    uint32_t fb[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) fb[s] = lds0 + st * SB + fpos[s];
#pragma unroll
    for (int z = 0; z < PF && z < Z; ++z) frag_read(fb, z);
  };
  if (PRE) {
    pre_reads(0);
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xf[0]), "+v"(xf[1]), "+v"(xf[2]));
  }

  // ---- tile i in stage ST = i % NS with accumulator set P = i % 2.  On
  // entry (after a barrier): stage ST holds tile i ready for the matrix
  // cores, stage ST+1 holds tile i+1 as loaded, stages ST+2 .. ST+NS-2 are
  // being loaded, stage ST+NS-1 is free; ct / slotv hold the epilogue inputs
  // of tile i-1.
  auto tile = [&](auto pc, int i, int ST) __attribute__((always_inline)) {
    constexpr int P = decltype(pc)::value;
    const int ST1 = ST + 1 == NS ? 0 : ST + 1;
    const int STF = ST == 0 ? NS - 1 : ST - 1;                 // the free stage
    const uint32_t sbx = lds0 + ST1 * SB + sposx;              // strip pass on tile i+1
    const uint32_t sby = sbx ^ 128u;
    uint32_t fa[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) fa[s] = lds0 + ST * SB + fpos[s];
    // LDS: strip coefficients and item 0 of tile i+1, operand reads of steps 0..PF-1
    if (KEYS) {
      strip_coef_read(lds0 + ST1 * SB);
      strip_read(sbx, sby, 0);
    }
    if (!PRE) {
#pragma unroll
      for (int z = 0; z < PF && z < Z; ++z) frag_read(fa, z);
    }
    // epilogue of tile i-1 (for tile 0: a tile before the part, nothing
    // stored); its two stores are issued during the contraction
    epilogue(P ^ 1, i - 1);

    // contraction: step z waits for its operand, issues the read for step
    // z + PF, then four matrix instructions with the strip pass between them;
    // tile i+3 is loaded into the free stage a few buffer loads per step, so
    // that no wave blocks on a full memory queue while its matrix core waits
#pragma unroll
    for (int z = 0; z < Z; ++z) {
      lds_wait_n(S::pend(z), xf[z % (PF + 1)]);
      const int jj = z / 4, w = z % 4, p = jj & 1;
      if (KEYS && w == 0) pin(sx[p], sy[p], scw[0], scw[1]);   // item jj and coefficients arrived
      if (KEYS && w == 1 && jj + 1 < K) strip_read(sbx, sby, jj + 1);
      if (z + PF < Z) frag_read(fa, z + PF);
      const u32x4_t& x = xf[z % (PF + 1)];
#pragma unroll
      for (int lb = 0; lb < 4; ++lb) {
        if (z == 0) mfma_init(acc[P][lb], wf[lb][z], x, bias[lb]);
        else mfma_acc(acc[P][lb], wf[lb][z], x);
        if (KEYS) strip_part(p, w, lb);
      }
      if (KEYS && w == 3) strip_write(sbx, sby, jj);
#pragma unroll
      for (int m = 0; m < N_VM; ++m)
        if (m * Z / N_VM == z) {
          if (m < N_DMA) dma_one(STF, i + NS - 1, m);
          else epilogue_store(m - N_DMA);
        }
      if (z == Z - 3) epilogue_reads(ST);
    }
    if (PRE) pre_reads(ST1);
    // tile i+2 is in LDS: loads into LDS retire in order among themselves
    vm_wait<WAIT_DMA>();
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(ct[0]), "+v"(ct[1]), "+v"(slotv));
    if (PRE) pin(xf[0], xf[1]), pin(xf[2]);
    __syncthreads();
  };

  // Two tiles per trip, so that the accumulator sets are constants.
  int st = 0;
  for (int i0 = 0; i0 < n_tiles; i0 += 2) {
    tile(std::integral_constant<int, 0>{}, i0, st);
    st = st + 1 == NS ? 0 : st + 1;
    if (i0 + 1 >= n_tiles) { epilogue(0, i0); epilogue_store(0); epilogue_store(1); break; }
    tile(std::integral_constant<int, 1>{}, i0 + 1, st);
    st = st + 1 == NS ? 0 : st + 1;
    if (i0 + 2 >= n_tiles) { epilogue(1, i0 + 1); epilogue_store(0); epilogue_store(1); break; }
  }
  // everything this unit issued has landed before the next one reuses LDS
  vm_wait<0>();
  __syncthreads();
}

template <int K, int STYLE, bool SLOTS, bool TGT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void map_pipe_kernel(const MapArgs a, const SweepPlan p) {
  __shared__ __attribute__((aligned(256))) char smem[Geo<K, SLOTS, TGT>::LDS];
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
      pipe_unit<K, STYLE, SLOTS, TGT, 0>(a, lds0, q, h, ll0, has1);
    else
      pipe_unit<K, STYLE, SLOTS, TGT, 1>(a, lds0, q, h, ll0, has1);
  }
}

template <int K, int STYLE, bool SLOTS, bool TGT>
hipError_t launch_pk(const MapArgs& a, const SweepPlan& p, hipStream_t stream) {
  if constexpr (Geo<K, SLOTS, TGT>::fits) {
    hipLaunchKernelGGL((map_pipe_kernel<K, STYLE, SLOTS, TGT>), dim3(256), dim3(NT), 0, stream, a, p);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <int K, int STYLE>
hipError_t launch_pslots(const MapArgs& a, const SweepPlan& p, hipStream_t stream) {
  const bool slots = a.slots != nullptr, tgt = a.cs16_tgt != a.cs16;
  if (slots)
    return tgt ? launch_pk<K, STYLE, true, true>(a, p, stream) : launch_pk<K, STYLE, true, false>(a, p, stream);
  return tgt ? launch_pk<K, STYLE, false, true>(a, p, stream) : launch_pk<K, STYLE, false, false>(a, p, stream);
}

template <int K>
hipError_t launch_pstyle(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  return style == 0 ? launch_pslots<K, 0>(a, p, stream) : launch_pslots<K, 1>(a, p, stream);
}

}  // namespace

bool map_pipe_supported(int k, int64_t T, int64_t tgt_rows, bool slots, bool tgt_rope) {
  // byte offsets within a plane, and of the tiles loaded ahead past its end,
  // must fit the 32-bit buffer offsets; the stages must fit the LDS
  if (T < 1 || (T + 64) * ROWB >= 0xffffff00LL || tgt_rows * ROWB >= 0xffffff00LL) return false;
  if (k < 1 || k > 4) return false;
  const int stage = 2 * k * SLOTB + (tgt_rope ? 2 : 1) * CSB + (slots ? 1024 : 0);
  return NSTAGE * stage <= 160 * 1024;   // value stages are smaller
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
