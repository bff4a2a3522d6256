// K-split layer-sweep map kernel for bf16 caches with head dimension 128 and
// k <= 4.
//
// The work decomposition across the chip is the layer sweep's: one workgroup
// per CU, 4 waves (one per SIMD, all 512 registers), a unit of work is (layer
// group, head, K|V), workgroup b runs on XCD b % 8 and takes CU slot b / 8 of
// it, and in a unit CU slot j owns a pair of target layers and a token part,
// so that one XCD sweeps every target layer of a (head, K|V) over the same
// tokens at the same time and each source row comes from HBM once.
//
// Within a workgroup the two waves of a target layer split the reduction
// (Eq. ridge_kv: the concatenation of the k source blocks times the map)
// instead of the output channels.  Wave (s, h) of layer s holds in AGPRs the
// map rows of reduction steps h * 2k .. h * 2k + 2k - 1 for all 128 output
// channels (8 output blocks x 2k steps of v_mfma_f32_16x16x32_bf16
// A-fragments), so every operand fragment read from LDS has exactly one
// consumer and feeds eight matrix instructions.  For keys the wave removes the
// source RoPE (Sec. 3.3) from each fragment in registers, one step ahead of
// its use, between the matrix instructions; nothing is written back to LDS.
// At the end of a tile each wave writes the partial sums of the output
// channels its partner owns to LDS and, at the start of the next tile, adds
// the partner's partial sums of its own channels, then applies the target
// RoPE (keys), rounds to bf16 and stores.  The bias is the initial value of
// the owner's accumulators.
//
// Source rows go from memory straight into LDS (buffer loads with the LDS
// flag), two or more tiles ahead, through a ring of stages; loads into LDS are
// the only loads in flight during the sweep.  One barrier per tile orders the
// partial-sum exchange and the reuse of stages.
//
// LDS: [exchange: 2 tile parities x 4 waves x 4 output blocks x 64 lanes x 16
// bytes] then the stage ring.  A stage holds 2k source slots (slot 2i + s =
// block i of layer s of the pair; a pair with one layer repeats its rows),
// each 16 token rows of 256 bytes with 16-byte chunk q of token r at position
// q ^ (r & M), then (keys) the tile's source (and target) RoPE (cos, sin) fp16
// pairs and (slot-addressed targets) its slot indices.  M is 7 for keys in the
// half-split layout, whose fragments are two 8-byte pieces 128 bytes apart
// (channels j..j+3 and j+64..j+67: both members of four RoPE planes), and 15
// otherwise.
#include "kvx_asm.h"
#include "kvx_bf16.h"
#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int D = 128;
constexpr int MT = 16;                   // tokens per tile
constexpr int NT = 256;                  // threads per workgroup
constexpr int ROWB = D * 2;              // bytes per token row
constexpr int SLOTB = MT * ROWB;         // bytes per source slot
constexpr int CSB = MT * 256;            // coefficient block: 16 tokens x 64 planes x 4 bytes
constexpr int XCH = 2 * 4 * 4 * 64 * 16; // partial-sum exchange
constexpr int LDS_MAX = 160 * 1024;

template <int K, bool SLOTS, bool TGT>
struct GeoKS {
  static constexpr int NSLOT = 2 * K;
  static constexpr int CS_OFF = NSLOT * SLOTB;             // source RoPE (cos, sin)
  static constexpr int CT_OFF = CS_OFF + CSB;              // target RoPE (cos, sin), TGT
  static constexpr int SL_OFF = CS_OFF + (TGT ? 2 : 1) * CSB;   // slot indices, 256 B per wave
  static constexpr int STAGE = SL_OFF + (SLOTS ? 1024 : 0);
  static constexpr int VSL_OFF = NSLOT * SLOTB;
  static constexpr int VSTAGE = VSL_OFF + (SLOTS ? 1024 : 0);
  static constexpr int cap(int n, int m) { return n < m ? n : m; }
  static constexpr int NK = cap((LDS_MAX - XCH) / STAGE, 4);    // stages, key units
  static constexpr int NV = cap((LDS_MAX - XCH) / VSTAGE, 5);   // stages, value units
  static constexpr int LDS = XCH + (NK * STAGE > NV * VSTAGE ? NK * STAGE : NV * VSTAGE);
  static constexpr int ZH = 2 * K;                          // reduction steps per wave
  static constexpr bool fits = NK >= 3 && NV >= 3 && LDS <= LDS_MAX;
};

struct KsCtx {
  int lane, wave, c, row, sl;
  int64_t t_begin, t_end;
  int n_tiles;
};

// One unit (layer group, head, K|V) for wave (sl, KH) of one workgroup.  KV is
// 0 for keys.  TGT: the target RoPE differs from the source RoPE.
template <int K, int STYLE, bool SLOTS, bool TGT, int KV, int KH>
__device__ __forceinline__ void ks_unit(const MapArgs& a, uint32_t lds0, const KsCtx& q, int h,
                                        int ll0, bool has1) {
  using G = GeoKS<K, SLOTS, TGT>;
  constexpr int ZH = G::ZH;
  constexpr int NSLOT = G::NSLOT;
  constexpr bool KEYS = KV == 0;
  constexpr bool SPLIT = KEYS && STYLE == 0;   // fragment: 4 channels + their RoPE partners
  constexpr int RM = SPLIT ? 7 : 15;           // row mask of the chunk swizzle
  constexpr int N_DMA = NSLOT + (KEYS ? 1 : 0) + (KEYS && TGT ? 1 : 0) + (SLOTS ? 1 : 0);
  constexpr int N_VM = N_DMA + 2;
  constexpr int NS = KEYS ? G::NK : G::NV;     // stages of the ring
  constexpr int SB = KEYS ? G::STAGE : G::VSTAGE;
  constexpr int SLOFF = KEYS ? G::SL_OFF : G::VSL_OFF;
  // at the end of tile i tile i+1 must have landed; the loads of tiles
  // i+2 .. i+NS-1 are the only loads into LDS issued after it
  constexpr int WAIT_DMA = (NS - 2) * N_DMA;
  constexpr int Z0 = KH * ZH;                  // this wave's first reduction step
  constexpr int OH = KH;                       // output half owned: channels 32 OH + .. and 64 + 32 OH + ..

  const int c = q.c, row = q.row, sl = q.sl, wave = q.wave;
  const bool mine = sl == 0 || has1;
  const int T = a.T;
  const int64_t t_begin = q.t_begin, t_end = q.t_end;
  const int n_tiles = q.n_tiles;
  const uint32_t plane_bytes = (uint32_t)T * ROWB;
  const uint32_t ring0 = lds0 + XCH;

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

  // ---- this wave's map rows in AGPRs: block b, step Z0 + zz.  Accumulator
  // element i of block b is output channel 32 (b / 2) + 8 c + 4 (b % 2) + i;
  // the wave owns the blocks with (b / 2) % 2 == OH.
  u32x4_t wf[8][ZH];
  f32x4_t bias[4];   // owned blocks 2 OH, 2 OH + 1, 4 + 2 OH, 5 + 2 OH
  {
    const int l = a.l0 + ll0 + (mine ? sl : 0);
    const uint16_t* img = reinterpret_cast<const uint16_t*>(a.wpack) +
                          (((int64_t)l * a.H + h) * 2 + KV) * (int64_t)D * (K * D);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint16_t* r0 = img + (int64_t)(16 * b + row) * (K * D);
#pragma unroll
      for (int zz = 0; zz < ZH; ++zz) {
        if (SPLIT) {
          // the map rows of input features 16 s + 4 c .. + 3 of source u and
          // of their RoPE partners 64 later: halves of chunks q and q + 8
          const int z = Z0 + zz, u = z >> 2, s = z & 3;
          const int q1 = 16 * u + 2 * s + (c >> 1);
          const uint2 lo = *reinterpret_cast<const uint2*>(r0 + 8 * (q1 ^ row) + 4 * (c & 1));
          const uint2 hi = *reinterpret_cast<const uint2*>(r0 + 8 * ((q1 + 8) ^ row) + 4 * (c & 1));
          wf[b][zz] = (u32x4_t){lo.x, lo.y, hi.x, hi.y};
        } else {
          wf[b][zz] = *reinterpret_cast<const u32x4_t*>(r0 + 8 * ((4 * (Z0 + zz) + c) ^ row));
        }
      }
    }
    const uint16_t* bp = reinterpret_cast<const uint16_t*>(KV ? a.bv : a.bk);
    u32x4_t bw[2] = {{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
    if (bp != nullptr) {
#pragma unroll
      for (int x = 0; x < 2; ++x)
        bw[x] = *reinterpret_cast<const u32x4_t*>(bp + ((int64_t)l * a.H + h) * D + 64 * x + 32 * OH + 8 * c);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; i += 2) {
        const uint32_t wd = bw[j >> 1][2 * (j & 1) + i / 2];
        bias[j][i] = lo_bf16(wd);
        bias[j][i + 1] = hi_bf16(wd);
      }
  }
  // The map and bias loads are the compiler's own: wait for them here, with a
  // wait it knows of, so that it inserts none inside the tile loop.
  __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0)

  // ---- per-lane LDS offsets that do not change from tile to tile
  // DMA: wave w loads tokens 4w .. 4w+3 of every slot; lane -> (token tr,
  // position lane & 15), which holds chunk position ^ (tr & RM)
  const int tr = 4 * wave + (q.lane >> 4);
  const uint32_t vo_row = (uint32_t)(tr * ROWB + 16 * ((q.lane & 15) ^ (tr & RM)));
  const uint32_t vo_slot = (uint32_t)(4 * (q.lane & 15));
  // fragment of step s (within a slot) of this lane: half-split keys: channels
  // 16 s + 4 c .. +3 (8 bytes) and their partners 64 later; otherwise the
  // chunk 4 s + c (channels 32 s + 8 c .. +7)
  uint32_t fpos[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    fpos[s] = (uint32_t)(sl * SLOTB + row * ROWB +
                         (SPLIT ? 16 * ((2 * s + (c >> 1)) ^ (row & RM)) + 8 * (c & 1)
                                : 16 * ((4 * s + c) ^ (row & RM))));
  // source RoPE (cos, sin) of the planes of step s: piece 4 s + c of the row
  uint32_t cpos[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) cpos[s] = (uint32_t)(G::CS_OFF + row * 256 + 16 * ((4 * s + c) ^ (row & RM)));
  // epilogue: target RoPE of the owned planes and the output columns
  const int eq0 = STYLE == 0 ? 8 * OH + 2 * c : 4 * OH + c;
  const int eq1 = STYLE == 0 ? 8 * OH + 2 * c + 1 : 8 + 4 * OH + c;
  const uint32_t vct0 = (uint32_t)((TGT ? G::CT_OFF : G::CS_OFF) + row * 256 + 16 * (eq0 ^ (row & RM)));
  const uint32_t vct1 = (uint32_t)((TGT ? G::CT_OFF : G::CS_OFF) + row * 256 + 16 * (eq1 ^ (row & RM)));
  const uint32_t colb = (uint32_t)(2 * (32 * OH + 8 * c));
  // exchange: [parity][writer wave][block j][lane]; a wave writes its
  // partner's four blocks and reads its own from the partner's area
  const uint32_t xw = lds0 + (uint32_t)(wave * 4096 + q.lane * 16);
  const uint32_t xr = lds0 + (uint32_t)((wave ^ 1) * 4096 + q.lane * 16);

  auto stage_base = [&](int st) __attribute__((always_inline)) -> uint32_t {
    return ring0 + (uint32_t)(st * SB);
  };
  // Load m of tile j into stage st.  The tile's row offset goes into the
  // voffset, which the buffer's range check covers (soffset is left out of
  // it): with each range ending at the end of its plane (table, slot array),
  // a tile past the end and the rows of the last tile past T read as zero
  // without touching memory, and nothing of them is stored.
  auto dma_one = [&](int st, int j, int m) __attribute__((always_inline)) {
    const uint32_t row0 = __builtin_amdgcn_readfirstlane((uint32_t)(t_begin + (int64_t)MT * j));
    const uint32_t base = stage_base(st) + (uint32_t)(wave * 1024);
    const uint32_t vo = vo_row + row0 * (uint32_t)ROWB;
    if (m < NSLOT) {
      dma16z(base + m * SLOTB, vo, rs_src[m]);
    } else if (KEYS && m == NSLOT) {
      dma16z(base + G::CS_OFF, vo, rs_cs);
    } else if (KEYS && TGT && m == NSLOT + 1) {
      dma16z(base + G::CT_OFF, vo, rs_ct);
    } else {
      dma4z(stage_base(st) + (uint32_t)(SLOFF + wave * 256), vo_slot + row0 * 4u, rs_slot);
    }
  };
  auto dma_tile = [&](int st, int j) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < N_DMA; ++m) dma_one(st, j, m);
  };

  // ---- accumulators: set P of tile i; the owned blocks of tile i-1 wait in
  // set P ^ 1 for the partner's partial sums
  f32x4_t acc[2][8];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[p][b] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  // ---- epilogue of tile j: owned blocks of set p plus the partner's partial
  // sums (xs), target RoPE (keys), rounding, two 16-byte stores per lane
  u32x4_t ct[2] = {{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
  uint32_t slotv = 0;
  u32x4_t ev[2];
  uint32_t eo = 0;
  auto epilogue = [&](int p, int j, const u32x4_t (&xs)[4]) __attribute__((always_inline)) {
    float y[2][8];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        y[x][i] = acc[p][4 * x + 2 * OH][i] + __uint_as_float(xs[2 * x][i]);
        y[x][4 + i] = acc[p][4 * x + 2 * OH + 1][i] + __uint_as_float(xs[2 * x + 1][i]);
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
    const int64_t tl = t_begin + (int64_t)MT * j + row;
    const int64_t orow = SLOTS ? (int64_t)(int32_t)slotv : tl;
    const bool ok = mine && j >= 0 && tl < t_end && orow >= 0 && orow < a.tgt_rows;
    eo = ok ? (uint32_t)orow * ROWB + colb : 0xffffff00u;
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      ev[x][0] = pack2(y[x][0], y[x][1]);
      ev[x][1] = pack2(y[x][2], y[x][3]);
      ev[x][2] = pack2(y[x][4], y[x][5]);
      ev[x][3] = pack2(y[x][6], y[x][7]);
    }
  };
  auto epilogue_store = [&](int x) __attribute__((always_inline)) {
    if (x == 0) vstore16<0>(ev[0], eo, rs_out);
    else vstore16<128>(ev[1], eo, rs_out);
  };
  // partner's partial sums of the owned blocks of the tile of parity p
  auto exchange_read = [&](int p, u32x4_t (&xs)[4]) __attribute__((always_inline)) {
    const uint32_t base = xr + (uint32_t)(p * 16384);
    lds_read<0>(xs[0], base);
    lds_read<1024>(xs[1], base);
    lds_read<2048>(xs[2], base);
    lds_read<3072>(xs[3], base);
  };
  // this wave's partial sums of the partner's blocks (set p)
  auto exchange_write = [&](int p) __attribute__((always_inline)) {
    constexpr int PB = 2 * (1 - OH);   // partner's first owned block
    const uint32_t base = xw + (uint32_t)(p * 16384);
    lds_write<0>(base, __builtin_bit_cast(u32x4_t, acc[p][PB]));
    lds_write<1024>(base, __builtin_bit_cast(u32x4_t, acc[p][PB + 1]));
    lds_write<2048>(base, __builtin_bit_cast(u32x4_t, acc[p][PB + 4]));
    lds_write<3072>(base, __builtin_bit_cast(u32x4_t, acc[p][PB + 5]));
  };
  // epilogue inputs of the tile in stage st: target coefficients, slot
  auto epilogue_reads = [&](int st) __attribute__((always_inline)) {
    const uint32_t base = stage_base(st);
    if (KEYS) {
      lds_read<0>(ct[0], base + vct0);
      lds_read<0>(ct[1], base + vct1);
    }
    if (SLOTS) lds_read_b32(slotv, base + (uint32_t)(SLOFF + row * 4));
  };

  // ---- operand fragments: a ring of three (step zz uses fr[zz % 3], the
  // next is stripped meanwhile, the one after is being read)
  u32x4_t fr[3];
  u32x4_t cs[4];
  auto frag_read = [&](uint32_t sbase, int zz) __attribute__((always_inline)) {
    const int z = Z0 + zz;
    const uint32_t addr = sbase + fpos[z % 4];
    u32x4_t& d = fr[zz % 3];
    if (SPLIT) {
      switch (z / 4) {   // slot 2 (z / 4) + sl; x and y pieces 128 bytes apart
        case 0: lds_read2_b64<0, 16>(d, addr); break;
        case 1: lds_read2_b64<0, 16>(d, addr + 2 * SLOTB); break;
        case 2: lds_read2_b64<0, 16>(d, addr + 4 * SLOTB); break;
        default: lds_read2_b64<0, 16>(d, addr + 6 * SLOTB); break;
      }
    } else {
      switch (z / 4) {
        case 0: lds_read<0>(d, addr); break;
        case 1: lds_read<2 * SLOTB>(d, addr); break;
        case 2: lds_read<4 * SLOTB>(d, addr); break;
        default: lds_read<6 * SLOTB>(d, addr); break;
      }
    }
  };
  // strip the source RoPE from fragment zz, part pt of 8 (one after each
  // matrix instruction)
  float su[2], sv[2];
  auto strip_part = [&](int zz, int pt) __attribute__((always_inline)) {
    u32x4_t& f = fr[zz % 3];
    const u32x4_t& cf = cs[(Z0 + zz) % 4];
    if (SPLIT) {
      // words: (x0, x1), (x2, x3), (y0, y1), (y2, y3); plane e = (x_e, y_e)
      const int hw = pt < 4 ? 0 : 1;     // words hw and 2 + hw
      const int ph = pt & 3;
      if (ph == 0) {
        uint32_t xa = f[hw], ya = f[2 + hw];
        pin(xa, ya);
        su[0] = lo_bf16(xa);
        su[1] = hi_bf16(xa);
        sv[0] = lo_bf16(ya);
        sv[1] = hi_bf16(ya);
        pin(su[0], su[1], sv[0], sv[1]);
      } else if (ph == 1) {
        strip(su[0], sv[0], cf[2 * hw]);
        pin(su[0], su[1], sv[0], sv[1]);
      } else if (ph == 2) {
        strip(su[1], sv[1], cf[2 * hw + 1]);
        pin(su[0], su[1], sv[0], sv[1]);
      } else {
        uint32_t xa = pack2(su[0], su[1]), ya = pack2(sv[0], sv[1]);
        pin(xa, ya);
        f[hw] = xa;
        f[2 + hw] = ya;
      }
    } else {
      // words: (x, y) of planes 0..3
      const int e = pt >> 1;
      if ((pt & 1) == 0) {
        uint32_t wa = f[e];
        pin(wa);
        su[0] = lo_bf16(wa);
        sv[0] = hi_bf16(wa);
        strip(su[0], sv[0], cf[e]);
        pin(su[0], sv[0]);
      } else {
        uint32_t wa = pack2(su[0], sv[0]);
        pin(wa);
        f[e] = wa;
      }
    }
  };

  // ---- pipeline prologue: tiles 0 .. NS-2 in flight
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) dma_tile(j, j);
  vm_wait<WAIT_DMA>();                         // tile 0 is in LDS
  __syncthreads();

  // ---- tile i in stage st with accumulator set P = i % 2.  On entry (after a
  // barrier): stage st holds tile i, the exchange area of parity P ^ 1 holds
  // the partner's partial sums of tile i-1, ct / slotv hold its epilogue
  // inputs.
  auto tile = [&](auto pc, int i, int st) __attribute__((always_inline)) {
    constexpr int P = decltype(pc)::value;
    const int stf = st == 0 ? NS - 1 : st - 1;    // the stage tile i-1 used: free now
    const uint32_t sbase = stage_base(st);
    // LDS: partner sums (4), [keys: coefficients (4)], fragments 0 and 1
    u32x4_t xs[4];
    exchange_read(P ^ 1, xs);
    if (KEYS) {
#pragma unroll
      for (int s = 0; s < 4; ++s) lds_read<0>(cs[s], sbase + cpos[s]);
    }
    frag_read(sbase, 0);
    if (ZH > 1) frag_read(sbase, 1);
    constexpr int AFTER_X = (KEYS ? 4 : 0) + (ZH > 1 ? 2 : 1);
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(xs[0]), "+v"(xs[1]), "+v"(xs[2]), "+v"(xs[3]) : "n"(AFTER_X));
    epilogue(P ^ 1, i - 1, xs);
    if (KEYS) {
      // coefficients and fragment 0 arrived: strip fragment 0
      if (ZH > 1) {
        asm volatile("s_waitcnt lgkmcnt(1)" : "+v"(fr[0]), "+v"(cs[0]), "+v"(cs[1]), "+v"(cs[2]));
      } else {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fr[0]), "+v"(cs[0]), "+v"(cs[1]), "+v"(cs[2]));
      }
      pin(cs[3]);
#pragma unroll
      for (int pt = 0; pt < 8; ++pt) strip_part(0, pt);
    }

    // contraction: step zz multiplies fragment zz with the 8 map blocks; for
    // keys fragment zz + 1 is stripped between the matrix instructions
#pragma unroll
    for (int zz = 0; zz < ZH; ++zz) {
      if (KEYS || zz + 1 >= ZH) {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fr[0]), "+v"(fr[1]), "+v"(fr[2]));
      } else {
        asm volatile("s_waitcnt lgkmcnt(1)" : "+v"(fr[zz % 3]));
      }
      if (zz + 2 < ZH) frag_read(sbase, zz + 2);
      const u32x4_t x = fr[zz % 3];
      // a matrix instruction reading a register that a vector instruction
      // wrote (the strip) needs two wait states in between
      if (KEYS) asm volatile("s_nop 1");
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        if (zz == 0) {
          if (((b >> 1) & 1) == OH) mfma_init(acc[P][b], wf[b][zz], x, bias[(b >> 2) * 2 + (b & 1)]);
          else mfma_zero(acc[P][b], wf[b][zz], x);
        } else {
          mfma_acc(acc[P][b], wf[b][zz], x);
        }
        if (KEYS && zz + 1 < ZH) strip_part(zz + 1, b);
      }
#pragma unroll
      for (int m = 0; m < N_VM; ++m)
        if (m * ZH / N_VM == zz) {
          if (m < N_DMA) dma_one(stf, i + NS - 1, m);
          else epilogue_store(m - N_DMA);
        }
    }
    // the partial sums of the partner's blocks, after the matrix results land
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc[P][0]), "+v"(acc[P][1]), "+v"(acc[P][2]),
                 "+v"(acc[P][3]));
    asm volatile("" : "+v"(acc[P][4]), "+v"(acc[P][5]), "+v"(acc[P][6]), "+v"(acc[P][7]));
    exchange_write(P);
    epilogue_reads(st);
    // tile i+1 is in LDS: loads into LDS retire in order among themselves
    vm_wait<WAIT_DMA>();
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(ct[0]), "+v"(ct[1]), "+v"(slotv));
    __syncthreads();
  };
  auto final_epilogue = [&](int p, int j) __attribute__((always_inline)) {
    u32x4_t xs[4];
    exchange_read(p, xs);
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xs[0]), "+v"(xs[1]), "+v"(xs[2]), "+v"(xs[3]));
    epilogue(p, j, xs);
    epilogue_store(0);
    epilogue_store(1);
  };

  // Two tiles per trip, so that the accumulator sets are constants.
  int st = 0;
  for (int i0 = 0; i0 < n_tiles; i0 += 2) {
    tile(std::integral_constant<int, 0>{}, i0, st);
    st = st + 1 == NS ? 0 : st + 1;
    if (i0 + 1 >= n_tiles) { final_epilogue(0, i0); break; }
    tile(std::integral_constant<int, 1>{}, i0 + 1, st);
    st = st + 1 == NS ? 0 : st + 1;
    if (i0 + 2 >= n_tiles) { final_epilogue(1, i0 + 1); break; }
  }
  // everything this unit issued has landed, and every wave is done with the
  // exchange area, before the next unit reuses LDS
  vm_wait<0>();
  __syncthreads();
}

template <int K, int STYLE, bool SLOTS, bool TGT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void map_ks_kernel(const MapArgs a, const SweepPlan p) {
  __shared__ __attribute__((aligned(256))) char smem[GeoKS<K, SLOTS, TGT>::LDS];
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_u32(smem));

  KsCtx q;
  q.lane = threadIdx.x & 63;
  q.wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  q.c = q.lane >> 4;        // reduction chunk of an MFMA fragment
  q.row = q.lane & 15;      // token (B, D) or map row (A) within a block
  q.sl = q.wave >> 1;       // layer slot of the pair
  const int kh = q.wave & 1;   // half of the reduction

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
    if (kv == 0) {
      if (kh == 0) ks_unit<K, STYLE, SLOTS, TGT, 0, 0>(a, lds0, q, h, ll0, has1);
      else ks_unit<K, STYLE, SLOTS, TGT, 0, 1>(a, lds0, q, h, ll0, has1);
    } else {
      if (kh == 0) ks_unit<K, STYLE, SLOTS, TGT, 1, 0>(a, lds0, q, h, ll0, has1);
      else ks_unit<K, STYLE, SLOTS, TGT, 1, 1>(a, lds0, q, h, ll0, has1);
    }
  }
}

template <int K, int STYLE, bool SLOTS, bool TGT>
hipError_t launch_ksk(const MapArgs& a, const SweepPlan& p, hipStream_t stream) {
  if constexpr (GeoKS<K, SLOTS, TGT>::fits) {
    hipLaunchKernelGGL((map_ks_kernel<K, STYLE, SLOTS, TGT>), dim3(256), dim3(NT), 0, stream, a, p);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <int K, int STYLE>
hipError_t launch_ksslots(const MapArgs& a, const SweepPlan& p, hipStream_t stream) {
  const bool slots = a.slots != nullptr, tgt = a.cs16_tgt != a.cs16;
  if (slots)
    return tgt ? launch_ksk<K, STYLE, true, true>(a, p, stream) : launch_ksk<K, STYLE, true, false>(a, p, stream);
  return tgt ? launch_ksk<K, STYLE, false, true>(a, p, stream) : launch_ksk<K, STYLE, false, false>(a, p, stream);
}

template <int K>
hipError_t launch_ksstyle(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  return style == 0 ? launch_ksslots<K, 0>(a, p, stream) : launch_ksslots<K, 1>(a, p, stream);
}

}  // namespace

bool map_ks_supported(int k, int64_t T, int64_t tgt_rows, bool slots, bool tgt_rope) {
  // byte offsets within a plane, and of the tiles loaded ahead past its end,
  // must fit the 32-bit buffer offsets; the stages must fit the LDS
  if (T < 1 || (T + 80) * ROWB >= 0xffffff00LL || tgt_rows * ROWB >= 0xffffff00LL) return false;
  switch (k) {
    case 1: return slots ? (tgt_rope ? GeoKS<1, true, true>::fits : GeoKS<1, true, false>::fits)
                         : (tgt_rope ? GeoKS<1, false, true>::fits : GeoKS<1, false, false>::fits);
    case 2: return slots ? (tgt_rope ? GeoKS<2, true, true>::fits : GeoKS<2, true, false>::fits)
                         : (tgt_rope ? GeoKS<2, false, true>::fits : GeoKS<2, false, false>::fits);
    case 3: return slots ? (tgt_rope ? GeoKS<3, true, true>::fits : GeoKS<3, true, false>::fits)
                         : (tgt_rope ? GeoKS<3, false, true>::fits : GeoKS<3, false, false>::fits);
    case 4: return slots ? (tgt_rope ? GeoKS<4, true, true>::fits : GeoKS<4, true, false>::fits)
                         : (tgt_rope ? GeoKS<4, false, true>::fits : GeoKS<4, false, false>::fits);
    default: return false;
  }
}

hipError_t launch_map_ks(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream) {
  if (a.T == 0 || a.nl == 0) return hipSuccess;
  switch (a.k) {
    case 1: return launch_ksstyle<1>(a, p, style, stream);
    case 2: return launch_ksstyle<2>(a, p, style, stream);
    case 3: return launch_ksstyle<3>(a, p, style, stream);
    case 4: return launch_ksstyle<4>(a, p, style, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kvx
