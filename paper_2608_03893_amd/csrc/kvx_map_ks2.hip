// K-split layer-sweep map kernel with a mid-tile barrier, for bf16 caches
// with head dimension 128 and k = 2 or 4.
//
// Work decomposition across the chip and within a workgroup are those of the
// k-split kernel: one workgroup per CU, 4 waves (one per SIMD), a unit is
// (layer group, head, K|V), CU slot j of an XCD owns a pair of target layers
// and a token part; wave (s, h) holds in AGPRs the map rows of reduction
// steps h * 2k .. h * 2k + 2k - 1 of layer s of the pair (Eq. ridge_kv), for
// all 128 output channels, and the two waves of a layer add their partial
// sums through LDS.  What changes is the schedule inside a tile, which here
// keeps the matrix pipe busy across tile boundaries:
//
//  * With k even the reduction half of a wave is k / 2 whole source layers,
//    and each wave loads (buffer loads straight into LDS) those: 4 token rows
//    of 256 contiguous bytes per load.  A source that both layers of the pair
//    list is loaded once, by the first layer's wave; the second layer's wave
//    reads that slot and issues null loads (an empty buffer range) in its
//    place, so the wait counts stay those of the schedule.  The host pairs
//    the target layers of a group so that as many pairs as possible share a
//    source.  The loads of a tile land before the mid-tile barrier of the
//    tile before it, and a barrier at the start of each tile keeps the loads
//    into a stage behind every wave's last read of it.
//  * The one barrier per tile sits in the middle of the tile, between two
//    matrix instructions.  Before it a wave has written the partial sums of
//    the previous tile that its partner owns and checked that the
//    coefficients of the next tile have landed; after it the wave reads its
//    partner's sums of the previous tile, finishes that tile (sum, target
//    RoPE for keys, bf16 rounding) between the matrix instructions of the
//    later steps and stores it.
//  * Fragment reads run two steps ahead, across tile boundaries; for keys the
//    source RoPE of the next fragment is removed between the matrix
//    instructions of the current step.
//  * Loads of tile i + NS - 1 go out in the first half of tile i, stores in
//    the second half, one memory instruction between two matrix instructions.
//    Each load carries its tile's row offset in the range-checked voffset,
//    so tiles past the end (and the rows of the last tile past T) read zeros
//    without touching memory.
//
// Every LDS and memory instruction comes from inline assembly at a fixed
// place in the tile, so the waits are computed at compile time from that
// schedule (struct Ks2Sched).
//
// LDS: [exchange: 2 tile parities x 4 waves x 4 output blocks x 64 lanes x 16
// bytes] then the stage ring.  A stage holds each wave's source slots (wave
// w, slot u at (2 w k + 4 u) KB: 16 token rows of 256 bytes, 16-byte chunk q
// of token r at position q ^ (r & M)), then (keys) the tile's source (and
// target) RoPE (cos, sin) fp16 pairs, 16 token rows of 256 bytes with piece q
// of token r at position q ^ r, and (slot-addressed targets) each wave's copy
// of the tile's slot indices.  M is 7 for keys in the half-split layout, whose
// fragments are two 8-byte pieces 128 bytes apart (channels j..j+3 and
// j+64..j+67: both members of four RoPE planes), and 15 otherwise.
#include <type_traits>

#include "kvx_asm.h"
#include "kvx_bf16.h"
#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int D = 128;
constexpr int MT = 16;                   // tokens per tile
constexpr int NT = 256;                  // threads per workgroup
constexpr int ROWB = D * 2;              // bytes per token row
constexpr int STEPB = 1024;              // one reduction step of one wave
constexpr int CSB = MT * 256;            // coefficient block: 16 tokens x 64 planes x 4 bytes
constexpr int XCH = 2 * 4 * 4 * 64 * 16; // partial-sum exchange
constexpr int LDS_MAX = 160 * 1024;

template <int K, bool SLOTS, bool TGT>
struct GeoK2 {
  static constexpr int ZH = 2 * K;                          // reduction steps per wave
  static constexpr int OWN = 4 * ZH * STEPB;                // the four waves' source slots
  static constexpr int CS_OFF = OWN;                        // source RoPE (cos, sin)
  static constexpr int CT_OFF = OWN + CSB;                  // target RoPE, TGT
  static constexpr int SL_OFF = OWN + (TGT ? 2 : 1) * CSB;  // slot indices, 256 B per wave
  static constexpr int KSTAGE = SL_OFF + (SLOTS ? 1024 : 0);
  static constexpr int VSL_OFF = OWN;
  static constexpr int VSTAGE = OWN + (SLOTS ? 1024 : 0);
  static constexpr int cap(int n, int m) { return n < m ? n : m; }
  static constexpr int NK = cap((LDS_MAX - XCH) / KSTAGE, 4);   // stages, key units
  static constexpr int NV = cap((LDS_MAX - XCH) / VSTAGE, 5);   // stages, value units
  static constexpr int LDS = XCH + (NK * KSTAGE > NV * VSTAGE ? NK * KSTAGE : NV * VSTAGE);
  static constexpr bool fits = (K == 2 || K == 4) && NK >= 3 && NV >= 3 && LDS <= LDS_MAX;
};

// The fixed schedule of one tile and the wait counts it implies.  Every
// operation has a place (step, j, o): after the j-th matrix instruction of
// the step, in the order o.  At most one LDS operation and one memory
// instruction follow a matrix instruction (spread over the tile).
//   o 1  [mid step MB, j 0] wait for loads and LDS, barrier
//     2  [j 0] fragment read, two steps ahead
//     3  [MB, j 1..4] reads of the partner's partial sums of tile i-1
//     4  [step 0, j 1..4] writes of the partial sums of tile i-1 that the
//        partner owns; [j 5, 6] reads of the target coefficients (keys) and
//        [j 7] of the slot indices (slots) that finish tile i-1
//     5..8  coefficient reads for the next tile (keys), from j 5 on
//     7  [j 0] wait before the step's vector work (strip, epilogue)
//     8  the stores of tile i-1 [step ZH - 1]
//     9  loads: source rows of tile i+NS-1 [steps < MB, j 3 and 6],
//        coefficients and slot indices [MB, j 5..7]
// LDS operations complete in order; loads into LDS complete in order among
// themselves, and the waits for them do not count stores.
template <int ZH, int Z0, bool KEYS, bool SLOTS, bool TGT>
struct Ks2Sched {
  static_assert(ZH == 4 || ZH == 8, "k = 2 or 4");
  static constexpr int MB = ZH / 2;
  static constexpr int EPI = ZH == 8 ? 5 : 3;   // step that finishes tile i-1
  static constexpr int ST = ZH - 1;             // step of its stores
  static constexpr int S0J = ZH == 8 ? 1 : 7;   // matrix instruction before each store
  static constexpr int S1J = ZH == 8 ? 4 : 7;
  static constexpr int NC = (KEYS ? 1 : 0) + (KEYS && TGT ? 1 : 0) + (SLOTS ? 1 : 0);
  static constexpr int NL = ZH + NC;                           // loads per tile
  static constexpr int key(int step, int j, int o) { return step * 100 + j * 10 + o; }
  static constexpr int sof(int f) { return (Z0 + f) % 4; }     // channel quarter of fragment f
  static constexpr bool cs_used(int s) {
    if (!KEYS) return false;
    for (int f = 0; f < ZH; ++f)
      if (sof(f) == s) return true;
    return false;
  }
  // Fragment f is stripped in step f - 1 (fragment 0 in the last step of the
  // tile before), so the coefficients of quarter s for the next tile can be
  // read once the last strip of this tile that uses them is done, and after
  // the barrier that makes them visible.
  static constexpr int cs_step(int s) {
    int r = -1;
    for (int f = 1; f < ZH; ++f)
      if (sof(f) == s) r = f - 1;
    return r + 1 > MB ? r + 1 : MB;
  }
  static constexpr int cs_rank(int s) {
    int n = 0;
    for (int t = 0; t < s; ++t)
      if (cs_used(t) && cs_step(t) == cs_step(s)) ++n;
    return n;
  }
  static constexpr int cs_j(int s) { return cs_rank(s) < 3 ? 5 + cs_rank(s) : 7; }
  static constexpr int cs_key(int s) { return key(cs_step(s), cs_j(s), 5 + cs_rank(s)); }
  static constexpr int fr_key(int z) { return key(z, 0, 2); }
  static constexpr int xr_key(int k) { return key(MB, 1 + k, 3); }
  static constexpr int xw_key(int k) { return key(0, 1 + k, 4); }            // k < 4
  static constexpr int ct_key(int k) { return key(0, 5 + k, 4); }            // keys
  static constexpr int sl_key() { return key(0, 7, 4); }                     // slots
  // LDS operations of one tile placed before key kk
  static constexpr int ops_before(int kk) {
    int n = 0;
    for (int z = 0; z < ZH; ++z) n += fr_key(z) < kk;
    for (int k = 0; k < 4; ++k) n += (xr_key(k) < kk) + (xw_key(k) < kk);
    if (KEYS)
      for (int k = 0; k < 2; ++k) n += ct_key(k) < kk;
    if (SLOTS) n += sl_key() < kk;
    for (int s = 0; s < 4; ++s) n += cs_used(s) && cs_key(s) < kk;
    return n;
  }
  static constexpr int NOPS = ops_before(100 * ZH);
  // at most this many LDS operations outstanding at key w: the operation at
  // key x of this tile (dt = 0) or of the tile before (dt = -1) has completed
  static constexpr int need(int x, int dt, int w) { return ops_before(w) - (dt * NOPS + ops_before(x)) - 1; }
  static constexpr int mn(int a, int b) { return a < b ? a : b; }
  // values: before the first matrix instruction of step zz, fragment zz
  // (read in step zz - 2)
  static constexpr int v_wait(int zz) {
    return zz >= 2 ? need(fr_key(zz - 2), 0, key(zz, 0, 0)) : need(fr_key(zz - 2 + ZH), -1, key(zz, 0, 0));
  }
  // keys: before the strip of fragment zz + 1 in step zz, that fragment (read
  // in step zz - 1) and its coefficients; in step EPI also the partner's sums
  static constexpr int k_wait(int zz) {
    const int w = key(zz, 0, 7);
    const int a = zz >= 1 ? need(fr_key(zz - 1), 0, w) : need(fr_key(ZH - 1), -1, w);
    const int f = zz + 1;
    const int b = f < ZH ? need(cs_key(sof(f)), -1, w) : need(cs_key(sof(0)), 0, w);
    const int r = mn(a, b);
    return zz == EPI ? mn(r, need(xr_key(3), 0, w)) : r;
  }
  // values, step EPI: the partner's sums
  static constexpr int e_wait() { return need(xr_key(3), 0, key(EPI, 0, 7)); }
  // before the barrier: the writes of step 0 and the epilogue input reads
  static constexpr int bar_wait() {
    const int x = SLOTS ? sl_key() : KEYS ? ct_key(1) : xw_key(3);
    return need(x, 0, key(MB, 0, 1));
  }

  // loads
  static constexpr int own_key(int m) { return key(m / 2, (m & 1) ? 6 : 3, 9); }
  static constexpr int c_key(int c) { return key(MB, 5 + c, 9); }
  static constexpr int loads_before(int kk) {
    int n = 0;
    for (int m = 0; m < ZH; ++m) n += own_key(m) < kk;
    for (int c = 0; c < NC; ++c) n += c_key(c) < kk;
    return n;
  }
  // at the barrier: the last load of tile i + 1 (issued during tile i + 2 - NS)
  static constexpr int vm_mid(int NS) { return loads_before(key(MB, 0, 1)) + (NS - 3) * NL; }

  static constexpr bool valid() {
    for (int z = 0; z < ZH; ++z) {
      if (KEYS && k_wait(z) < 0) return false;
      if (!KEYS && v_wait(z) < 0) return false;
    }
    if (KEYS)
      for (int s = 0; s < 4; ++s)
        if (cs_used(s) && (cs_step(s) >= ZH || cs_rank(s) > 3)) return false;
    // the loads of tile i + 1 are all issued before the barrier's wait, in
    // the tile that issues them
    if (loads_before(key(MB, 0, 1)) != ZH) return false;
    return e_wait() >= 0 && bar_wait() >= 0 && EPI > MB && (EPI < ST || ZH == 4);
  }
};

// Block of the j-th matrix instruction of a step for the wave that owns
// output half oh: the partner's four blocks first, so that their sums are
// final early in the next tile.
constexpr int ks2_block(int j, int oh) {
  return (j < 4 ? 2 * (1 - oh) : 2 * oh) + (j & 1) + 4 * ((j & 3) >> 1);
}

struct Ks2Ctx {
  int lane, wave, c, row, sl;
  int64_t t_begin, t_end;
  int n_tiles;
};

template <int N>
__device__ __forceinline__ void vm_wait_c() { asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N < 63 ? N : 63) : "memory"); }
template <int N>
__device__ __forceinline__ void lgk_wait_c() { asm volatile("s_waitcnt lgkmcnt(%0)" : : "n"(N < 15 ? N : 15) : "memory"); }

template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// One unit (layer group, head, K|V) for wave (sl, KH).  KV is 0 for keys.
// TGT: the target RoPE differs from the source RoPE.
template <int K, int STYLE, bool SLOTS, bool TGT, int KV, int KH>
__device__ __forceinline__ void ks2_unit(const MapArgs& a, uint32_t lds0, const Ks2Ctx& q, int h,
                                         int l_a, int l_b, bool has1) {
  using G = GeoK2<K, SLOTS, TGT>;
  constexpr int ZH = G::ZH;
  constexpr bool KEYS = KV == 0;
  constexpr bool SPLIT = KEYS && STYLE == 0;   // fragment: 4 channels + their RoPE partners
  constexpr int RM = SPLIT ? 7 : 15;           // row mask of the chunk swizzle
  constexpr int Z0 = KH * ZH;                  // this wave's first reduction step
  constexpr int OH = KH;                       // output half owned: channels 32 OH + .. and 64 + 32 OH + ..
  using S = Ks2Sched<ZH, Z0, KEYS, SLOTS, TGT>;
  static_assert(S::valid(), "tile schedule");
  constexpr int MB = S::MB;
  constexpr int EPI = S::EPI;
  constexpr int NS = KEYS ? G::NK : G::NV;     // stages of the ring
  constexpr int SB = KEYS ? G::KSTAGE : G::VSTAGE;
  constexpr int SLOFF = KEYS ? G::SL_OFF : G::VSL_OFF;
  constexpr int U0 = Z0 / 4;                   // first source of this wave
  static_assert(Z0 % 4 == 0, "a wave's reduction half is whole source layers");
  constexpr int PB = 2 * (1 - OH);

  // The per-lane offsets below are rebuilt in every unit from an opaque copy
  // of the lane index, so that the compiler does not hoist those of all four
  // unit kinds out of the unit loop and keep them live together.
  int lane = q.lane;
  asm volatile("" : "+v"(lane));
  const int c = lane >> 4, row = lane & 15;
  const int sl = q.sl, wave = q.wave;
  const bool mine = sl == 0 || has1;
  const int lw = mine ? (sl == 0 ? l_a : l_b) : l_a;   // a pair with one layer computes it twice
  const int T = a.T;
  const int64_t t_begin = q.t_begin, t_end = q.t_end;
  const int n_tiles = q.n_tiles;
  const uint32_t plane_bytes = (uint32_t)T * ROWB;
  const uint32_t ring0 = lds0 + XCH;

  // ---- the stage offsets of this wave's source slots.  A source of the
  // pair's second layer that the first layer also lists is read from the
  // first layer's slot; its own loads are null (an empty buffer range: they
  // write zeros to the unused slot without touching memory).
  uint32_t sbase[2];
  bool dup[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    sbase[u] = (uint32_t)((wave * ZH + 4 * u) * STEPB);
    dup[u] = false;
    if (sl == 1 && has1 && U0 + u < K) {
      const int s_u = a.idx[l_b * K + U0 + u];
      for (int r = 0; r < K; ++r)
        if (!dup[u] && a.idx[l_a * K + r] == s_u) {
          sbase[u] = (uint32_t)(((r / (K / 2)) * ZH + 4 * (r % (K / 2))) * STEPB);
          dup[u] = true;
        }
    }
  }
  // ---- buffers: the (one or two) source planes of this wave, the RoPE
  // tables, the slot indices, the target plane
  i32x4_t rs_own[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int uu = U0 + u < K ? U0 + u : K - 1;
    const int sidx = a.idx[lw * K + uu];
    rs_own[u] = make_rsrc(static_cast<const char*>(a.src) +
                              (((int64_t)sidx * 2 + KV) * a.H + h) * (int64_t)plane_bytes,
                          dup[u] ? 0u : plane_bytes);
  }
  const i32x4_t rs_cs = make_rsrc(a.cs16, plane_bytes);
  const i32x4_t rs_ct = make_rsrc(a.cs16_tgt, plane_bytes);
  const i32x4_t rs_slot = make_rsrc(a.slots, (uint32_t)T * 4u);
  const uint32_t out_bytes = (uint32_t)a.tgt_rows * ROWB;
  const i32x4_t rs_out = make_rsrc(static_cast<char*>(a.tgt) +
                                       (((int64_t)(a.l0 + lw) * 2 + KV) * a.H + h) *
                                           (int64_t)out_bytes,
                                   out_bytes);

  // ---- this wave's map rows in AGPRs: block b, step Z0 + zz.  Accumulator
  // element i of block b is output channel 32 (b / 2) + 8 c + 4 (b % 2) + i;
  // the wave owns the blocks with (b / 2) % 2 == OH.
  u32x4_t wf[8][ZH];
  f32x4_t bias[4];   // owned blocks 2 OH, 2 OH + 1, 4 + 2 OH, 5 + 2 OH
  {
    const int l = a.l0 + lw;
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

  // ---- per-lane offsets that do not change from tile to tile
  // source row loads: load g of a slot fetches tokens 4 g .. 4 g + 3; lane ->
  // (token tk, position lane & 15, which holds chunk position ^ (tk & RM))
  uint32_t vo_row[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int tk = 4 * g + (lane >> 4);
    vo_row[g] = (uint32_t)(tk * ROWB + 16 * ((lane & 15) ^ (tk & RM)));
  }
  // fragment of quarter s of a slot for lane (c, row): half-split keys:
  // channels 16 s + 4 c .. + 3 (8 bytes) and their partners 64 later;
  // otherwise chunk 4 s + c (channels 32 s + 8 c .. + 7)
  const uint32_t wbase = (uint32_t)(wave * ZH * STEPB);
  constexpr int NSLOT = ZH / 4;                // source slots of a wave
  uint32_t fpos[NSLOT][4];
#pragma unroll
  for (int u = 0; u < NSLOT; ++u)
#pragma unroll
    for (int s = 0; s < 4; ++s)
      fpos[u][s] = sbase[u] + (uint32_t)(row * ROWB +
                                         (SPLIT ? 16 * ((2 * s + (c >> 1)) ^ (row & RM)) + 8 * (c & 1)
                                                : 16 * ((4 * s + c) ^ (row & RM))));
  // coefficient loads: wave w fetches tokens 4 w .. 4 w + 3; lane -> (token
  // tr, position lane & 15, which holds piece position ^ tr)
  const int tr = 4 * wave + (lane >> 4);
  const uint32_t vo_cs = (uint32_t)(tr * ROWB + 16 * ((lane & 15) ^ tr));
  const uint32_t vo_slot = (uint32_t)(4 * (lane & 15));
  // source RoPE (cos, sin) of the planes of quarter s: piece 4 s + c of the row
  uint32_t cpos[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) cpos[s] = (uint32_t)(G::CS_OFF + row * 256 + 16 * ((4 * s + c) ^ row));
  // epilogue: target RoPE of the owned planes and the output columns
  const int eq0 = STYLE == 0 ? 8 * OH + 2 * c : 4 * OH + c;
  const int eq1 = STYLE == 0 ? 8 * OH + 2 * c + 1 : 8 + 4 * OH + c;
  const uint32_t vct0 = (uint32_t)((TGT ? G::CT_OFF : G::CS_OFF) + row * 256 + 16 * (eq0 ^ row));
  const uint32_t vct1 = (uint32_t)((TGT ? G::CT_OFF : G::CS_OFF) + row * 256 + 16 * (eq1 ^ row));
  // stores: lane (c, row) writes channels 32 OH + 8 c .. + 7 of each output
  // half of token row, 16 bytes
  const uint32_t colb = (uint32_t)(2 * (32 * OH + 8 * c));
  const uint32_t t_begin32 = (uint32_t)t_begin, t_end32 = (uint32_t)t_end;
  const uint32_t rows32 = (uint32_t)a.tgt_rows;
  // exchange: [parity][writer wave][block j][lane]; a wave writes its
  // partner's four blocks and reads its own from the partner's area
  const uint32_t xw = lds0 + (uint32_t)(wave * 4096 + lane * 16);
  const uint32_t xr = lds0 + (uint32_t)((wave ^ 1) * 4096 + lane * 16);

  auto stage_base = [&](int st) __attribute__((always_inline)) -> uint32_t {
    return ring0 + (uint32_t)(st * SB);
  };
  // Row offsets of tile j, carried in the loads' voffsets: the range check
  // of a buffer covers voffset (not soffset), so with each buffer's range
  // ending at the end of its plane (table, slot array), a tile past the end
  // and the rows of the last tile past T read as zero without touching
  // memory; nothing of them is stored.  TileVo holds the voffsets of a tile.
  struct TileVo {
    uint32_t row[4], cs, sl;
  };
  auto tile_vo = [&](int j) __attribute__((always_inline)) -> TileVo {
    const uint32_t row0 = __builtin_amdgcn_readfirstlane((uint32_t)(t_begin + (int64_t)MT * j));
    TileVo v;
#pragma unroll
    for (int g = 0; g < 4; ++g) v.row[g] = vo_row[g] + row0 * (uint32_t)ROWB;
    v.cs = vo_cs + row0 * (uint32_t)ROWB;
    v.sl = vo_slot + row0 * 4u;
    return v;
  };
  // Loads of a tile into stage base sb with its voffsets tv.
  // load m: slot m / 4 of this wave, tokens 4 (m % 4) .. + 3.  NEAR: no
  // vector write of an SGPR the load reads within five wait states.
  auto own_load = [&](uint32_t sb, const TileVo& tv, int m, auto near) __attribute__((always_inline)) {
    if constexpr (decltype(near)::value) dma16z_near(sb + wbase + (uint32_t)(m * STEPB), tv.row[m & 3], rs_own[m >> 2]);
    else dma16z(sb + wbase + (uint32_t)(m * STEPB), tv.row[m & 3], rs_own[m >> 2]);
  };
  // coefficient and slot load n of a tile: source coefficients (keys),
  // target coefficients (keys, TGT), slot indices (slots)
  auto c_load = [&](uint32_t sb, const TileVo& tv, int n, auto near) __attribute__((always_inline)) {
    const int kind = KEYS ? (n == 0 ? 0 : (TGT && n == 1) ? 1 : 2) : 2;
    if constexpr (decltype(near)::value) {
      if (kind == 0) dma16z_near(sb + (uint32_t)(G::CS_OFF + wave * 1024), tv.cs, rs_cs);
      else if (kind == 1) dma16z_near(sb + (uint32_t)(G::CT_OFF + wave * 1024), tv.cs, rs_ct);
      else dma4z_near(sb + (uint32_t)(SLOFF + wave * 256), tv.sl, rs_slot);
    } else {
      if (kind == 0) dma16z(sb + (uint32_t)(G::CS_OFF + wave * 1024), tv.cs, rs_cs);
      else if (kind == 1) dma16z(sb + (uint32_t)(G::CT_OFF + wave * 1024), tv.cs, rs_ct);
      else dma4z(sb + (uint32_t)(SLOFF + wave * 256), tv.sl, rs_slot);
    }
  };

  // ---- accumulators: set P of tile i; the owned blocks of tile i-1 wait in
  // set P ^ 1 for the partner's partial sums
  f32x4_t acc[2][8];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[p][b] = (f32x4_t){0.f, 0.f, 0.f, 0.f};

  // ---- epilogue state of tile i-1
  u32x4_t ct[2] = {{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
  uint32_t slotv = 0;
  u32x4_t xs[4];
  u32x4_t ev[2];
  uint32_t eo = 0;
  float y[2][8];
  // part e (0..7) of the epilogue of tile j from accumulator set p: element e
  // of both output halves; the target RoPE and the rounding once both members
  // of a plane are there
  auto epilogue_part = [&](int p, int j, int e) __attribute__((always_inline)) {
    if (e == 0) {
      // output row of the token this lane stores (32-bit: every byte offset
      // of the target plane fits)
      const uint32_t tl = t_begin32 + (uint32_t)(MT * j + row);
      const uint32_t orow = SLOTS ? slotv : tl;
      const bool ok = mine && j >= 0 && tl < t_end32 && orow < rows32;
      eo = ok ? orow * (uint32_t)ROWB + colb : 0xffffff00u;
    }
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int bb = 4 * x + 2 * OH + (e >> 2);
      y[x][e] = acc[p][bb][e & 3] + __uint_as_float(xs[2 * x + (e >> 2)][e & 3]);
    }
    if (KEYS) {
      const uint32_t cwd = ct[e >> 2][e & 3];
      if (STYLE == 0) {
        rot_fwd16(y[0][e], y[1][e], cwd);
      } else if (e & 1) {
        // planes (e - 1, e) of each half: coefficient word 4 x + e / 2
        rot_fwd16(y[0][e - 1], y[0][e], ct[0][e >> 1]);
        rot_fwd16(y[1][e - 1], y[1][e], ct[1][e >> 1]);
      }
    }
    if (e & 1) {
      ev[0][e >> 1] = pack2(y[0][e - 1], y[0][e]);
      ev[1][e >> 1] = pack2(y[1][e - 1], y[1][e]);
      pin(ev[0], ev[1]);
    } else {
      pin(y[0][e], y[1][e]);
    }
  };
  auto epilogue_store = [&](int x) __attribute__((always_inline)) {
    if (x == 0) vstore16_near<0>(ev[0], eo, rs_out);   // rs_out: formed at the unit's start
    else vstore16_near<128>(ev[1], eo, rs_out);
  };
  auto exchange_read = [&](int p, int k) __attribute__((always_inline)) {
    const uint32_t base = xr + (uint32_t)(p * 16384);
    switch (k) {
      case 0: lds_read<0>(xs[0], base); break;
      case 1: lds_read<1024>(xs[1], base); break;
      case 2: lds_read<2048>(xs[2], base); break;
      default: lds_read<3072>(xs[3], base); break;
    }
  };
  auto exchange_write = [&](int p, int k) __attribute__((always_inline)) {
    const uint32_t base = xw + (uint32_t)(p * 16384);
    switch (k) {
      case 0: lds_write<0>(base, __builtin_bit_cast(u32x4_t, acc[p][PB])); break;
      case 1: lds_write<1024>(base, __builtin_bit_cast(u32x4_t, acc[p][PB + 1])); break;
      case 2: lds_write<2048>(base, __builtin_bit_cast(u32x4_t, acc[p][PB + 4])); break;
      default: lds_write<3072>(base, __builtin_bit_cast(u32x4_t, acc[p][PB + 5])); break;
    }
  };
  // epilogue inputs of the tile in stage base sb: target coefficients, slot
  // index of the token this lane stores
  auto ct_read = [&](uint32_t sb, int k) __attribute__((always_inline)) {
    if (k == 0) lds_read<0>(ct[0], sb + vct0);
    else lds_read<0>(ct[1], sb + vct1);
  };
  auto sl_read = [&](uint32_t sb) __attribute__((always_inline)) {
    lds_read_b32(slotv, sb + (uint32_t)(SLOFF + wave * 256 + row * 4));
  };

  // ---- operand fragments: a ring of four; fragment f of tile i sits in
  // fr[(i * ZH + f) % 4]
  u32x4_t fr[4];
  u32x4_t cs[4];
  // fragment f (quarter f % 4 of slot f / 4) of the tile in stage base sb
  auto frag_read = [&](uint32_t sb, u32x4_t& d, int f) __attribute__((always_inline)) {
    if (SPLIT) {
      // the x and y pieces 128 bytes apart
      lds_read2_b64<0, 16>(d, sb + fpos[f >> 2][f & 3]);
    } else {
      lds_read<0>(d, sb + fpos[f >> 2][f & 3]);
    }
  };
  // strip the source RoPE from fragment register f with coefficients cf, part
  // pt of 8 (one after each matrix instruction)
  float su[2], sv[2];
  auto strip_part = [&](u32x4_t& f, const u32x4_t& cf, int pt) __attribute__((always_inline)) {
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

  // ---- pipeline prologue: tiles 0 .. NS-2 in flight, then tile 0's
  // coefficients and fragments 0 and 1 in registers, fragment 0 stripped
#pragma unroll
  for (int j = 0; j < NS - 1; ++j) {
    const uint32_t sb = stage_base(j);
    const TileVo tv = tile_vo(j);
#pragma unroll
    for (int f = 0; f < ZH; ++f) own_load(sb, tv, f, std::false_type{});
#pragma unroll
    for (int n = 0; n < S::NC; ++n) c_load(sb, tv, n, std::false_type{});
  }
  vm_wait_c<(NS - 2) * S::NL>();               // tile 0 is in LDS
  __syncthreads();
  {
    const uint32_t sb = stage_base(0);
    if (KEYS) {
#pragma unroll
      for (int s = 0; s < 4; ++s)
        if (S::cs_used(s)) lds_read<0>(cs[s], sb + cpos[s]);
    }
    frag_read(sb, fr[0], 0);
    frag_read(sb, fr[1], 1);
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fr[0]), "+v"(fr[1]), "+v"(cs[0]), "+v"(cs[1]));
    pin(cs[2], cs[3]);
    if (KEYS) {
#pragma unroll
      for (int pt = 0; pt < 8; ++pt) strip_part(fr[0], cs[S::sof(0)], pt);
    }
  }

  // ---- tile i in stage st with accumulator set P = i % 2
  auto tile = [&](auto pc, int i, int st) __attribute__((always_inline)) {
    constexpr int P = decltype(pc)::value;
    constexpr int FB = (P * ZH) % 4;           // fragment ring base of this tile
    const int stp = st == 0 ? NS - 1 : st - 1;    // tile i-1's stage: loads of tile i+NS-1 go there
    const int stn = st + 1 == NS ? 0 : st + 1;    // tile i+1's stage
    const uint32_t sb_cur = stage_base(st), sb_prev = stage_base(stp), sb_next = stage_base(stn);
    // the voffsets of the tile loaded in this one
    const TileVo tl = tile_vo(i + NS - 1);

    static_for<0, ZH>([&](auto zc) __attribute__((always_inline)) {
      constexpr int zz = decltype(zc)::value;
      constexpr int F2 = zz + 2;               // fragment read in this step
      constexpr int FS = zz + 1;               // fragment stripped in this step (keys)
      u32x4_t& xcur = fr[(FB + zz) % 4];
      if constexpr (!KEYS) lgk_wait_c<S::v_wait(zz)>();
      asm volatile("" : "+v"(xcur));
      const u32x4_t x = xcur;
      if constexpr (KEYS) asm volatile("s_nop 1");
      static_for<0, 8>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        constexpr int b = ks2_block(j, OH);
        if constexpr (zz == 0) {
          if constexpr (((b >> 1) & 1) == OH) mfma_init(acc[P][b], wf[b][zz], x, bias[(b >> 2) * 2 + (b & 1)]);
          else mfma_zero(acc[P][b], wf[b][zz], x);
        } else {
          mfma_acc(acc[P][b], wf[b][zz], x);
        }
        // o 1: the mid-tile barrier
        if constexpr (zz == MB && j == 0) {
          vm_wait_c<S::vm_mid(NS)>();
          lgk_wait_c<S::bar_wait()>();
          __builtin_amdgcn_s_barrier();
        }
        // o 2: fragment read two steps ahead
        if constexpr (j == 0) {
          if constexpr (F2 < ZH) frag_read(sb_cur, fr[(FB + F2) % 4], F2);
          else frag_read(sb_next, fr[(FB + F2) % 4], F2 - ZH);
        }
        // o 3: the partner's sums of tile i-1
        if constexpr (zz == MB && j >= 1 && j <= 4) exchange_read(P ^ 1, j - 1);
        // o 4: the partner's blocks of tile i-1, once the matrix results are
        // readable; the epilogue inputs of tile i-1
        if constexpr (zz == 0 && j == 1)
          asm volatile("s_nop 7\n\ts_nop 3" : "+v"(acc[P ^ 1][PB]), "+v"(acc[P ^ 1][PB + 1]),
                       "+v"(acc[P ^ 1][PB + 4]), "+v"(acc[P ^ 1][PB + 5]));
        if constexpr (zz == 0 && j >= 1 && j <= 4) exchange_write(P ^ 1, j - 1);
        if constexpr (zz == 0 && KEYS && (j == 5 || j == 6)) ct_read(sb_prev, j - 5);
        if constexpr (zz == 0 && SLOTS && j == 7) sl_read(sb_prev);
        // o 5..8: coefficients of tile i+1
        if constexpr (KEYS) {
          static_for<0, 4>([&](auto sc) __attribute__((always_inline)) {
            constexpr int s = decltype(sc)::value;
            if constexpr (S::cs_used(s) && S::cs_step(s) == zz && S::cs_j(s) == j)
              lds_read<0>(cs[s], sb_next + cpos[s]);
          });
        }
        // o 7: inputs of this step's vector work
        if constexpr (j == 0) {
          if constexpr (KEYS) {
            lgk_wait_c<S::k_wait(zz)>();
            asm volatile("" : "+v"(fr[(FB + FS) % 4]), "+v"(cs[S::sof(FS % ZH)]));
          } else if constexpr (zz == EPI) {
            lgk_wait_c<S::e_wait()>();
          }
          if constexpr (zz == EPI) {
            asm volatile("" : "+v"(xs[0]), "+v"(xs[1]), "+v"(xs[2]), "+v"(xs[3]));
            asm volatile("" : "+v"(ct[0]), "+v"(ct[1]), "+v"(slotv));
          }
        }
        // o 8: the stores of tile i-1
        if constexpr (zz == S::ST && j == S::S0J) {
          epilogue_store(0);
          if constexpr (S::S1J == S::S0J) epilogue_store(1);
        }
        if constexpr (zz == S::ST && j == S::S1J && S::S1J != S::S0J) epilogue_store(1);
        // the stage these loads overwrite held tile i-1, whose fragments
        // another wave may have read (a shared source slot): every wave is
        // done with them here
        if constexpr (zz == 0 && j == 2) __builtin_amdgcn_s_barrier();
        // o 9: loads of tile i+NS-1
        if constexpr (zz < MB && j == 3) own_load(sb_prev, tl, 2 * zz, std::true_type{});
        if constexpr (zz < MB && j == 6) own_load(sb_prev, tl, 2 * zz + 1, std::true_type{});
        if constexpr (zz == MB && j >= 5 && j < 5 + S::NC) c_load(sb_prev, tl, j - 5, std::true_type{});
        // vector work: strip the next fragment (keys), finish tile i-1
        if constexpr (KEYS) strip_part(fr[(FB + FS) % 4], cs[S::sof(FS % ZH)], j);
        if constexpr (zz == EPI) {
          if constexpr (ZH == 8) {
            epilogue_part(P ^ 1, i - 1, j);
          } else if constexpr (j < 4) {
            epilogue_part(P ^ 1, i - 1, 2 * j);
            epilogue_part(P ^ 1, i - 1, 2 * j + 1);
          }
        }
      });
    });
  };
  // the last tile j (set p): its partner sums through LDS, then its epilogue
  auto final_epilogue = [&](int p, int j, int st) __attribute__((always_inline)) {
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc[p][0]), "+v"(acc[p][1]), "+v"(acc[p][2]),
                 "+v"(acc[p][3]));
    asm volatile("" : "+v"(acc[p][4]), "+v"(acc[p][5]), "+v"(acc[p][6]), "+v"(acc[p][7]));
#pragma unroll
    for (int k = 0; k < 4; ++k) exchange_write(p, k);
    if (KEYS) {
      ct_read(stage_base(st), 0);
      ct_read(stage_base(st), 1);
    }
    if (SLOTS) sl_read(stage_base(st));
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(ct[0]), "+v"(ct[1]), "+v"(slotv));
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) exchange_read(p, k);
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xs[0]), "+v"(xs[1]), "+v"(xs[2]), "+v"(xs[3]));
#pragma unroll
    for (int e = 0; e < 8; ++e) epilogue_part(p, j, e);
    epilogue_store(0);
    epilogue_store(1);
  };

  // Two tiles per trip, so that the accumulator sets and the fragment ring
  // positions are constants.
  int st = 0;
  for (int i0 = 0; i0 < n_tiles; i0 += 2) {
    tile(std::integral_constant<int, 0>{}, i0, st);
    if (i0 + 1 >= n_tiles) { final_epilogue(0, i0, st); break; }
    st = st + 1 == NS ? 0 : st + 1;
    tile(std::integral_constant<int, 1>{}, i0 + 1, st);
    if (i0 + 2 >= n_tiles) { final_epilogue(1, i0 + 1, st); break; }
    st = st + 1 == NS ? 0 : st + 1;
  }
  // everything this unit issued has landed, and every wave is done with the
  // exchange area and the stages, before the next unit reuses LDS
  vm_wait_c<0>();
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __syncthreads();
}

// The sweep plan and the order in which each layer group's target layers
// are paired: positions 2 j and 2 j + 1 of a group form pair j, and
// order[position] is the layer's index within its group.
struct Ks2Plan {
  SweepPlan sp;
  uint8_t order[kMaxIdx / 2];   // k >= 2: at most kMaxIdx / 2 target layers
};
static_assert(sizeof(MapArgs) + sizeof(Ks2Plan) <= 4096, "kernel arguments");

template <int K, int STYLE, bool SLOTS, bool TGT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void map_ks2_kernel(const MapArgs a, const Ks2Plan kp) {
  const SweepPlan& p = kp.sp;
  __shared__ __attribute__((aligned(256))) char smem[GeoK2<K, SLOTS, TGT>::LDS];
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_u32(smem));

  Ks2Ctx q;
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
    const bool has1 = 2 * pair + 1 < g_n;
    const int l_a = g0 + kp.order[g0 + 2 * pair];
    const int l_b = has1 ? g0 + kp.order[g0 + 2 * pair + 1] : l_a;
    if (kv == 0) {
      if (kh == 0) ks2_unit<K, STYLE, SLOTS, TGT, 0, 0>(a, lds0, q, h, l_a, l_b, has1);
      else ks2_unit<K, STYLE, SLOTS, TGT, 0, 1>(a, lds0, q, h, l_a, l_b, has1);
    } else {
      if (kh == 0) ks2_unit<K, STYLE, SLOTS, TGT, 1, 0>(a, lds0, q, h, l_a, l_b, has1);
      else ks2_unit<K, STYLE, SLOTS, TGT, 1, 1>(a, lds0, q, h, l_a, l_b, has1);
    }
  }
}

template <int K, int STYLE, bool SLOTS, bool TGT>
hipError_t launch_ks2k(const MapArgs& a, const Ks2Plan& p, hipStream_t stream) {
  if constexpr (GeoK2<K, SLOTS, TGT>::fits) {
    hipLaunchKernelGGL((map_ks2_kernel<K, STYLE, SLOTS, TGT>), dim3(256), dim3(NT), 0, stream, a, p);
    return hipGetLastError();
  } else {
    return hipErrorInvalidValue;
  }
}

template <int K, int STYLE>
hipError_t launch_ks2slots(const MapArgs& a, const Ks2Plan& p, hipStream_t stream) {
  const bool slots = a.slots != nullptr, tgt = a.cs16_tgt != a.cs16;
  if (slots)
    return tgt ? launch_ks2k<K, STYLE, true, true>(a, p, stream) : launch_ks2k<K, STYLE, true, false>(a, p, stream);
  return tgt ? launch_ks2k<K, STYLE, false, true>(a, p, stream) : launch_ks2k<K, STYLE, false, false>(a, p, stream);
}

template <int K>
hipError_t launch_ks2style(const MapArgs& a, const Ks2Plan& p, int style, hipStream_t stream) {
  return style == 0 ? launch_ks2slots<K, 0>(a, p, stream) : launch_ks2slots<K, 1>(a, p, stream);
}

template <int K>
bool ks2_fits(bool slots, bool tgt) {
  return slots ? (tgt ? GeoK2<K, true, true>::fits : GeoK2<K, true, false>::fits)
               : (tgt ? GeoK2<K, false, true>::fits : GeoK2<K, false, false>::fits);
}

}  // namespace

bool map_ks2_supported(int k, int64_t T, int64_t tgt_rows, bool slots, bool tgt_rope) {
  // byte offsets within a plane, and of the tiles loaded ahead past its end,
  // must fit the 32-bit buffer offsets; the stages must fit the LDS
  if (T < 1 || (T + 80) * ROWB >= 0xffffff00LL || tgt_rows * ROWB >= 0xffffff00LL) return false;
  switch (k) {
    case 2: return ks2_fits<2>(slots, tgt_rope);
    case 4: return ks2_fits<4>(slots, tgt_rope);
    default: return false;   // a wave's reduction half would split a source layer
  }
}

static void ks2_pair_order(const uint8_t* idx, int k, int g0, int g_n, uint8_t* order) {
  // sh[i][j]: sources of layer j that layer i also lists (the slots of a
  // pair's second layer that read the first layer's)
  int sh[64][64];
  for (int i = 0; i < g_n; ++i)
    for (int j = 0; j < g_n; ++j) {
      int n = 0;
      for (int r = 0; r < k; ++r)
        for (int t = 0; t < k; ++t)
          if (idx[(g0 + j) * k + r] == idx[(g0 + i) * k + t]) {
            ++n;
            break;
          }
      sh[i][j] = n;
    }
  auto s = [&](int i, int j) { return sh[i][j] > sh[j][i] ? sh[i][j] : sh[j][i]; };
  // Each CU keeps its pair for the whole launch, so the pairs that share
  // nothing set the time: match as many layers as possible to a partner that
  // shares a source.  Min-degree greedy: the unmatched layer with the fewest
  // unmatched sharing partners takes the partner that shares the most (then
  // the one with the fewest partners left); the rest are paired in order.
  bool used[64] = {};
  int deg[64];
  for (int i = 0; i < g_n; ++i) {
    deg[i] = 0;
    for (int j = 0; j < g_n; ++j) deg[i] += j != i && s(i, j) > 0;
  }
  int n = 0;
  for (;;) {
    int i = -1;
    for (int c = 0; c < g_n; ++c)
      if (!used[c] && deg[c] > 0 && (i < 0 || deg[c] < deg[i])) i = c;
    if (i < 0) break;
    int j = -1;
    for (int c = 0; c < g_n; ++c)
      if (!used[c] && c != i && s(i, c) > 0 &&
          (j < 0 || s(i, c) > s(i, j) || (s(i, c) == s(i, j) && deg[c] < deg[j])))
        j = c;
    const int a = sh[i][j] >= sh[j][i] ? i : j, b = a == i ? j : i;
    order[g0 + n++] = (uint8_t)a;
    order[g0 + n++] = (uint8_t)b;
    used[i] = used[j] = true;
    for (int c = 0; c < g_n; ++c)
      if (!used[c]) deg[c] -= (s(c, i) > 0) + (s(c, j) > 0);
  }
  for (int c = 0; c < g_n; ++c)
    if (!used[c]) order[g0 + n++] = (uint8_t)c;
}

hipError_t launch_map_ks2(const MapArgs& a, const SweepPlan& sp, int style, hipStream_t stream) {
  if (a.T == 0 || a.nl == 0) return hipSuccess;
  if (a.nl > kMaxIdx / 2) return hipErrorInvalidValue;
  Ks2Plan p;
  p.sp = sp;
  int g0 = 0;
  for (int g = 0; g < sp.n_groups; ++g) {
    const int g_n = g < sp.full_groups ? 64 : sp.rest_len[g - sp.full_groups];
    ks2_pair_order(a.idx, a.k, g0, g_n, p.order);
    g0 += g_n;
  }
  switch (a.k) {
    case 2: return launch_ks2style<2>(a, p, style, stream);
    case 4: return launch_ks2style<4>(a, p, style, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kvx
