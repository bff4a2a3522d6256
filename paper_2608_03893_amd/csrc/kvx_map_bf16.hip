// W-stationary map kernel for bf16 caches with head dimension 128 and k <= 4.
//
// One workgroup (8 waves, two per SIMD) owns one (target layer, head, K|V)
// task and a contiguous token range.  It stages the task's map W^T
// ([128 output dims] x [k*128 input features], bf16) once into LDS and then
// streams the range in tiles of 256 tokens, 32 per wave:
//
//   1. each lane loads its token's rows of the k selected source layers
//      straight from HBM into registers (no LDS round trip for the cache),
//      one source block ahead of the one being multiplied;
//   2. keys are stripped of the source RoPE in registers (Sec. 3.3), with the
//      tile's cos/sin held in registers as fp16 pairs and consumed by mixed
//      fp16/fp32 FMAs, then rounded once to bf16;
//   3. the contraction runs as C^T = W^T X^T on v_mfma_f32_32x32x16_bf16
//      (Eq. ridge_kv): W^T fragments come from LDS, X^T fragments come from
//      registers and are reused by all four 32-row output blocks;
//   4. bias, target RoPE and the bf16 rounding happen in registers and each
//      lane stores 16 contiguous output channels per 32-channel block.
// Two waves per SIMD let one wave's matrix-core work overlap the other's
// memory waits and RoPE arithmetic.
//
// Operand layout.  In the 32x32x16 instruction lane L supplies operand row /
// column L % 32 and reduction indices 8*(L/32) .. 8*(L/32)+7 of the 16-wide
// step; accumulator register r of lane L holds output row 8*(r/4)+4*(L/32)+r%4
// and column L % 32.  Two permutations, applied once while W^T is staged, make
// these positions convenient:
//   input  sigma: step s (0..7) of a source block, lane half g, element q maps
//          to channel 32g + 8s + q for s < 4 and 64 + 32g + 8(s-4) + q for
//          s >= 4, so a lane holds both channels j and j+64 of every RoPE plane
//          it touches and reads 64 contiguous bytes per half row;
//   output pi: accumulator row 8a + 4g + b of a 32-row block maps to output
//          channel 16g + 4a + b of that block, so register r of lane L is
//          channel 32*nb + 16*(L/32) + r.
// A reduction is invariant under a common permutation of its index, and the
// output permutation is undone by where each lane stores.
#include "kvx_internal.h"

#include <hip/hip_fp16.h>

namespace kvx {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int D = 128;
constexpr int HALF = 64;

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  __bf16 a = (__bf16)lo;
  __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

// Inverse rotation of plane (u, v) by the angle whose (cos, sin) is the fp16
// pair cs.  fma(x, y, 0) keeps the fp16 operand inside a mixed-precision FMA.
__device__ __forceinline__ void strip(float& u, float& v, uint32_t cs) {
  const __half2 h = __builtin_bit_cast(__half2, cs);
  const float c = __low2float(h), s = __high2float(h);
  const float u0 = u, v0 = v;
  u = __builtin_fmaf(u0, c, __builtin_fmaf(v0, s, 0.0f));
  v = __builtin_fmaf(v0, c, -__builtin_fmaf(u0, s, 0.0f));
}

// Strip 8 planes whose first channels are packed in a and second channels in
// b (half-split layout: channels j and j+64 in matching positions).
__device__ __forceinline__ void strip_halfsplit(uint4& a, uint4& b, const uint32_t* cs) {
  uint32_t* pa = reinterpret_cast<uint32_t*>(&a);
  uint32_t* pb = reinterpret_cast<uint32_t*>(&b);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float u0 = lo_bf16(pa[w]), u1 = hi_bf16(pa[w]);
    float v0 = lo_bf16(pb[w]), v1 = hi_bf16(pb[w]);
    strip(u0, v0, cs[2 * w]);
    strip(u1, v1, cs[2 * w + 1]);
    pa[w] = pack2(u0, u1);
    pb[w] = pack2(v0, v1);
  }
}

// Strip the 4 interleaved planes (2m, 2m+1) held in one 8-channel group.
__device__ __forceinline__ void strip_interleaved(uint4& a, const uint32_t* cs) {
  uint32_t* pa = reinterpret_cast<uint32_t*>(&a);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float u = lo_bf16(pa[w]), v = hi_bf16(pa[w]);
    strip(u, v, cs[w]);
    pa[w] = pack2(u, v);
  }
}

// Packed map image.  For one task the LDS image of W^T is dense:
// [128 accumulator rows rho][k*128 reduction columns kappa] bf16, where row rho
// holds output channel pi(rho) and column kappa = 16*(8i + s) + 8g + q holds
// input feature 128*i + sigma(s, g, q).  Each 16-byte chunk c = kappa / 8 of
// row rho is stored at chunk position c ^ (rho & 15), so that the 32 rows read
// by one MFMA fragment load fall on distinct LDS banks.  pack_w_kernel writes
// this image to global memory once per call; workgroups copy it to LDS as is.
__device__ __forceinline__ int pi_inv(int n) {  // output channel -> row
  const int nb = n / 32, m = n % 32;
  return 32 * nb + 8 * ((m % 16) / 4) + 4 * (m / 16) + (m % 4);
}

// One thread per (task, 8 input rows, 8 output columns): read the 8x8 block of
// W, transpose it in registers and write 8 chunks of the packed image.
template <int K>
__global__ __launch_bounds__(256) void pack_w_kernel(const uint16_t* __restrict__ wk,
                                                     const uint16_t* __restrict__ wv,
                                                     uint16_t* __restrict__ wp, int l0, int nl,
                                                     int H) {
  constexpr int KD = K * D;
  constexpr int BLOCKS = (KD / 8) * (D / 8);
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n_tasks = (int64_t)nl * H * 2;
  if (gid >= n_tasks * BLOCKS) return;
  const int64_t task = gid / BLOCKS;          // ((l - l0) * H + h) * 2 + kv
  const int blk = (int)(gid % BLOCKS);
  const int kv = (int)(task & 1);
  const int64_t lh = (int64_t)l0 * H + (task >> 1);   // l * H + h
  const uint16_t* W = (kv ? wv : wk) + lh * (int64_t)KD * D;
  uint16_t* out = wp + (lh * 2 + kv) * (int64_t)D * KD;
  const int rb = blk / (D / 8);  // input rows 8rb .. 8rb+7
  const int cb = blk % (D / 8);  // output columns 8cb .. 8cb+7
  uint4 r[8];
#pragma unroll
  for (int q = 0; q < 8; ++q)
    r[q] = *reinterpret_cast<const uint4*>(W + (int64_t)(8 * rb + q) * D + 8 * cb);
  // input rows -> reduction chunk (sigma^-1)
  const int i = (8 * rb) / D;
  const int d0 = (8 * rb) % D;
  const int upper = d0 / HALF, dd = d0 % HALF;
  const int g = dd / 32, s = (dd % 32) / 8 + 4 * upper;
  const int chunk = 2 * (8 * i + s) + g;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int rho = pi_inv(8 * cb + c);
    uint32_t w4[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t* a0 = reinterpret_cast<const uint32_t*>(&r[2 * p]);
      const uint32_t* a1 = reinterpret_cast<const uint32_t*>(&r[2 * p + 1]);
      const uint32_t e0 = (c & 1) ? (a0[c / 2] >> 16) : (a0[c / 2] & 0xffffu);
      const uint32_t e1 = (c & 1) ? (a1[c / 2] >> 16) : (a1[c / 2] & 0xffffu);
      w4[p] = e0 | (e1 << 16);
    }
    *reinterpret_cast<uint4*>(out + (int64_t)rho * KD + 8 * (chunk ^ (rho & 15))) =
        make_uint4(w4[0], w4[1], w4[2], w4[3]);
  }
}

// Copy one task's packed image into LDS: all loads are issued before any store.
template <int K, int NT>
__device__ __forceinline__ void stage_wt(uint16_t* Wt, const uint16_t* __restrict__ img, int tid) {
  constexpr int CHUNKS = D * K * D / 8;   // 16-byte chunks
  constexpr int PER = CHUNKS / NT;
  static_assert(CHUNKS % NT == 0, "image must split evenly over the workgroup");
  uint4 v[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) v[j] = reinterpret_cast<const uint4*>(img)[tid + j * NT];
#pragma unroll
  for (int j = 0; j < PER; ++j) reinterpret_cast<uint4*>(Wt)[tid + j * NT] = v[j];
}

// Forward rotation of plane (u, v) by the angle whose (cos, sin) is the fp16
// pair cs.
__device__ __forceinline__ void rot_fwd16(float& u, float& v, uint32_t cs) {
  const __half2 h = __builtin_bit_cast(__half2, cs);
  const float c = __low2float(h), s = __high2float(h);
  const float u0 = u, v0 = v;
  u = __builtin_fmaf(u0, c, -__builtin_fmaf(v0, s, 0.0f));
  v = __builtin_fmaf(v0, c, __builtin_fmaf(u0, s, 0.0f));
}

// NW waves per workgroup, each owning TB 32-token blocks of every tile; PD
// source blocks (1 or 2) in flight ahead of the one being multiplied.
template <int K, int STYLE, bool SLOTS, int NW, int TB, int PD>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4)))
void map_w_kernel(const MapArgs a) {
  constexpr int KD = K * D;
  constexpr int NT = NW * 64;
  constexpr int TILE = NW * 32 * TB;
  __shared__ __attribute__((aligned(16))) uint16_t Wt[D * KD];
  __shared__ __attribute__((aligned(16))) float Bs[D];  // bias, fp32
  // per-wave staging of one 32-channel output block, [TB*32 tokens][32] bf16:
  // lets each store instruction write 64 contiguous bytes of 16 rows
  __shared__ __attribute__((aligned(16))) uint16_t Ys[NW][TB * 32 * 32];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 5;     // lane half
  const int row = lane & 31;   // token within a 32-token block

  // ---- work item: (head, K|V, layer, token range)
  int h, kv, ll, range;
  {
    const int item = blockIdx.x;
    if (a.H % 8 == 0) {
      // workgroup i runs on XCD i % 8: give each XCD its own heads so the
      // workgroups resident on one XCD share source rows in its L2
      const int xcd = item & 7;
      int slot = item >> 3;
      const int hg = a.H / 8;
      h = xcd + 8 * (slot % hg);
      slot /= hg;
      ll = slot % a.nl;
      slot /= a.nl;
      kv = slot & 1;
      range = slot >> 1;
    } else {
      const int n_tasks = a.nl * a.H * 2;
      range = item / n_tasks;
      const int task = item % n_tasks;
      ll = task % a.nl;
      kv = (task / a.nl) & 1;
      h = task / (a.nl * 2);
    }
  }
  const int l = a.l0 + ll;
  const int64_t T = a.T;
  const int64_t t_begin = (int64_t)range * a.range_len;
  const int64_t t_end = t_begin + a.range_len < T ? t_begin + a.range_len : T;

  // ---- stage W^T and the bias (content space, NULL = zero) in LDS
  stage_wt<K, NT>(Wt, reinterpret_cast<const uint16_t*>(a.wpack) +
                          (((int64_t)l * a.H + h) * 2 + kv) * (int64_t)D * KD, tid);
  {
    const uint16_t* bias = reinterpret_cast<const uint16_t*>(kv ? a.bv : a.bk);
    if (tid < D)
      Bs[tid] = bias != nullptr ? lo_bf16(bias[((int64_t)l * a.H + h) * D + tid]) : 0.0f;
  }
  __syncthreads();

  uint16_t* out = reinterpret_cast<uint16_t*>(a.tgt) + (((int64_t)l * 2 + kv) * a.H + h) * a.tgt_rows * D;
  const uint32_t* cs_s = reinterpret_cast<const uint32_t*>(a.cs16);
  const uint32_t* cs_t = reinterpret_cast<const uint32_t*>(a.cs16_tgt);

  // Rows of the k selected source layers for this (head, K|V): scalar pointers.
  const uint16_t* Xb[K];
#pragma unroll
  for (int i = 0; i < K; ++i)
    Xb[i] = reinterpret_cast<const uint16_t*>(a.src) +
            (((int64_t)a.idx[ll * K + i] * 2 + kv) * a.H + h) * T * D;

  // Token row of block tb of this lane in the tile starting at tt, clamped to
  // the range so every load is in bounds and unconditional; a clamped row only
  // feeds its own (discarded) output column of C^T.
  auto lane_row = [&](int64_t tt, int tb) -> int64_t {
    const int64_t t = tt + 32 * (TB * wave + tb) + row;
    return t < t_end ? t : t_end - 1;
  };
  // Channels 32g..32g+31 (xu) and 64+32g..64+32g+31 (xv) of one source row.
  auto load_block = [&](const uint16_t* X, int64_t t, uint4 (&xu)[4], uint4 (&xv)[4]) {
    const uint16_t* p = X + t * D + 32 * g;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      xu[s] = *reinterpret_cast<const uint4*>(p + 8 * s);
      xv[s] = *reinterpret_cast<const uint4*>(p + HALF + 8 * s);
    }
  };
  // fp16 (cos, sin) pairs of the 32 planes the strip touches (source RoPE):
  // half-split planes 32g .. 32g+31; interleaved planes 16g..16g+15 and
  // 32+16g .. 32+16g+15.
  auto load_cs_strip = [&](int64_t t, uint32_t (&cs)[32]) {
    const uint32_t* p = cs_s + t * HALF;
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      const int j0 = (STYLE == 0) ? 32 * g + 4 * v
                                  : (v < 4 ? 16 * g + 4 * v : 32 + 16 * g + 4 * (v - 4));
      const uint4 c4 = *reinterpret_cast<const uint4*>(p + j0);
      cs[4 * v] = c4.x; cs[4 * v + 1] = c4.y; cs[4 * v + 2] = c4.z; cs[4 * v + 3] = c4.w;
    }
  };
  // fp16 (cos, sin) pairs of the 32 planes the epilogue touches (target RoPE):
  // half-split planes 32nb + 16g + r (nb < 2); interleaved planes
  // 16nb + 8g + r/2 (nb < 4).
  auto load_cs_out = [&](int64_t t, uint32_t (&cs)[32]) {
    const uint32_t* p = cs_t + t * HALF;
#pragma unroll
    for (int v = 0; v < 8; ++v) {
      const int j0 = (STYLE == 0) ? 32 * (v / 4) + 16 * g + 4 * (v % 4)
                                  : 16 * (v / 2) + 8 * g + 4 * (v % 2);
      const uint4 c4 = *reinterpret_cast<const uint4*>(p + j0);
      cs[4 * v] = c4.x; cs[4 * v + 1] = c4.y; cs[4 * v + 2] = c4.z; cs[4 * v + 3] = c4.w;
    }
  };

  // Software pipeline over the stream of (tile, source block) steps: the rows
  // of the next PD steps are always in flight while the current block is
  // stripped and multiplied.  The coefficient registers hold the strip pairs
  // of the current tile until its last strip, then the epilogue pairs, then
  // the next tile's strip pairs.
  uint4 qxu[PD][TB][4], qxv[PD][TB][4];   // queue of loaded blocks, [0] oldest
  uint32_t cs[TB][32];
  // Block j (0 <= j < PD) of the stream starting at tile tt: tile tt + TILE *
  // ((i0 + j) / K), source block (i0 + j) % K.
  auto issue = [&](int64_t tt, int ib, uint4 (&xu)[TB][4], uint4 (&xv)[TB][4]) {
    const int64_t tq = tt + (int64_t)TILE * (ib / K);
    const int64_t tl = tq < t_end ? tq : tt;   // past the range: reload (and discard) tile tt
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) load_block(Xb[ib % K], lane_row(tl, tb), xu[tb], xv[tb]);
  };
#pragma unroll
  for (int j = 0; j < PD; ++j) issue(t_begin, j, qxu[j], qxv[j]);
  if (kv == 0) {
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) load_cs_strip(lane_row(t_begin, tb), cs[tb]);
  }

  for (int64_t tt = t_begin; tt < t_end; tt += TILE) {
    // the last tile prefetches (and discards) its own rows again
    const int64_t tt_next = tt + TILE < t_end ? tt + TILE : tt;
    int64_t t_here[TB], t_next[TB], orow[TB];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      t_here[tb] = lane_row(tt, tb);
      t_next[tb] = lane_row(tt_next, tb);
      // destination row (slot index loaded here, long before it is needed)
      orow[tb] = SLOTS ? (int64_t)a.slots[t_here[tb]] : tt + 32 * (TB * wave + tb) + row;
    }

    f32x16_t acc[TB][4];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[tb][nb][r] = 0.0f;

#pragma unroll
    for (int i = 0; i < K; ++i) {
      uint4 xu[TB][4], xv[TB][4];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          xu[tb][s] = qxu[0][tb][s];
          xv[tb][s] = qxv[0][tb][s];
        }
#pragma unroll
      for (int j = 0; j + 1 < PD; ++j)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            qxu[j][tb][s] = qxu[j + 1][tb][s];
            qxv[j][tb][s] = qxv[j + 1][tb][s];
          }
      // the step PD ahead: within this tile, or in the next one
      const bool ahead_in_tile = i + PD < K;
      if (ahead_in_tile) issue(tt, i + PD, qxu[PD - 1], qxv[PD - 1]);
      __builtin_amdgcn_sched_barrier(0);
      // ---- strip the source RoPE (keys)
      if (kv == 0) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb)
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            if (STYLE == 0) {
              strip_halfsplit(xu[tb][s], xv[tb][s], &cs[tb][8 * s]);
            } else {
              strip_interleaved(xu[tb][s], &cs[tb][4 * s]);
              strip_interleaved(xv[tb][s], &cs[tb][16 + 4 * s]);
            }
          }
        if (i + 1 == K) {
#pragma unroll
          for (int tb = 0; tb < TB; ++tb) load_cs_out(t_here[tb], cs[tb]);
        }
      }
      if (!ahead_in_tile) issue(tt, i + PD, qxu[PD - 1], qxv[PD - 1]);
      __builtin_amdgcn_sched_barrier(0);
      // ---- contraction: 8 reduction steps of 16; each W^T fragment feeds
      // the TB token blocks of the wave
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int chunk = (2 * (8 * i + s) + g) ^ (row & 15);
        bf16x8_t wa[4];
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          wa[nb] = *reinterpret_cast<const bf16x8_t*>(Wt + (32 * nb + row) * KD + 8 * chunk);
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          const bf16x8_t xb = as_bf16x8(s < 4 ? xu[tb][s] : xv[tb][s - 4]);
#pragma unroll
          for (int nb = 0; nb < 4; ++nb)
            acc[tb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[nb], xb, acc[tb][nb], 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue: bias, target RoPE, round, store (channel 32nb + 16g + r).
    // Stores are issued last: the memory counter retires loads and stores in
    // order, so anything loaded after a store would wait for it.
    float y[TB][4][16];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
#pragma unroll
        for (int r = 0; r < 16; r += 4) {
          const float4 b = *reinterpret_cast<const float4*>(&Bs[32 * nb + 16 * g + r]);
          y[tb][nb][r] = acc[tb][nb][r] + b.x;
          y[tb][nb][r + 1] = acc[tb][nb][r + 1] + b.y;
          y[tb][nb][r + 2] = acc[tb][nb][r + 2] + b.z;
          y[tb][nb][r + 3] = acc[tb][nb][r + 3] + b.w;
        }
      }
      if (kv == 0) {
        if (STYLE == 0) {
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              rot_fwd16(y[tb][nb][r], y[tb][nb + 2][r], cs[tb][16 * nb + r]);
        } else {
#pragma unroll
          for (int nb = 0; nb < 4; ++nb)
#pragma unroll
            for (int r = 0; r < 16; r += 2)
              rot_fwd16(y[tb][nb][r], y[tb][nb][r + 1], cs[tb][8 * nb + r / 2]);
        }
        // coefficient registers are free again: next tile's strip pairs
        load_cs_strip(t_next[tb], cs[tb]);
      }
    }
    // Stores go through the wave's LDS staging buffer one 32-channel block at a
    // time: lane (row, g) writes its 16 channels of token row, then lane j
    // stores bytes 16*(j%4) .. +16 of the 64-byte segment of token j/4 (+16q).
    uint16_t* ys = Ys[wave];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
#pragma unroll
      for (int tb = 0; tb < TB; ++tb) {
        uint4 w0, w1;
        w0.x = pack2(y[tb][nb][0], y[tb][nb][1]);   w0.y = pack2(y[tb][nb][2], y[tb][nb][3]);
        w0.z = pack2(y[tb][nb][4], y[tb][nb][5]);   w0.w = pack2(y[tb][nb][6], y[tb][nb][7]);
        w1.x = pack2(y[tb][nb][8], y[tb][nb][9]);   w1.y = pack2(y[tb][nb][10], y[tb][nb][11]);
        w1.z = pack2(y[tb][nb][12], y[tb][nb][13]); w1.w = pack2(y[tb][nb][14], y[tb][nb][15]);
        uint16_t* yrow = ys + (32 * tb + row) * 32 + 16 * g;
        *reinterpret_cast<uint4*>(yrow) = w0;
        *reinterpret_cast<uint4*>(yrow + 8) = w1;
      }
#pragma unroll
      for (int q = 0; q < 2 * TB; ++q) {
        const int tk = 16 * q + (lane >> 2);        // token within the wave's rows
        const int c = lane & 3;                     // 16-byte chunk of the segment
        const uint4 v = *reinterpret_cast<const uint4*>(ys + tk * 32 + 8 * c);
        const int tb = tk / 32;
        const int64_t tok = tt + 32 * (TB * wave + tb) + (tk % 32);
        int64_t dst = tok;
        if (SLOTS) {
          // the slot of token tk was loaded by lane tk % 32 (either half)
          int64_t mine = orow[0];
#pragma unroll
          for (int u = 1; u < TB; ++u)
            if (u == tb) mine = orow[u];
          dst = (int64_t)__shfl((long long)mine, tk % 32, 64);
        }
        const bool store = tok < t_end && (!SLOTS || (dst >= 0 && dst < a.tgt_rows));
        if (store) *reinterpret_cast<uint4*>(out + dst * D + 32 * nb + 8 * c) = v;
      }
    }
  }
}

template <int K, int STYLE, int NW, int TB, int PD>
hipError_t launch_shape(const MapArgs& a, hipStream_t stream) {
  const int64_t n_ranges = ((int64_t)a.T + a.range_len - 1) / a.range_len;
  const int64_t items64 = n_ranges * a.nl * a.H * 2;
  if (items64 > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const unsigned items = (unsigned)items64;
  if (a.slots != nullptr)
    hipLaunchKernelGGL((map_w_kernel<K, STYLE, true, NW, TB, PD>), dim3(items), dim3(NW * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((map_w_kernel<K, STYLE, false, NW, TB, PD>), dim3(items), dim3(NW * 64), 0, stream, a);
  return hipGetLastError();
}

template <int K, int STYLE>
hipError_t launch_k(const MapArgs& a, hipStream_t stream) {
  // workgroup shape: 8 waves x 32 tokens (two waves per SIMD) or 4 waves x 64
  // tokens (one wave per SIMD, each W^T fragment feeds two MFMAs)
  if (a.wave_tokens == 64)
    return a.prefetch == 2 ? launch_shape<K, STYLE, 4, 2, 2>(a, stream)
                           : launch_shape<K, STYLE, 4, 2, 1>(a, stream);
  return launch_shape<K, STYLE, 8, 1, 1>(a, stream);
}

template <int K>
hipError_t launch_style(const MapArgs& a, int style, hipStream_t stream) {
  return style == 0 ? launch_k<K, 0>(a, stream) : launch_k<K, 1>(a, stream);
}

}  // namespace

bool map_w_supported(int dtype, int d, int k) { return dtype == 0 && d == 128 && k >= 1 && k <= 4; }

size_t packed_w_bytes(int L_t, int H, int k) { return (size_t)L_t * H * 2 * D * k * D * 2; }

hipError_t launch_pack_w(const MapArgs& a, void* wp, hipStream_t stream) {
  const int64_t threads = (int64_t)a.nl * a.H * 2 * (a.k * D / 8) * (D / 8);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  const uint16_t* wk = reinterpret_cast<const uint16_t*>(a.wk);
  const uint16_t* wv = reinterpret_cast<const uint16_t*>(a.wv);
  uint16_t* out = reinterpret_cast<uint16_t*>(wp);
  switch (a.k) {
    case 1: hipLaunchKernelGGL(pack_w_kernel<1>, dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    case 2: hipLaunchKernelGGL(pack_w_kernel<2>, dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    case 3: hipLaunchKernelGGL(pack_w_kernel<3>, dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    case 4: hipLaunchKernelGGL(pack_w_kernel<4>, dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_map_w(const MapArgs& a, int style, hipStream_t stream) {
  if (a.T == 0 || a.nl == 0) return hipSuccess;
  switch (a.k) {
    case 1: return launch_style<1>(a, style, stream);
    case 2: return launch_style<2>(a, style, stream);
    case 3: return launch_style<3>(a, style, stream);
    case 4: return launch_style<4>(a, style, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kvx
