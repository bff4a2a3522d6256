// Cross-head map (bf16, head dimension 64 or 128): Eq. ridge_kv with the
// features of Sec. 3.2, where the input of every target head concatenates all
// KV heads of each selected source layer.  Per target layer and K|V this is one
// dense contraction  Y[T, H_t*d] = X[T, k*H_s*d] * W[k*H_s*d, H_t*d],  large
// enough to be bound by the matrix cores, so it runs as a tiled matrix-core
// product with the RoPE strip done beforehand and the bias, target RoPE and
// rounding fused into the store:
//
//   xhead_strip_kernel  keys of every source layer and head, stripped of the
//                       source RoPE (Sec. 3.3) and rounded once to bf16, into
//                       the workspace (each source row is an input of about
//                       L_t*k/L_s target layers; stripping it once costs one
//                       read and one write of the key planes, and one read of
//                       the RoPE table);
//   xhead_pack_kernel   W^{l,h} [k*H_s*d, d] -> per (l, K|V) rows n = h*d + c
//                       of length k*H_s*d (the contraction index contiguous),
//                       in the order the product kernel's lanes hold outputs;
//   xhead_gemm_kernel   256 tokens x 256 outputs per workgroup, 64-wide
//                       reduction steps staged in LDS by buffer loads, fp32
//                       accumulation, then bias, target RoPE, RNE, store.
#include "kvx_asm.h"
#include "kvx_internal.h"

#include <algorithm>
#include <type_traits>

namespace kvx {
namespace {

constexpr int XBM = 256;   // tokens per workgroup tile
constexpr int XBN = 256;   // outputs (target head x channel) per workgroup tile
constexpr int XBK = 64;    // reduction step staged per LDS stage
constexpr int XSTAGE = (XBM + XBN) * XBK * 2;   // 64 KB: token rows, then output rows

__device__ __forceinline__ void unpack8(const uint4& q, float* f) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = lo_bf16(w[i]);
    f[2 * i + 1] = hi_bf16(w[i]);
  }
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack2(f[0], f[1]), pack2(f[2], f[3]), pack2(f[4], f[5]), pack2(f[6], f[7]));
}

// ---------------------------------------------------------------------------
// Strip: xs[s][g][t][:] = bf16( R_src(p_t)^-1 K_src[s][g][t][:] ).  One thread
// handles 8 planes of one row: channels (8q + e, d/2 + 8q + e) in the
// half-split layout, (16q + 2e, 16q + 2e + 1) in the interleaved one.
template <int D, int STYLE>
__global__ __launch_bounds__(256) void xhead_strip_kernel(const uint16_t* __restrict__ src,
                                                          const float2* __restrict__ cs,
                                                          uint16_t* __restrict__ xs, int L_s,
                                                          int H, int T) {
  // thread = (token t, 8 planes q); it loads their (cos, sin) once and strips
  // the row of every (layer, head) key plane, so the table is read once
  constexpr int TPR = D / 16;   // threads per row
  const int i = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (i >= T * TPR) return;     // T * d * 2 < 2^32 (checked on the host)
  const int t = i / TPR, q = i % TPR;
  const float2* c = cs + (int64_t)t * (D / 2) + 8 * q;
  float2 w[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) w[e] = c[e];
  const int o1 = STYLE == 0 ? 8 * q : 16 * q;
  const int o2 = STYLE == 0 ? D / 2 + 8 * q : 16 * q + 8;
  const int64_t row = (int64_t)t * D;
  const int64_t plane = (int64_t)T * D;
  for (int s = 0; s < L_s; ++s) {
    const uint16_t* in = src + (int64_t)s * 2 * H * plane + row;   // key planes of layer s
    uint16_t* out = xs + (int64_t)s * H * plane + row;
    for (int g = 0; g < H; ++g, in += plane, out += plane) {
      float a[8], b[8];
      unpack8(*reinterpret_cast<const uint4*>(in + o1), a);
      unpack8(*reinterpret_cast<const uint4*>(in + o2), b);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // plane e: (u, v) = (a[e], b[e]) half-split; consecutive pairs interleaved
        float& u = STYLE == 0 ? a[e] : (e < 4 ? a[2 * e] : b[2 * e - 8]);
        float& v = STYLE == 0 ? b[e] : (e < 4 ? a[2 * e + 1] : b[2 * e - 7]);
        const float u0 = u, v0 = v;
        u = __builtin_fmaf(u0, w[e].x, v0 * w[e].y);    // inverse rotation: angle -a
        v = __builtin_fmaf(v0, w[e].x, -(u0 * w[e].y));
      }
      *reinterpret_cast<uint4*>(out + o1) = pack8(a);
      *reinterpret_cast<uint4*>(out + o2) = pack8(b);
    }
  }
}

// ---------------------------------------------------------------------------
// Pack.  For output n = h*d + c of target layer l and K|V, row P of the packed
// image holds column n of W^{l,h}, i.e. W[l][h][0 .. F-1][c] with
// F = k*H_s*d.  Within each aligned block of 128 outputs, the row order is the
// one in which the product kernel's lanes hold results: row
// p = 16*nb + 4*g + r holds channel 64*(nb>>2) + 32*((nb>>1)&1) + 8*g +
// 4*(nb&1) + r, so each lane ends up with 8 consecutive outputs from two
// 16-row blocks, and both channels of a RoPE plane in the same lane.
__device__ __forceinline__ int xhead_row_of(int n) {
  const int base = n & ~127, c = n & 127;
  const int nb = 4 * (c >> 6) + 2 * ((c >> 5) & 1) + ((c >> 2) & 1);
  return base + 16 * nb + 4 * ((c >> 3) & 3) + (c & 3);
}

// One workgroup: 64 reduction rows x 64 outputs of one head of (l, K|V).
template <int D>
__global__ __launch_bounds__(256) void xhead_pack_kernel(const uint16_t* __restrict__ wk,
                                                         const uint16_t* __restrict__ wv,
                                                         uint16_t* __restrict__ wp, int H_t,
                                                         int F, int l0) {
  __shared__ uint16_t tile[64][64 + 2];
  const int f0 = blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;            // 64 outputs inside one head (D is 64 or 128)
  const int lk = 2 * l0 + (int)blockIdx.z;   // l * 2 + kv
  const int l = lk >> 1, kv = lk & 1;
  const int h = n0 / D, c0 = n0 - h * D;
  const int N = H_t * D;
  const uint16_t* w = (kv ? wv : wk) + (((int64_t)l * H_t + h) * F) * D;
  // read 64 rows x 64 channels: thread -> row f0 + (tid >> 3) (+32), 8 channels
  for (int rr = threadIdx.x >> 3; rr < 64; rr += 32) {
    const int c8 = (threadIdx.x & 7) * 8;
    const uint4 v = *reinterpret_cast<const uint4*>(w + (int64_t)(f0 + rr) * D + c0 + c8);
    const uint32_t x[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tile[rr][c8 + 2 * e] = (uint16_t)(x[e] & 0xffffu);
      tile[rr][c8 + 2 * e + 1] = (uint16_t)(x[e] >> 16);
    }
  }
  __syncthreads();
  // write 64 packed rows x 64 reduction values: thread -> output column, 8 values
  uint16_t* dst = wp + (int64_t)lk * N * F;
  for (int cc = threadIdx.x >> 3; cc < 64; cc += 32) {
    const int f8 = (threadIdx.x & 7) * 8;
    uint32_t x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      x[e] = (uint32_t)tile[f8 + 2 * e][cc] | ((uint32_t)tile[f8 + 2 * e + 1][cc] << 16);
    const int P = xhead_row_of(n0 + cc);
    *reinterpret_cast<uint4*>(dst + (int64_t)P * F + f0 + f8) = make_uint4(x[0], x[1], x[2], x[3]);
  }
}

// ---------------------------------------------------------------------------
// Product.  Workgroup: 4 waves; wave (wn, wt) = (wave & 1, wave >> 1) owns
// outputs [128 wn, +128) x tokens [128 wt, +128) of the tile: 8 x 8 blocks of
// v_mfma_f32_16x16x32_bf16 (A = packed map rows, B = token rows), 256
// accumulator registers.  LDS stage = token rows [256][64] then packed rows
// [256][64], 128 bytes per row, 16-byte chunk q of row R stored at position
// q ^ (R & 7) so that the fragment reads of 8 consecutive lanes hit distinct
// banks.  Two stages and one barrier per step, in its middle: each half of a
// step runs its 64 matrix instructions on fragments read during the previous
// half; after the barrier the stage of step s is free and step s + 2 is
// loaded into it (one load per four matrix instructions), with a full step to
// land before the barrier that needs it.
template <int D, int STYLE>
__global__ __launch_bounds__(256, 1) void xhead_gemm_kernel(const XArgs a) {
  // two stages, then this target layer's source-layer indices (one byte each)
  __shared__ __attribute__((aligned(256))) char smem[2 * XSTAGE + kMaxIdx];
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_u32(smem));
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int wn = wave & 1, wt = wave >> 1;

  // XCD-aware order: the workgroups of one XCD (blockIdx % 8) take a
  // contiguous range of tiles, output tiles fastest, so the CUs of an XCD share
  // token rows and packed rows in their L2.
  const int xcd = blockIdx.x & 7, qx = blockIdx.x >> 3;
  const int id = xcd * a.tiles_per_xcd + qx;
  if (id >= a.tiles_total) return;
  const int ntile = id % a.n_tiles_n;
  int rest = id / a.n_tiles_n;
  const int ttile = rest % a.n_tiles_t;
  rest /= a.n_tiles_t;
  const int kv = rest & 1, l = a.l0 + (rest >> 1);
  const int T = a.T, Hs = a.H_s, Ht = a.H_t;
  const int N = Ht * D, F = a.k * Hs * D;
  const int t0 = ttile * XBM, n0 = ntile * XBN;
  const int nsteps = F / XBK;

  // buffer loads: lane -> row 8j + (lane >> 3) of the wave's 64 rows, chunk
  // (lane & 7) ^ (lane >> 3) of the 64-wide step (stored at chunk lane & 7)
  const int r8 = lane >> 3, gch = (lane & 7) ^ r8;
  const int64_t lk = (int64_t)l * 2 + kv;
  const i32x4_t rw = make_rsrc(a.wp + lk * N * F, (uint32_t)((int64_t)N * F * 2));
  uint32_t vo_t[8], vo_n[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = 64 * wave + 8 * j + r8;
    // (T + 256) * d * 2 and (N + 256) * F * 2 are below 2^32 (checked on the host)
    vo_t[j] = (uint32_t)(t0 + row) * (uint32_t)(D * 2) + 16u * gch;
    vo_n[j] = (uint32_t)(n0 + row) * (uint32_t)F * 2u + 16u * gch;
  }
  const uint16_t* plane0 = kv ? a.src : a.xs;
  const int64_t plane_stride = (int64_t)T * D;
  auto load_step = [&](int s, int st) __attribute__((always_inline)) {
    const int f = s * XBK;
    const int b = f / D, c0 = f - b * D;
    const int i = b / Hs, g = b - i * Hs;
    const int src_l = a.idx[(l - a.l0) * a.k + i];
    // key planes: xs[src_l][g]; value planes: src[src_l][1][g]
    const int64_t pl = kv ? ((int64_t)(src_l * 2 + 1) * Hs + g) : ((int64_t)src_l * Hs + g);
    const i32x4_t rt = make_rsrc(plane0 + pl * plane_stride, (uint32_t)(plane_stride * 2));
    const uint32_t so_t = __builtin_amdgcn_readfirstlane((uint32_t)(c0 * 2));
    const uint32_t so_n = __builtin_amdgcn_readfirstlane((uint32_t)(f * 2));
    const uint32_t base = lds0 + (uint32_t)(st * XSTAGE);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      dma16(base + (uint32_t)(8192 * wave + 1024 * j), vo_t[j], rt, so_t);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      dma16(base + (uint32_t)(XBM * 128 + 8192 * wave + 1024 * j), vo_n[j], rw, so_n);
  };

  // Accumulators live in AGPRs; every matrix instruction, LDS read and wait of
  // the loop is issued from inline assembly so that the schedule below holds.
  f32x4_t acc[8][8];
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int y = 0; y < 8; ++y) {
      acc[x][y] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
      asm volatile("" : "+a"(acc[x][y]));
    }

  // Fragment read addresses within a stage: row R, 16-byte chunk q stored at
  // q ^ (R & 7); half h of a step is chunks 4h .. 4h+3.
  const int fr_row = lane & 15, fr_q = lane >> 4;
  uint32_t rd_t[2], rd_n[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t ch = (uint32_t)(((4 * h + fr_q) ^ (fr_row & 7)) * 16);
    rd_t[h] = lds0 + (uint32_t)((128 * wt + fr_row) * 128) + ch;
    rd_n[h] = lds0 + (uint32_t)(XBM * 128 + (128 * wn + fr_row) * 128) + ch;
  }
  // fragments of the two halves of a step: X (token rows) 0..7, W (map rows) 0..7
  u32x4_t f0[16], f1[16];
  auto read_frag = [&](u32x4_t* f, int i, uint32_t stage_off, int h) __attribute__((always_inline)) {
    // i < 8: token block i; i >= 8: map block i - 8 (16 rows = 2048 bytes apart)
    if (i < 8) lds_read<0>(f[i], rd_t[h] + stage_off + (uint32_t)(2048 * i));
    else lds_read<0>(f[i], rd_n[h] + stage_off + (uint32_t)(2048 * (i - 8)));
  };
  auto pin8 = [&](u32x4_t* f) __attribute__((always_inline)) {
    asm volatile("" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]),
                 "+v"(f[6]), "+v"(f[7]));
  };
  auto wait_all = [&](u32x4_t* f) __attribute__((always_inline)) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    pin8(f);
    pin8(f + 8);
  };
  auto mfma = [&](f32x4_t& c, const u32x4_t& w, const u32x4_t& xt) __attribute__((always_inline)) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(w), "v"(xt));
  };

  // this layer's index list into LDS (read once per step below, far ahead of use)
  for (int i = threadIdx.x; i < a.k; i += 256)
    reinterpret_cast<uint8_t*>(smem + 2 * XSTAGE)[i] = a.idx[(l - a.l0) * a.k + i];
  const uint32_t idx_lds = lds0 + 2 * XSTAGE;
  // (selected layer, source head, channel) of the next step to load: step 2
  int li = 0, lg = 0, lc = 2 * XBK;
  while (lc >= D) {
    lc -= D;
    if (++lg == Hs) {
      lg = 0;
      ++li;
    }
  }

  // prologue: step 0 into stage 0, step 1 into stage 1, fragments of half 0 of step 0
  load_step(0, 0);
  vm_wait<0>();
  __syncthreads();
  if (nsteps > 1) load_step(1, 1);
#pragma unroll
  for (int i = 0; i < 16; ++i) read_frag(f0, i, 0u, 0);

  // One reduction step.  RD: read the next step's half-0 fragments; LD: load
  // step s + 2.  Instantiated three times (steady state, last step but one,
  // last step) so that the loop body is straight-line code.
  auto step = [&](int s, auto RD, auto LD) __attribute__((always_inline)) {
    const uint32_t cur = (uint32_t)((s & 1) * XSTAGE), nxt = (uint32_t)(((s + 1) & 1) * XSTAGE);
    // half 0: the fragments read during the previous half; read half 1's
    // fragments between the first 32 matrix instructions
    wait_all(f0);
    uint32_t sl = 0;   // source layer of step s + 2, read now, used after the barrier
    if constexpr (decltype(LD)::value)
      asm volatile("ds_read_u8 %0, %1" : "=v"(sl) : "v"(idx_lds + (uint32_t)li));
#pragma unroll
    for (int m = 0; m < 64; ++m) {
      mfma(acc[m >> 3][m & 7], f0[8 + (m >> 3)], f0[m & 7]);
      if (m % 2 == 0 && m < 32) read_frag(f1, m / 2, cur, 1);
    }
    // mid-step: half 1 fragments in registers (this wave is done with the
    // current stage); the next step's rows landed (every wave)
    wait_all(f1);   // also covers the index read
    asm volatile("" : "+v"(sl));
    vm_wait<0>();
    __syncthreads();
    // half 1: read the next step's half-0 fragments and load step s + 2 into
    // the stage just released
    i32x4_t rt2 = rw;
    uint32_t so_t2 = 0, so_n2 = 0;
    if constexpr (decltype(LD)::value) {
      const int srcl2 = (int)__builtin_amdgcn_readfirstlane(sl);
      const int64_t pl = kv ? ((int64_t)(srcl2 * 2 + 1) * Hs + lg) : ((int64_t)srcl2 * Hs + lg);
      rt2 = make_rsrc(plane0 + pl * plane_stride, (uint32_t)(plane_stride * 2));
      so_t2 = __builtin_amdgcn_readfirstlane((uint32_t)(lc * 2));
      so_n2 = __builtin_amdgcn_readfirstlane((uint32_t)((s + 2) * XBK * 2));
      lc += XBK;
      if (lc == D) {
        lc = 0;
        if (++lg == Hs) {
          lg = 0;
          ++li;
        }
      }
      // five wait states between these scalar operands and the loads below
      asm volatile("s_nop 4" : : "s"(rt2), "s"(so_t2), "s"(so_n2));
    }
#pragma unroll
    for (int m = 0; m < 64; ++m) {
      mfma(acc[m >> 3][m & 7], f1[8 + (m >> 3)], f1[m & 7]);
      if constexpr (decltype(RD)::value)
        if (m % 4 == 0) read_frag(f0, m / 4, nxt, 0);
      if constexpr (decltype(LD)::value)
        if (m % 4 == 1) {   // one load per four matrix instructions: a single
          const int j = m / 4;   // wave stalls less on each than when they are bunched
          const uint32_t dst =
              lds0 + cur + (uint32_t)((j < 8 ? 0 : XBM * 128) + 8192 * wave + 1024 * (j & 7));
          if (j < 8) dma16_near(dst, vo_t[j & 7], rt2, so_t2);
          else dma16_near(dst, vo_n[j & 7], rw, so_n2);
        }
    }
  };
  int s = 0;
  for (; s + 2 < nsteps; ++s) step(s, std::true_type{}, std::true_type{});
  if (s + 1 < nsteps) {
    step(s, std::true_type{}, std::false_type{});
    ++s;
  }
  step(s, std::false_type{}, std::false_type{});

  // The results are read by vector instructions below: wait states after the
  // last matrix instruction, tied to every accumulator so no read moves above.
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]),
                 "+a"(acc[0][4]), "+a"(acc[0][5]), "+a"(acc[0][6]), "+a"(acc[0][7]));
#pragma unroll
  for (int x = 1; x < 8; ++x)
    asm volatile("" : "+a"(acc[x][0]), "+a"(acc[x][1]), "+a"(acc[x][2]), "+a"(acc[x][3]),
                 "+a"(acc[x][4]), "+a"(acc[x][5]), "+a"(acc[x][6]), "+a"(acc[x][7]));

  // Epilogue.  Lane holds, for token block y, token 128 wt + 16 y + (lane & 15)
  // and, in block x, packed rows 16 x + 4 g + r (g = lane >> 4): channels
  // ch = 64 (x >> 2) + 32 ((x >> 1) & 1) + 8 g + 4 (x & 1) + r of the wave's
  // 128 outputs.  Group (hi, u) = 8 consecutive channels 64 hi + 32 u + 8 g ..
  // from blocks x = 4 hi + 2 u and x + 1.
  const int g = lane >> 4;
  const uint16_t* bias = kv ? a.bv : a.bk;
  float bv[2][2][8];
  int head[2][2], cin[2][2];
  bool nok[2][2];
#pragma unroll
  for (int hi = 0; hi < 2; ++hi)
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int n = n0 + 128 * wn + 64 * hi + 32 * u + 8 * g;
      nok[hi][u] = n < N;
      head[hi][u] = n / D;
      cin[hi][u] = n - head[hi][u] * D;
      if (bias != nullptr && nok[hi][u]) {
        unpack8(*reinterpret_cast<const uint4*>(bias + ((int64_t)l * Ht + head[hi][u]) * D + cin[hi][u]),
                bv[hi][u]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) bv[hi][u][e] = 0.f;
      }
    }
  // dense target: row t of each (layer, K|V, head) plane; slot-addressed
  // target: row slots[t] of a plane of tgt_rows rows, skipped when out of range
  uint16_t* out = a.tgt + lk * (int64_t)Ht * a.tgt_rows * D;
#pragma unroll
  for (int y = 0; y < 8; ++y) {
    const int t = t0 + 128 * wt + 16 * y + (lane & 15);
    if (t >= T) continue;
    const int64_t row = a.slots != nullptr ? (int64_t)a.slots[t] : (int64_t)t;
    if (row < 0 || row >= a.tgt_rows) continue;
    float v[2][2][8];
#pragma unroll
    for (int hi = 0; hi < 2; ++hi)
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[hi][u][e] = acc[4 * hi + 2 * u + (e >> 2)][y][e & 3] + bv[hi][u][e];
    if (kv == 0) {
      const float2* cs = a.cs_tgt + (int64_t)t * (D / 2);
      if (STYLE == 0) {
        // plane partner: the other half of the head, 64 channels away for
        // d = 128 (group hi ^ 1), 32 for d = 64 (group u ^ 1)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            float& x1 = D == 128 ? v[0][p][e] : v[p][0][e];
            float& x2 = D == 128 ? v[1][p][e] : v[p][1][e];
            const int j = (D == 128 ? cin[0][p] : cin[p][0]) + e;   // plane = channel in the first half
            const float2 w = cs[j];
            const float u0 = x1, v0 = x2;
            x1 = __builtin_fmaf(u0, w.x, -(v0 * w.y));
            x2 = __builtin_fmaf(v0, w.x, u0 * w.y);
          }
      } else {
#pragma unroll
        for (int hi = 0; hi < 2; ++hi)
#pragma unroll
          for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
              const float2 w = cs[(cin[hi][u] + e) >> 1];
              const float u0 = v[hi][u][e], v0 = v[hi][u][e + 1];
              v[hi][u][e] = __builtin_fmaf(u0, w.x, -(v0 * w.y));
              v[hi][u][e + 1] = __builtin_fmaf(v0, w.x, u0 * w.y);
            }
      }
    }
#pragma unroll
    for (int hi = 0; hi < 2; ++hi)
#pragma unroll
      for (int u = 0; u < 2; ++u)
        if (nok[hi][u])
          *reinterpret_cast<uint4*>(out + ((int64_t)head[hi][u] * a.tgt_rows + row) * D + cin[hi][u]) =
              pack8(v[hi][u]);
  }
}

template <int D>
hipError_t launch_all_d(const XArgs& a, int style, bool strip, bool pack, const uint16_t* wk,
                        const uint16_t* wv, const float2* cs_src, hipStream_t stream) {
  const int F = a.k * a.H_s * D, N = a.H_t * D;
  if (strip) {
    const dim3 grid((unsigned)((a.T * (D / 16) + 255) / 256));
    if (style == 0)
      hipLaunchKernelGGL((xhead_strip_kernel<D, 0>), grid, dim3(256), 0, stream, a.src, cs_src,
                         const_cast<uint16_t*>(a.xs), a.L_s, a.H_s, a.T);
    else
      hipLaunchKernelGGL((xhead_strip_kernel<D, 1>), grid, dim3(256), 0, stream, a.src, cs_src,
                         const_cast<uint16_t*>(a.xs), a.L_s, a.H_s, a.T);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  if (pack) {
    hipLaunchKernelGGL((xhead_pack_kernel<D>), dim3(F / 64, N / 64, a.nl * 2), dim3(256), 0,
                       stream, wk, wv, const_cast<uint16_t*>(a.wp), a.H_t, F, a.l0);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  const unsigned grid = (unsigned)(8 * a.tiles_per_xcd);
  if (style == 0)
    hipLaunchKernelGGL((xhead_gemm_kernel<D, 0>), dim3(grid), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((xhead_gemm_kernel<D, 1>), dim3(grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_strip_keys(const uint16_t* src, const float2* cs, uint16_t* xs, int L_s, int H,
                             int T, int d, int style, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  if (d == 128) {
    const dim3 grid((unsigned)((T * (128 / 16) + 255) / 256));
    if (style == 0)
      hipLaunchKernelGGL((xhead_strip_kernel<128, 0>), grid, dim3(256), 0, stream, src, cs, xs, L_s, H, T);
    else
      hipLaunchKernelGGL((xhead_strip_kernel<128, 1>), grid, dim3(256), 0, stream, src, cs, xs, L_s, H, T);
  } else if (d == 64) {
    const dim3 grid((unsigned)((T * (64 / 16) + 255) / 256));
    if (style == 0)
      hipLaunchKernelGGL((xhead_strip_kernel<64, 0>), grid, dim3(256), 0, stream, src, cs, xs, L_s, H, T);
    else
      hipLaunchKernelGGL((xhead_strip_kernel<64, 1>), grid, dim3(256), 0, stream, src, cs, xs, L_s, H, T);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t xhead_strip_bytes(int L_s, int H_s, int T, int d) {
  return ((size_t)L_s * H_s * (size_t)T * d * 2 + 255) / 256 * 256;
}

size_t xhead_packed_bytes(int L_t, int H_s, int H_t, int k, int d) {
  return ((size_t)L_t * 2 * (size_t)H_t * d * (size_t)k * H_s * d * 2 + 255) / 256 * 256;
}

hipError_t launch_xhead(XArgs& a, int d, int style, bool strip, bool pack, const void* wk,
                        const void* wv, const float2* cs_src, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const int N = a.H_t * d;
  a.n_tiles_t = (a.T + XBM - 1) / XBM;
  a.n_tiles_n = (N + XBN - 1) / XBN;
  const int64_t total = (int64_t)a.nl * 2 * a.n_tiles_t * a.n_tiles_n;
  if (total > (int64_t)1 << 30) return hipErrorInvalidValue;
  a.tiles_total = (int)total;
  a.tiles_per_xcd = (int)((total + 7) / 8);
  const auto* k16 = static_cast<const uint16_t*>(wk);
  const auto* v16 = static_cast<const uint16_t*>(wv);
  if (d == 128) return launch_all_d<128>(a, style, strip, pack, k16, v16, cs_src, stream);
  if (d == 64) return launch_all_d<64>(a, style, strip, pack, k16, v16, cs_src, stream);
  return hipErrorInvalidValue;
}

}  // namespace kvx
