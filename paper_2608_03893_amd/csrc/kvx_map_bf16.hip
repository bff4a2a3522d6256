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
constexpr int NW = 8;                  // waves per workgroup
constexpr int TB = 1;                  // 32-token blocks per wave
constexpr int NT = NW * 64;            // threads per workgroup
constexpr int TILE = NW * 32 * TB;     // tokens per workgroup step

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

// Stage W^T of one task into LDS with both operand permutations.
template <int K>
__device__ __forceinline__ void stage_wt(uint16_t* Wt, const uint16_t* __restrict__ W, int tid) {
  constexpr int WS = K * D + 8;
  for (int blk = tid; blk < (K * D / 8) * (D / 8); blk += NT) {
    const int rb = blk / (D / 8);  // 8 input rows 8rb .. 8rb+7
    const int cb = blk % (D / 8);  // 8 output columns 8cb .. 8cb+7
    uint4 r[8];
#pragma unroll
    for (int q = 0; q < 8; ++q)
      r[q] = *reinterpret_cast<const uint4*>(W + (int64_t)(8 * rb + q) * D + 8 * cb);
    // input rows -> reduction column (sigma^-1)
    const int i = (8 * rb) / D;
    const int d0 = (8 * rb) % D;
    const int upper = d0 / HALF, dd = d0 % HALF;
    const int g = dd / 32, s = (dd % 32) / 8 + 4 * upper;
    const int kcol = 16 * (8 * i + s) + 8 * g;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      // output column n -> accumulator row (pi^-1)
      const int n = 8 * cb + c;
      const int nb = n / 32, m = n % 32;
      const int rho = 32 * nb + 8 * ((m % 16) / 4) + 4 * (m / 16) + (m % 4);
      uint32_t w4[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t* a0 = reinterpret_cast<const uint32_t*>(&r[2 * p]);
        const uint32_t* a1 = reinterpret_cast<const uint32_t*>(&r[2 * p + 1]);
        const uint32_t e0 = (c & 1) ? (a0[c / 2] >> 16) : (a0[c / 2] & 0xffffu);
        const uint32_t e1 = (c & 1) ? (a1[c / 2] >> 16) : (a1[c / 2] & 0xffffu);
        w4[p] = e0 | (e1 << 16);
      }
      *reinterpret_cast<uint4*>(Wt + rho * WS + kcol) = make_uint4(w4[0], w4[1], w4[2], w4[3]);
    }
  }
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

template <int K, int STYLE, bool SLOTS>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void map_w_kernel(const MapArgs a) {
  constexpr int KD = K * D;
  constexpr int WS = KD + 8;
  __shared__ __attribute__((aligned(16))) uint16_t Wt[D * WS];
  __shared__ __attribute__((aligned(16))) float Bs[D];  // bias, fp32

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
  stage_wt<K>(Wt, reinterpret_cast<const uint16_t*>(kv ? a.wv : a.wk) +
                      ((int64_t)l * a.H + h) * (int64_t)KD * D, tid);
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

  // Token row of this lane in the tile starting at tt, clamped to the range so
  // every load is in bounds and unconditional; a clamped row only feeds its
  // own (discarded) output column of C^T.
  auto lane_row = [&](int64_t tt) -> int64_t {
    const int64_t t = tt + 32 * wave + row;
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

  // Software pipeline: the rows of the next source block are always in flight
  // while the current block is stripped and multiplied.  The coefficient
  // registers hold the strip pairs of the current tile until its last strip,
  // then the epilogue pairs, then the next tile's strip pairs.
  uint4 nxu[4], nxv[4];
  uint32_t cs[32];
  {
    const int64_t t0 = lane_row(t_begin);
    load_block(Xb[0], t0, nxu, nxv);
    if (kv == 0) load_cs_strip(t0, cs);
  }

  for (int64_t tt = t_begin; tt < t_end; tt += TILE) {
    const int64_t t_here = lane_row(tt);
    // the last tile prefetches (and discards) its own rows again
    const int64_t t_next = lane_row(tt + TILE < t_end ? tt + TILE : tt);
    const int64_t tok = tt + 32 * wave + row;
    const bool ok = tok < t_end;
    int64_t orow = tok;
    if (SLOTS) orow = a.slots[t_here];

    f32x16_t acc[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[nb][r] = 0.0f;

#pragma unroll
    for (int i = 0; i < K; ++i) {
      uint4 xu[4], xv[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        xu[s] = nxu[s];
        xv[s] = nxv[s];
      }
      if (i + 1 < K) load_block(Xb[i + 1], t_here, nxu, nxv);
      __builtin_amdgcn_sched_barrier(0);
      // ---- strip the source RoPE (keys)
      if (kv == 0) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (STYLE == 0) {
            strip_halfsplit(xu[s], xv[s], &cs[8 * s]);
          } else {
            strip_interleaved(xu[s], &cs[4 * s]);
            strip_interleaved(xv[s], &cs[16 + 4 * s]);
          }
        }
        if (i + 1 == K) load_cs_out(t_here, cs);
      }
      if (i + 1 == K) load_block(Xb[0], t_next, nxu, nxv);
      __builtin_amdgcn_sched_barrier(0);
      // ---- contraction: 8 reduction steps of 16
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int kof = 16 * (8 * i + s) + 8 * g;
        bf16x8_t wa[4];
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          wa[nb] = *reinterpret_cast<const bf16x8_t*>(Wt + (32 * nb + row) * WS + kof);
        const bf16x8_t xb = as_bf16x8(s < 4 ? xu[s] : xv[s - 4]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[nb], xb, acc[nb], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue: bias, target RoPE, round, store (channel 32nb + 16g + r)
    float y[4][16];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
#pragma unroll
      for (int r = 0; r < 16; r += 4) {
        const float4 b = *reinterpret_cast<const float4*>(&Bs[32 * nb + 16 * g + r]);
        y[nb][r] = acc[nb][r] + b.x;
        y[nb][r + 1] = acc[nb][r + 1] + b.y;
        y[nb][r + 2] = acc[nb][r + 2] + b.z;
        y[nb][r + 3] = acc[nb][r + 3] + b.w;
      }
    }
    if (kv == 0) {
      if (STYLE == 0) {
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) rot_fwd16(y[nb][r], y[nb + 2][r], cs[16 * nb + r]);
      } else {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
          for (int r = 0; r < 16; r += 2) rot_fwd16(y[nb][r], y[nb][r + 1], cs[8 * nb + r / 2]);
      }
      // coefficient registers are free again: next tile's strip pairs
      load_cs_strip(t_next, cs);
    }
    const bool store = ok && (!SLOTS || (orow >= 0 && orow < a.tgt_rows));
    if (store) {
      uint16_t* o = out + orow * D + 16 * g;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        uint4 w0, w1;
        w0.x = pack2(y[nb][0], y[nb][1]);   w0.y = pack2(y[nb][2], y[nb][3]);
        w0.z = pack2(y[nb][4], y[nb][5]);   w0.w = pack2(y[nb][6], y[nb][7]);
        w1.x = pack2(y[nb][8], y[nb][9]);   w1.y = pack2(y[nb][10], y[nb][11]);
        w1.z = pack2(y[nb][12], y[nb][13]); w1.w = pack2(y[nb][14], y[nb][15]);
        *reinterpret_cast<uint4*>(o + 32 * nb) = w0;
        *reinterpret_cast<uint4*>(o + 32 * nb + 8) = w1;
      }
    }
  }
}

template <int K, int STYLE>
hipError_t launch_k(const MapArgs& a, hipStream_t stream) {
  const int64_t n_ranges = ((int64_t)a.T + a.range_len - 1) / a.range_len;
  const int64_t items64 = n_ranges * a.nl * a.H * 2;
  if (items64 > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const unsigned items = (unsigned)items64;
  if (a.slots != nullptr)
    hipLaunchKernelGGL((map_w_kernel<K, STYLE, true>), dim3(items), dim3(NT), 0, stream, a);
  else
    hipLaunchKernelGGL((map_w_kernel<K, STYLE, false>), dim3(items), dim3(NT), 0, stream, a);
  return hipGetLastError();
}

template <int K>
hipError_t launch_style(const MapArgs& a, int style, hipStream_t stream) {
  return style == 0 ? launch_k<K, 0>(a, stream) : launch_k<K, 1>(a, stream);
}

}  // namespace

bool map_w_supported(int dtype, int d, int k) { return dtype == 0 && d == 128 && k >= 1 && k <= 4; }

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
