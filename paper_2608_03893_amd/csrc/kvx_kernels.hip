// HIP kernels of the KV-cache mapper for CDNA4 (gfx950).
//
// Two kernels make one mapping call:
//   rope_table_kernel  cos/sin of every (token, plane) for the source and the
//                      target RoPE (Sec. 3.3), angle p * w_j reduced in float64
//                      and stored as float32 [T][d/2] (cos, sin) pairs;
//   map_kernel         for one (target layer, head, K|V) task and one tile of
//                      64 tokens: gather the k selected source layers, strip
//                      the source RoPE from keys (Sec. 3.3) into an LDS operand
//                      tile, contract with the layer's [k*d, d] map on the
//                      matrix cores (Eq. ridge_kv, Sec. 3.1), add the bias in
//                      content space, re-apply the target RoPE and store.
//
// Matrix-core use.  bf16 operands go through v_mfma_f32_32x32x16_bf16 (fp32
// accumulation); fp32 operands through v_mfma_f32_32x32x2_f32.  For both, lane
// L of a wave holds operand row/column (L % 32); the bf16 form gives it the 8
// consecutive reduction indices 8*(L/32) .. 8*(L/32)+7 of a 16-wide step, the
// fp32 form the single index L/32 of a 2-wide step.  Accumulator register r of
// lane L holds output row 8*(r/4) + 4*(L/32) + (r%4), column L % 32.
#include "kvx_internal.h"

#include <type_traits>

namespace kvx {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------- RoPE table

__device__ __forceinline__ uint32_t half2_bits(double c, double s) {
  // (cos, sin) rounded once from float64 to fp16, cos in the low half
  const _Float16 hc = (_Float16)c, hs = (_Float16)s;
  return (uint32_t)__builtin_bit_cast(uint16_t, hc) |
         ((uint32_t)__builtin_bit_cast(uint16_t, hs) << 16);
}

__global__ __launch_bounds__(256) void rope_table_kernel(
    const int32_t* __restrict__ pos, int T, int half, const InvFreq fs,
    const InvFreq ft, int both, float2* __restrict__ cs_src,
    float2* __restrict__ cs_tgt, uint32_t* __restrict__ cs16,
    uint32_t* __restrict__ cs16_tgt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)T * half) return;
  const int t = (int)(i / half);
  const int j = (int)(i - (int64_t)t * half);
  const double p = (double)pos[t];
  double s, c;
  sincos(p * fs.w[j], &s, &c);
  cs_src[i] = make_float2((float)c, (float)s);
  cs16[i] = half2_bits(c, s);
  if (both) {
    sincos(p * ft.w[j], &s, &c);
    cs_tgt[i] = make_float2((float)c, (float)s);
    cs16_tgt[i] = half2_bits(c, s);
  }
}

// ------------------------------------------------------------ element access

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  // round-to-nearest-even conversion of two floats, packed low/high
  __bf16 a = (__bf16)lo;
  __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Load 8 consecutive elements starting at p (16-byte aligned) as floats.
template <bool BF>
__device__ __forceinline__ void load8(const void* p, float (&v)[8]) {
  if constexpr (BF) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    v[0] = bf16_bits_to_f32(u.x & 0xffffu); v[1] = __uint_as_float(u.x & 0xffff0000u);
    v[2] = bf16_bits_to_f32(u.y & 0xffffu); v[3] = __uint_as_float(u.y & 0xffff0000u);
    v[4] = bf16_bits_to_f32(u.z & 0xffffu); v[5] = __uint_as_float(u.z & 0xffff0000u);
    v[6] = bf16_bits_to_f32(u.w & 0xffffu); v[7] = __uint_as_float(u.w & 0xffff0000u);
  } else {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

// Store 8 floats to p (16-byte aligned), rounding to bf16 when BF.
template <bool BF>
__device__ __forceinline__ void store8(void* p, const float (&v)[8]) {
  if constexpr (BF) {
    uint4 u;
    u.x = pack_bf16x2(v[0], v[1]);
    u.y = pack_bf16x2(v[2], v[3]);
    u.z = pack_bf16x2(v[4], v[5]);
    u.w = pack_bf16x2(v[6], v[7]);
    *reinterpret_cast<uint4*>(p) = u;
  } else {
    reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

__device__ __forceinline__ void load_cs8(const float2* p, float (&c)[8], float (&s)[8]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    const float4 f = q[n];
    c[2 * n] = f.x; s[2 * n] = f.y; c[2 * n + 1] = f.z; s[2 * n + 1] = f.w;
  }
}

__device__ __forceinline__ void load_cs4(const float2* p, float (&c)[4], float (&s)[4]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const float4 f = q[n];
    c[2 * n] = f.x; s[2 * n] = f.y; c[2 * n + 1] = f.z; s[2 * n + 1] = f.w;
  }
}

// Rotate plane (u, v) by +a (forward) or -a (inverse) given cos a, sin a.
template <bool INVERSE>
__device__ __forceinline__ void rot(float& u, float& v, float c, float s) {
  const float u0 = u, v0 = v;
  if constexpr (INVERSE) {
    u = u0 * c + v0 * s;
    v = v0 * c - u0 * s;
  } else {
    u = u0 * c - v0 * s;
    v = v0 * c + u0 * s;
  }
}

// ------------------------------------------------------------------ map tile

template <bool BF, int D>
struct Tile {
  using OT = std::conditional_t<BF, uint16_t, float>;  // operand storage type
  static constexpr int BM = 64;                         // tokens per tile
  static constexpr int HALF = D / 2;
  static constexpr int XS = D + (BF ? 8 : 4);           // LDS row stride (elements)
  static constexpr int CS = D + 4;                      // fp32 result stride
  static constexpr int X_BYTES = BM * XS * (int)sizeof(OT);
  static constexpr int W_BYTES = D * XS * (int)sizeof(OT);
  static constexpr int C_BYTES = BM * CS * 4;
  static constexpr int LDS = (X_BYTES + W_BYTES) > C_BYTES ? (X_BYTES + W_BYTES) : C_BYTES;
  static constexpr int MB = BM / 32;                    // 32-row blocks
  static constexpr int NBW = (D / 32) * MB / 4;         // 32-col blocks per wave
  static constexpr int NB_STRIDE = 4 / MB;              // wave's blocks: nb0 + q*NB_STRIDE
};

template <bool BF, int D, int STYLE, bool SLOTS>
__global__ __launch_bounds__(256) void map_kernel(const MapArgs a) {
  using G = Tile<BF, D>;
  using OT = typename G::OT;
  constexpr int BM = G::BM, HALF = G::HALF, XS = G::XS, CS = G::CS;
  __shared__ __attribute__((aligned(16))) unsigned char smem[G::LDS];
  OT* Xs = reinterpret_cast<OT*>(smem);
  OT* Ws = reinterpret_cast<OT*>(smem + G::X_BYTES);
  float* Cs = reinterpret_cast<float*>(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int t0 = blockIdx.x * BM;
  const int task = blockIdx.y;
  const int kv = task & 1;
  const int h = (task >> 1) % a.H;
  const int ll = (task >> 1) / a.H;
  const int l = a.l0 + ll;
  const int64_t T = a.T;
  const int k = a.k;
  const int mb = wave % G::MB;
  const int nb0 = wave / G::MB;

  f32x16_t acc[G::NBW];
#pragma unroll
  for (int q = 0; q < G::NBW; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[q][r] = 0.0f;

  const OT* W = reinterpret_cast<const OT*>(kv ? a.wv : a.wk) +
                ((int64_t)l * a.H + h) * (int64_t)k * D * D;

  for (int i = 0; i < k; ++i) {
    const int s = a.idx[ll * k + i];
    const OT* X = reinterpret_cast<const OT*>(a.src) +
                  (((int64_t)s * 2 + kv) * a.H + h) * T * D;
    // ---- stage the operand tile: gather + inverse RoPE (keys) + round
    if (kv == 0 && STYLE == 0) {
      for (int it = tid; it < BM * (HALF / 8); it += 256) {
        const int r = it / (HALF / 8), g = it % (HALF / 8);
        const int64_t t = t0 + r;
        float u[8], v[8];
        if (t < T) {
          load8<BF>(X + t * D + 8 * g, u);
          load8<BF>(X + t * D + HALF + 8 * g, v);
          float c[8], sn[8];
          load_cs8(a.cs_src + t * HALF + 8 * g, c, sn);
#pragma unroll
          for (int q = 0; q < 8; ++q) rot<true>(u[q], v[q], c[q], sn[q]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) u[q] = v[q] = 0.0f;
        }
        store8<BF>(Xs + r * XS + 8 * g, u);
        store8<BF>(Xs + r * XS + HALF + 8 * g, v);
      }
    } else if (kv == 0) {  // interleaved planes (2j, 2j+1)
      for (int it = tid; it < BM * (D / 8); it += 256) {
        const int r = it / (D / 8), g = it % (D / 8);
        const int64_t t = t0 + r;
        float x[8];
        if (t < T) {
          load8<BF>(X + t * D + 8 * g, x);
          float c[4], sn[4];
          load_cs4(a.cs_src + t * HALF + 4 * g, c, sn);
#pragma unroll
          for (int q = 0; q < 4; ++q) rot<true>(x[2 * q], x[2 * q + 1], c[q], sn[q]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) x[q] = 0.0f;
        }
        store8<BF>(Xs + r * XS + 8 * g, x);
      }
    } else {  // values: plain gather
      for (int it = tid; it < BM * (D / 8); it += 256) {
        const int r = it / (D / 8), g = it % (D / 8);
        const int64_t t = t0 + r;
        float x[8];
        if (t < T) {
          load8<BF>(X + t * D + 8 * g, x);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) x[q] = 0.0f;
        }
        store8<BF>(Xs + r * XS + 8 * g, x);
      }
    }
    // ---- stage W block i transposed: Ws[n][kk] = W[i*D + kk][n]
    for (int it = tid; it < D * (D / 8); it += 256) {
      const int kk = it / (D / 8), ng = it % (D / 8);
      const OT* wrow = W + ((int64_t)i * D + kk) * D + 8 * ng;
      if constexpr (BF) {
        const uint4 u = *reinterpret_cast<const uint4*>(wrow);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          Ws[(8 * ng + 2 * q) * XS + kk] = (uint16_t)(w4[q] & 0xffffu);
          Ws[(8 * ng + 2 * q + 1) * XS + kk] = (uint16_t)(w4[q] >> 16);
        }
      } else {
        const float4 p0 = reinterpret_cast<const float4*>(wrow)[0];
        const float4 p1 = reinterpret_cast<const float4*>(wrow)[1];
        const float w8[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
        for (int q = 0; q < 8; ++q) Ws[(8 * ng + q) * XS + kk] = w8[q];
      }
    }
    __syncthreads();
    // ---- contraction on the matrix cores
    const int arow = mb * 32 + (lane & 31);
    if constexpr (BF) {
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const int kof = ks * 16 + 8 * (lane >> 5);
        const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(Xs + arow * XS + kof);
#pragma unroll
        for (int q = 0; q < G::NBW; ++q) {
          const int n = (nb0 + q * G::NB_STRIDE) * 32 + (lane & 31);
          const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(Ws + n * XS + kof);
          acc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[q], 0, 0, 0);
        }
      }
    } else {
#pragma unroll 4
      for (int ks = 0; ks < D / 2; ++ks) {
        const int kof = ks * 2 + (lane >> 5);
        const float av = Xs[arow * XS + kof];
#pragma unroll
        for (int q = 0; q < G::NBW; ++q) {
          const int n = (nb0 + q * G::NB_STRIDE) * 32 + (lane & 31);
          acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, Ws[n * XS + kof], acc[q], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // ---- accumulators to LDS (fp32), then bias + target RoPE + rounded store
#pragma unroll
  for (int q = 0; q < G::NBW; ++q) {
    const int col = (nb0 + q * G::NB_STRIDE) * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = mb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      Cs[row * CS + col] = acc[q][r];
    }
  }
  __syncthreads();

  OT* out = reinterpret_cast<OT*>(a.tgt) + (((int64_t)l * 2 + kv) * a.H + h) * a.tgt_rows * D;
  // NULL bias means zero; K and V biases are independent.
  const OT* bias = reinterpret_cast<const OT*>(kv ? a.bv : a.bk);
  if (bias != nullptr) bias += ((int64_t)l * a.H + h) * D;

  auto out_row = [&](int64_t t) -> int64_t {
    if constexpr (SLOTS) {
      const int64_t sl = a.slots[t];
      return (sl < 0 || sl >= a.tgt_rows) ? -1 : sl;
    } else {
      return t;
    }
  };
  auto bias8 = [&](int c0, float (&b)[8]) {
    if (bias != nullptr) {
      load8<BF>(bias + c0, b);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) b[q] = 0.0f;
    }
  };

  if (kv == 0 && STYLE == 0) {
    for (int it = tid; it < BM * (HALF / 8); it += 256) {
      const int r = it / (HALF / 8), g = it % (HALF / 8);
      const int64_t t = t0 + r;
      if (t >= T) continue;
      const int64_t orow = out_row(t);
      if (orow < 0) continue;
      float u[8], v[8], bu[8], bv[8], c[8], sn[8];
      bias8(8 * g, bu);
      bias8(HALF + 8 * g, bv);
      load_cs8(a.cs_tgt + t * HALF + 8 * g, c, sn);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        u[q] = Cs[r * CS + 8 * g + q] + bu[q];
        v[q] = Cs[r * CS + HALF + 8 * g + q] + bv[q];
        rot<false>(u[q], v[q], c[q], sn[q]);
      }
      store8<BF>(out + orow * D + 8 * g, u);
      store8<BF>(out + orow * D + HALF + 8 * g, v);
    }
  } else {
    for (int it = tid; it < BM * (D / 8); it += 256) {
      const int r = it / (D / 8), g = it % (D / 8);
      const int64_t t = t0 + r;
      if (t >= T) continue;
      const int64_t orow = out_row(t);
      if (orow < 0) continue;
      float x[8], b[8];
      bias8(8 * g, b);
#pragma unroll
      for (int q = 0; q < 8; ++q) x[q] = Cs[r * CS + 8 * g + q] + b[q];
      if (kv == 0) {  // interleaved keys
        float c[4], sn[4];
        load_cs4(a.cs_tgt + t * HALF + 4 * g, c, sn);
#pragma unroll
        for (int q = 0; q < 4; ++q) rot<false>(x[2 * q], x[2 * q + 1], c[q], sn[q]);
      }
      store8<BF>(out + orow * D + 8 * g, x);
    }
  }
}

template <bool BF, int D, int STYLE, bool SLOTS>
hipError_t launch_one(const MapArgs& a, hipStream_t stream) {
  using G = Tile<BF, D>;
  const dim3 grid((unsigned)((a.T + G::BM - 1) / G::BM), (unsigned)(a.nl * a.H * 2));
  hipLaunchKernelGGL((map_kernel<BF, D, STYLE, SLOTS>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <bool BF, int D, int STYLE>
hipError_t launch_style(const MapArgs& a, hipStream_t stream) {
  return a.slots != nullptr ? launch_one<BF, D, STYLE, true>(a, stream)
                            : launch_one<BF, D, STYLE, false>(a, stream);
}

template <bool BF, int D>
hipError_t launch_d(const MapArgs& a, int style, hipStream_t stream) {
  return style == 0 ? launch_style<BF, D, 0>(a, stream) : launch_style<BF, D, 1>(a, stream);
}

}  // namespace

hipError_t launch_rope_tables(const int32_t* positions, int T, int d,
                              const InvFreq& src, const InvFreq& tgt, bool same,
                              float2* cs_src, float2* cs_tgt, void* cs16,
                              void* cs16_tgt, hipStream_t stream) {
  const int half = d / 2;
  const int64_t n = (int64_t)T * half;
  if (n == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks), dim3(256), 0, stream,
                     positions, T, half, src, tgt, same ? 0 : 1, cs_src, cs_tgt,
                     reinterpret_cast<uint32_t*>(cs16), reinterpret_cast<uint32_t*>(cs16_tgt));
  return hipGetLastError();
}

hipError_t launch_map(const MapArgs& a, int dtype, int d, int style, hipStream_t stream) {
  if (a.T == 0 || a.nl == 0) return hipSuccess;
  if (dtype == 0) {
    if (d == 128) return launch_d<true, 128>(a, style, stream);
    if (d == 64) return launch_d<true, 64>(a, style, stream);
  } else if (dtype == 1) {
    if (d == 128) return launch_d<false, 128>(a, style, stream);
    if (d == 64) return launch_d<false, 64>(a, style, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace kvx
