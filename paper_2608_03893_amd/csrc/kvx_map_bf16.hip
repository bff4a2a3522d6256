// W-stationary map kernel for bf16 caches with head dimension 128 and k <= 4.
//
// One workgroup owns one (target layer, head, K|V) task and a contiguous token
// range.  It stages the task's map W^T ([128 output channels] x [k*128 input
// features], bf16) once into LDS and then streams the range in tiles, each
// wave taking TB blocks of 16 tokens:
//
//   1. each lane loads its token's rows of the k selected source layers
//      straight from HBM into registers, one source block ahead of the one
//      being multiplied (no LDS round trip for the cache);
//   2. keys are stripped of the source RoPE in registers (Sec. 3.3), with the
//      tile's cos/sin held as fp16 pairs and consumed by mixed fp16/fp32 FMAs,
//      then rounded once to bf16;
//   3. the contraction runs as C^T = W^T X^T on v_mfma_f32_16x16x32_bf16
//      (Eq. ridge_kv): W^T fragments come from LDS and feed the TB token
//      blocks of the wave, X^T fragments come from registers and feed all
//      eight 16-row output blocks;
//   4. bias, target RoPE and the bf16 rounding happen in registers; each lane
//      stores 8 contiguous output channels per instruction.
//
// Operand layout.  In the 16x16x32 instruction lane L supplies operand row /
// column L % 16 and reduction indices 8*(L/16) .. 8*(L/16)+7 of the 32-wide
// step; accumulator register r of lane L holds output row 4*(L/16) + r and
// column L % 16.  Two permutations, applied once when the map is packed, make
// these positions convenient for a lane with c = L/16:
//   input  sigma: step s (0..3) of a source block, element q maps to channel
//          64*(s/2) + 32*(s%2) + 8c + q.  For every s the four lanes of a
//          token read 64 contiguous bytes, and steps s and s+2 hold channels
//          j and j+64, so each RoPE plane (either layout) stays in one lane;
//   output pi: accumulator row 4c + r of the 16-row block b maps to channel
//          32*(b/2) + 8c + 4*(b%2) + r, so the lane holds channels
//          32x + 8c .. 32x + 8c + 7 for x = 0..3: four 16-byte stores, and
//          the four lanes of a token cover 64 contiguous bytes each time.
// A reduction is invariant under a common permutation of its index, and the
// output permutation is undone by where each lane stores.  The strip and the
// target rotation touch the same 16 planes of a token in a lane, so with equal
// RoPE on both sides the coefficients are loaded once per tile.
#include "kvx_internal.h"

#include <hip/hip_fp16.h>

namespace kvx {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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

// Forward rotation of plane (u, v) by the angle whose (cos, sin) is cs.
__device__ __forceinline__ void rot_fwd16(float& u, float& v, uint32_t cs) {
  const __half2 h = __builtin_bit_cast(__half2, cs);
  const float c = __low2float(h), s = __high2float(h);
  const float u0 = u, v0 = v;
  u = __builtin_fmaf(u0, c, -__builtin_fmaf(v0, s, 0.0f));
  v = __builtin_fmaf(v0, c, __builtin_fmaf(u0, s, 0.0f));
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

// ------------------------------------------------------------ packed map image
// For one task the LDS image of W^T is dense: [128 accumulator rows rho][k*128
// reduction columns kappa] bf16.  Row rho = 16b + 4c + r holds output channel
// pi(rho); column kappa = 32*(4i + s) + 8c' + q holds input feature
// 128i + sigma(s, c', q).  Each 16-byte chunk u = kappa / 8 of row rho is
// stored at chunk position u ^ (rho & 15), so the 16 rows read by one MFMA
// fragment load fall on distinct LDS banks.  pack_w_kernel writes this image
// to global memory once per call; workgroups copy it to LDS as is.
__device__ __forceinline__ int out_row(int n) {   // output channel -> rho
  const int b = 2 * (n / 32) + (n % 8) / 4;
  const int c = (n % 32) / 8;
  return 16 * b + 4 * c + (n % 4);
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
  // input rows -> reduction chunk (sigma^-1): channel d0 + q of source block i
  const int i = (8 * rb) / D;
  const int d0 = (8 * rb) % D;
  const int s = 2 * (d0 / HALF) + (d0 % HALF) / 32;
  const int cin = (d0 % 32) / 8;
  const int chunk = 4 * (4 * i + s) + cin;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int rho = out_row(8 * cb + c);
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

// ------------------------------------------------------------------ the kernel
// NW waves per workgroup, each owning TB 16-token blocks of every tile.
template <int K, int STYLE, bool SLOTS, int NW, int TB>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4)))
void map_w_kernel(const MapArgs a) {
  constexpr int KD = K * D;
  constexpr int NT = NW * 64;
  constexpr int TILE = NW * 16 * TB;
  __shared__ __attribute__((aligned(16))) uint16_t Wt[D * KD];
  __shared__ __attribute__((aligned(16))) float Bs[D];  // bias, fp32, by output channel

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c = lane >> 4;     // 8-element chunk of the 32-wide reduction step
  const int row = lane & 15;   // token within a 16-token block

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
  const bool same_rope = cs_s == cs_t;

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
    const int64_t t = tt + 16 * (TB * wave + tb) + row;
    return t < t_end ? t : t_end - 1;
  };
  // The four reduction steps of one source row: channels sigma(s, c, 0..7).
  auto load_block = [&](const uint16_t* X, int64_t t, uint4 (&x)[4]) {
    const uint16_t* p = X + t * D + 8 * c;
#pragma unroll
    for (int s = 0; s < 4; ++s) x[s] = *reinterpret_cast<const uint4*>(p + 64 * (s / 2) + 32 * (s % 2));
  };
  // fp16 (cos, sin) pairs of the 16 planes this lane touches:
  // half-split planes 8c .. 8c+7 and 32+8c .. 32+8c+7 (cs[8x + q]);
  // interleaved planes 16x + 4c .. 16x + 4c + 3 for x = 0..3 (cs[4x + q]).
  auto load_cs = [&](const uint32_t* table, int64_t t, uint32_t (&cs)[16]) {
    const uint32_t* p = table + t * HALF;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int j0 = (STYLE == 0) ? 32 * (v / 2) + 8 * c + 4 * (v % 2) : 16 * v + 4 * c;
      const uint4 c4 = *reinterpret_cast<const uint4*>(p + j0);
      cs[4 * v] = c4.x; cs[4 * v + 1] = c4.y; cs[4 * v + 2] = c4.z; cs[4 * v + 3] = c4.w;
    }
  };

  // Software pipeline: the rows of the next source block are always in flight
  // while the current block is stripped and multiplied.  The coefficient
  // registers hold the strip pairs of the current tile, which are also the
  // target pairs when both sides share a RoPE (otherwise the target pairs are
  // loaded after the last strip), then the next tile's strip pairs.
  uint4 nx[TB][4];
  uint32_t cs[TB][16];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    const int64_t t0 = lane_row(t_begin, tb);
    load_block(Xb[0], t0, nx[tb]);
    if (kv == 0) load_cs(cs_s, t0, cs[tb]);
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
      orow[tb] = SLOTS ? (int64_t)a.slots[t_here[tb]] : tt + 16 * (TB * wave + tb) + row;
    }

    f32x4_t acc[TB][8];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
#pragma unroll
      for (int b = 0; b < 8; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[tb][b][r] = 0.0f;

#pragma unroll
    for (int i = 0; i < K; ++i) {
      uint4 x[TB][4];
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
#pragma unroll
        for (int s = 0; s < 4; ++s) x[tb][s] = nx[tb][s];
      if (i + 1 < K) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) load_block(Xb[i + 1], t_here[tb], nx[tb]);
      }
      __builtin_amdgcn_sched_barrier(0);
      // ---- strip the source RoPE (keys)
      if (kv == 0) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          if (STYLE == 0) {
            strip_halfsplit(x[tb][0], x[tb][2], &cs[tb][0]);
            strip_halfsplit(x[tb][1], x[tb][3], &cs[tb][8]);
          } else {
#pragma unroll
            for (int s = 0; s < 4; ++s) strip_interleaved(x[tb][s], &cs[tb][4 * s]);
          }
        }
        if (i + 1 == K && !same_rope) {
#pragma unroll
          for (int tb = 0; tb < TB; ++tb) load_cs(cs_t, t_here[tb], cs[tb]);
        }
      }
      if (i + 1 == K) {
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) load_block(Xb[0], t_next[tb], nx[tb]);
      }
      __builtin_amdgcn_sched_barrier(0);
      // ---- contraction: 4 reduction steps of 32; each W^T fragment feeds
      // the TB token blocks of the wave
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int chunk = (4 * (4 * i + s) + c) ^ row;
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const bf16x8_t wa =
              *reinterpret_cast<const bf16x8_t*>(Wt + (16 * b + row) * KD + 8 * chunk);
#pragma unroll
          for (int tb = 0; tb < TB; ++tb)
            acc[tb][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, as_bf16x8(x[tb][s]), acc[tb][b], 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- epilogue: bias, target RoPE, round, store.  y[x][e] is channel
    // 32x + 8c + e, held in acc[2x + e/4][e%4].  Loads for the next tile are
    // issued before the stores (the memory counter retires them in order).
    float y[TB][4][8];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const float4 b0 = *reinterpret_cast<const float4*>(&Bs[32 * x + 8 * c]);
        const float4 b1 = *reinterpret_cast<const float4*>(&Bs[32 * x + 8 * c + 4]);
        y[tb][x][0] = acc[tb][2 * x][0] + b0.x;
        y[tb][x][1] = acc[tb][2 * x][1] + b0.y;
        y[tb][x][2] = acc[tb][2 * x][2] + b0.z;
        y[tb][x][3] = acc[tb][2 * x][3] + b0.w;
        y[tb][x][4] = acc[tb][2 * x + 1][0] + b1.x;
        y[tb][x][5] = acc[tb][2 * x + 1][1] + b1.y;
        y[tb][x][6] = acc[tb][2 * x + 1][2] + b1.z;
        y[tb][x][7] = acc[tb][2 * x + 1][3] + b1.w;
      }
      if (kv == 0) {
        if (STYLE == 0) {
#pragma unroll
          for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int e = 0; e < 8; ++e) rot_fwd16(y[tb][x][e], y[tb][x + 2][e], cs[tb][8 * x + e]);
        } else {
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int e = 0; e < 8; e += 2) rot_fwd16(y[tb][x][e], y[tb][x][e + 1], cs[tb][4 * x + e / 2]);
        }
        // coefficient registers are free again: next tile's strip pairs
        load_cs(cs_s, t_next[tb], cs[tb]);
      }
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int64_t tok = tt + 16 * (TB * wave + tb) + row;
      const bool store = tok < t_end && (!SLOTS || (orow[tb] >= 0 && orow[tb] < a.tgt_rows));
      if (store) {
        uint16_t* o = out + orow[tb] * D + 8 * c;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          uint4 w;
          w.x = pack2(y[tb][x][0], y[tb][x][1]);
          w.y = pack2(y[tb][x][2], y[tb][x][3]);
          w.z = pack2(y[tb][x][4], y[tb][x][5]);
          w.w = pack2(y[tb][x][6], y[tb][x][7]);
          *reinterpret_cast<uint4*>(o + 32 * x) = w;
        }
      }
    }
  }
}

template <int K, int STYLE, int NW, int TB>
hipError_t launch_shape(const MapArgs& a, hipStream_t stream) {
  const int64_t n_ranges = ((int64_t)a.T + a.range_len - 1) / a.range_len;
  const int64_t items64 = n_ranges * a.nl * a.H * 2;
  if (items64 > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const unsigned items = (unsigned)items64;
  if (a.slots != nullptr)
    hipLaunchKernelGGL((map_w_kernel<K, STYLE, true, NW, TB>), dim3(items), dim3(NW * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((map_w_kernel<K, STYLE, false, NW, TB>), dim3(items), dim3(NW * 64), 0, stream, a);
  return hipGetLastError();
}

template <int K, int STYLE>
hipError_t launch_k(const MapArgs& a, hipStream_t stream) {
  // workgroup shape: 8 waves x 32 tokens (two waves per SIMD) or 4 waves x 64
  // tokens (one wave per SIMD, each W^T fragment feeds four MFMAs)
  return a.wave_tokens == 64 ? launch_shape<K, STYLE, 4, 4>(a, stream)
                             : launch_shape<K, STYLE, 8, 2>(a, stream);
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
    case 1: hipLaunchKernelGGL((pack_w_kernel<1>), dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    case 2: hipLaunchKernelGGL((pack_w_kernel<2>), dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    case 3: hipLaunchKernelGGL((pack_w_kernel<3>), dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
    case 4: hipLaunchKernelGGL((pack_w_kernel<4>), dim3(blocks), dim3(256), 0, stream, wk, wv, out, a.l0, a.nl, a.H); break;
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
