// MLP mapper (Sec. 4.4, the nonlinear substitute for the ridge map): for
// target layer l, KV head h and K|V, a network
//   Linear(k*d, F) -> ReLU -> Linear(F, F) -> ReLU -> Linear(F, d)
// (F = 1024 in the paper's appendix) applied to the ridge map's input features
// (stripped keys or values of the selected source layers, concatenated in list
// order, Sec. 3.2 / 3.3); mapped keys get the target RoPE afterwards.
//
// Inference runs in bf16 with fp32 accumulation: the hidden activations are
// rounded to bf16 after bias and ReLU, as a bf16 network evaluates them.  Per
// target layer the three network layers are three launches of one tiled
// matrix-core product (all 2H networks of the layer in each launch):
//
//   mlp_gemm_kernel<1>  X [T, k*d] x W1^T + b1, ReLU -> H1 [T, F]; the rows of
//                       X are read straight from the stripped key planes (or
//                       the value planes) of the k source layers;
//   mlp_gemm_kernel<2>  H1 x W2^T + b2, ReLU -> H2 [T, F];
//   mlp_gemm_kernel<3>  H2 x W3^T + b3, target RoPE (keys), RNE -> target plane.
//
// Weights are taken in the layout of torch.nn.Linear, [out, in]: every row is
// the reduction vector of one output, which is the operand layout of the
// matrix instructions, so nothing is packed.  The key strip is the cross-head
// form's strip pass (every source key plane once, fp32 coefficients).
//
// Tile: 256 tokens x 256 outputs per workgroup for layers 1 and 2, 512 tokens
// x 128 outputs (the whole head) for layer 3; each of the 4 waves owns 128 x
// 128 outputs as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.  64-wide reduction
// steps in two LDS stages with one barrier per step, loaded by buffer loads
// straight into LDS; the schedule is the one of the cross-head product.
#include "kvx_asm.h"
#include "kvx_internal.h"

#include <type_traits>

namespace kvx {
namespace {

constexpr int D = 128;   // head dimension

template <int LAYER>
struct MlpTile {
  static constexpr int BM = LAYER == 3 ? 512 : 256;   // tokens per tile
  static constexpr int BN = LAYER == 3 ? 128 : 256;   // outputs per tile
  static constexpr int WN = BN / 128;                 // waves along the outputs
  static constexpr int STAGE = (BM + BN) * 128;       // one 64-wide step, bf16
  static constexpr int NT = BM / 32;                  // 1 KB token-row loads per wave per step
  static constexpr int NW = BN / 32;                  // 1 KB weight-row loads per wave per step
  static constexpr int NL = NT + NW;
  static constexpr int EXTRA = LAYER == 1 ? 4 * kMaxMlpK : 0;   // plane table
};

__device__ __forceinline__ void unpack4(const uint2& q, float* f) {
  f[0] = lo_bf16(q.x);
  f[1] = hi_bf16(q.x);
  f[2] = lo_bf16(q.y);
  f[3] = hi_bf16(q.y);
}

template <int LAYER, int STYLE>
__global__ __launch_bounds__(256, 1) void mlp_gemm_kernel(const MlpArgs a) {
  using G = MlpTile<LAYER>;
  constexpr int BM = G::BM, BN = G::BN, WN = G::WN, STAGE = G::STAGE;
  constexpr int NT = G::NT, NW = G::NW, NL = G::NL;
  __shared__ __attribute__((aligned(256))) char smem[2 * STAGE + G::EXTRA];
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_u32(smem));
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int wn = wave % WN, wt = wave / WN;

  // XCD-aware order: an XCD (blockIdx % 8) takes a contiguous range of tiles,
  // output tiles fastest, then token tiles, then networks, so its CUs share
  // token rows and weight rows in their L2.
  const int xcd = blockIdx.x & 7, qx = blockIdx.x >> 3;
  const int id = xcd * a.tiles_per_xcd + qx;
  if (id >= a.tiles_total) return;
  const int ntile = id % a.n_tiles_n;
  const int rest = id / a.n_tiles_n;
  const int ttile = rest % a.n_tiles_t;
  const int g = rest / a.n_tiles_t;   // network of this layer: kv * H + h
  const int kv = g / a.H, h = g - kv * a.H;
  const int T = a.T, F = a.F;
  const int N = LAYER == 3 ? D : F;            // outputs
  const int KR = LAYER == 1 ? a.k * D : F;     // reduction length
  const int t0 = ttile * BM, n0 = ntile * BN;
  const int nsteps = KR / 64;
  const int64_t net = (int64_t)a.l * a.H + h;

  // buffer loads: lane -> row 8j + (lane >> 3) of a 1 KB piece, chunk
  // (lane & 7) ^ (lane >> 3) of the 64-wide step, stored at chunk lane & 7
  const int r8 = lane >> 3, gch = (lane & 7) ^ r8;
  const i32x4_t rw = make_rsrc(a.w[kv] + net * N * KR, (uint32_t)((int64_t)N * KR * 2));
  const uint32_t row_bytes = (uint32_t)(LAYER == 1 ? D * 2 : F * 2);
  uint32_t vo_t[NT], vo_n[NW];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    // (T + 512) * row_bytes < 2^32 (checked on the host): rows past T stay
    // past the end of the range and read as zero
    vo_t[j] = (uint32_t)(t0 + (BM / 4) * wave + 8 * j + r8) * row_bytes + 16u * gch;
  }
#pragma unroll
  for (int j = 0; j < NW; ++j)
    vo_n[j] = (uint32_t)(n0 + (BN / 4) * wave + 8 * j + r8) * (uint32_t)KR * 2u + 16u * gch;

  // token rows: layer 1 reads source plane i = step / 2 (two 64-wide steps
  // per head of 128 channels); layers 2 and 3 read this network's activations
  const uint16_t* pbase = LAYER == 1 ? (kv ? a.src : a.xs) : a.act_in + (int64_t)g * T * F;
  const int64_t pstride = (int64_t)T * D;
  const uint32_t prange = (uint32_t)(LAYER == 1 ? pstride * 2 : (int64_t)T * F * 2);
  const uint32_t tab = lds0 + 2 * STAGE;   // layer 1: plane number of each selected layer
  if constexpr (LAYER == 1) {
    if (threadIdx.x < a.k) {
      const int s = a.src_l[threadIdx.x];
      reinterpret_cast<uint32_t*>(smem + 2 * STAGE)[threadIdx.x] =
          (uint32_t)(kv ? (s * 2 + 1) * a.H + h : s * a.H + h);
    }
    __syncthreads();
  }
  auto plane_rsrc = [&](uint32_t pl) __attribute__((always_inline)) {
    return make_rsrc(pbase + (int64_t)pl * pstride, prange);
  };
  i32x4_t rt;
  if constexpr (LAYER == 1) rt = plane_rsrc(reinterpret_cast<const uint32_t*>(smem + 2 * STAGE)[0]);
  else rt = make_rsrc(pbase, prange);
  // soffset of step s within a token row
  auto so_t_of = [&](int s) __attribute__((always_inline)) {
    return (uint32_t)(LAYER == 1 ? (s & 1) * 128 : s * 128);
  };

  auto load_step = [&](int s, int st) __attribute__((always_inline)) {
    const uint32_t so_t = __builtin_amdgcn_readfirstlane(so_t_of(s));
    const uint32_t so_n = __builtin_amdgcn_readfirstlane((uint32_t)(s * 128));
    const uint32_t base = lds0 + (uint32_t)(st * STAGE);
#pragma unroll
    for (int j = 0; j < NT; ++j) dma16(base + (uint32_t)(32 * BM * wave + 1024 * j), vo_t[j], rt, so_t);
#pragma unroll
    for (int j = 0; j < NW; ++j)
      dma16(base + (uint32_t)(BM * 128 + 32 * BN * wave + 1024 * j), vo_n[j], rw, so_n);
  };

  f32x4_t acc[8][8];
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int y = 0; y < 8; ++y) {
      acc[x][y] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
      asm volatile("" : "+a"(acc[x][y]));
    }

  // fragment addresses: row R, 16-byte chunk q stored at q ^ (R & 7); half hh
  // of a step is chunks 4 hh .. 4 hh + 3
  const int fr_row = lane & 15, fr_q = lane >> 4;
  uint32_t rd_t[2], rd_n[2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const uint32_t ch = (uint32_t)(((4 * hh + fr_q) ^ (fr_row & 7)) * 16);
    rd_t[hh] = lds0 + (uint32_t)((128 * wt + fr_row) * 128) + ch;
    rd_n[hh] = lds0 + (uint32_t)(BM * 128 + (128 * wn + fr_row) * 128) + ch;
  }
  u32x4_t f0[16], f1[16];   // 0..7 token blocks, 8..15 weight blocks
  auto read_frag = [&](u32x4_t* f, int i, uint32_t stage_off, int hh) __attribute__((always_inline)) {
    if (i < 8) lds_read<0>(f[i], rd_t[hh] + stage_off + (uint32_t)(2048 * i));
    else lds_read<0>(f[i], rd_n[hh] + stage_off + (uint32_t)(2048 * (i - 8)));
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

  // prologue: step 0 into stage 0, step 1 into stage 1, half-0 fragments of step 0
  load_step(0, 0);
  vm_wait<0>();
  __syncthreads();
  if (nsteps > 1) load_step(1, 1);
#pragma unroll
  for (int i = 0; i < 16; ++i) read_frag(f0, i, 0u, 0);

  // One reduction step (RD: read the next step's half-0 fragments; LD: load
  // step s + 2), instantiated three times so the loop body is straight-line.
  auto step = [&](int s, auto RD, auto LD) __attribute__((always_inline)) {
    const uint32_t cur = (uint32_t)((s & 1) * STAGE), nxt = (uint32_t)(((s + 1) & 1) * STAGE);
    wait_all(f0);
    uint32_t pl = 0;   // layer 1: plane of step s + 2, read now, used after the barrier
    if constexpr (LAYER == 1 && decltype(LD)::value)
      asm volatile("ds_read_b32 %0, %1" : "=v"(pl) : "v"(tab + 4u * (uint32_t)((s + 2) >> 1)));
#pragma unroll
    for (int m = 0; m < 64; ++m) {
      mfma(acc[m >> 3][m & 7], f0[8 + (m >> 3)], f0[m & 7]);
      if (m % 2 == 0 && m < 32) read_frag(f1, m / 2, cur, 1);
    }
    wait_all(f1);   // also covers the plane read
    asm volatile("" : "+v"(pl));
    vm_wait<0>();
    __syncthreads();
    i32x4_t rt2 = rt;
    uint32_t so_t2 = 0, so_n2 = 0;
    if constexpr (decltype(LD)::value) {
      if constexpr (LAYER == 1) rt2 = plane_rsrc((uint32_t)__builtin_amdgcn_readfirstlane(pl));
      so_t2 = __builtin_amdgcn_readfirstlane(so_t_of(s + 2));
      so_n2 = __builtin_amdgcn_readfirstlane((uint32_t)((s + 2) * 128));
      // five wait states between these scalar operands and the loads below
      asm volatile("s_nop 4" : : "s"(rt2), "s"(so_t2), "s"(so_n2));
    }
#pragma unroll
    for (int m = 0; m < 64; ++m) {
      mfma(acc[m >> 3][m & 7], f1[8 + (m >> 3)], f1[m & 7]);
      if constexpr (decltype(RD)::value)
        if (m % 4 == 0) read_frag(f0, m / 4, nxt, 0);
      if constexpr (decltype(LD)::value) {
        // the step's NL loads spread over the half: one per EVERY matrix
        // instructions (a wave stalls less on each than when they are bunched)
        constexpr int EVERY = NL <= 16 ? 4 : 3;
        static_assert(NL * EVERY <= 64, "loads of a step must fit in half a step");
        if (m % EVERY == 1) {
          const int j = m / EVERY;
          if (j < NT)
            dma16_near(lds0 + cur + (uint32_t)(32 * BM * wave + 1024 * j), vo_t[j < NT ? j : 0],
                       rt2, so_t2);
          else if (j < NL)
            dma16_near(lds0 + cur + (uint32_t)(BM * 128 + 32 * BN * wave + 1024 * (j - NT)),
                       vo_n[j < NT ? 0 : j - NT], rw, so_n2);
        }
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

  // wait states after the last matrix instruction, tied to every accumulator
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]),
                 "+a"(acc[0][4]), "+a"(acc[0][5]), "+a"(acc[0][6]), "+a"(acc[0][7]));
#pragma unroll
  for (int x = 1; x < 8; ++x)
    asm volatile("" : "+a"(acc[x][0]), "+a"(acc[x][1]), "+a"(acc[x][2]), "+a"(acc[x][3]),
                 "+a"(acc[x][4]), "+a"(acc[x][5]), "+a"(acc[x][6]), "+a"(acc[x][7]));

  // Epilogue.  Block (x, y) of a wave: lane holds outputs 16 x + 4 gq + r
  // (r = 0..3) of its 128 for token 16 y + (lane & 15) of its 128.
  const int gq = lane >> 4;
  const uint16_t* bias = a.b[kv];
  float bv[8][4];
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const int n = n0 + 128 * wn + 16 * x + 4 * gq;
    if (bias != nullptr && n < N) {
      unpack4(*reinterpret_cast<const uint2*>(bias + net * N + n), bv[x]);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) bv[x][r] = 0.f;
    }
  }
  if constexpr (LAYER < 3) {
    uint16_t* out = a.act_out + (int64_t)g * T * F;
#pragma unroll
    for (int y = 0; y < 8; ++y) {
      const int t = t0 + 128 * wt + 16 * y + (lane & 15);
      if (t >= T) continue;
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const int n = n0 + 128 * wn + 16 * x + 4 * gq;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[x][y][r] + bv[x][r], 0.f);
        *reinterpret_cast<uint2*>(out + (int64_t)t * F + n) =
            make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
      }
    }
  } else {
    // the whole head: outputs = channels 0 .. 127 (wn == 0, n0 == 0)
    uint16_t* out = a.tgt + (((int64_t)a.l * 2 + kv) * a.H + h) * T * D;
#pragma unroll
    for (int y = 0; y < 8; ++y) {
      const int t = t0 + 128 * wt + 16 * y + (lane & 15);
      if (t >= T) continue;
      float v[8][4];
#pragma unroll
      for (int x = 0; x < 8; ++x)
#pragma unroll
        for (int r = 0; r < 4; ++r) v[x][r] = acc[x][y][r] + bv[x][r];
      if (kv == 0) {
        const float2* cs = a.cs_tgt + (int64_t)t * (D / 2);
        if (STYLE == 0) {
          // plane j = channel j of the first half: partner 64 channels on,
          // block x + 4, same lane and register
#pragma unroll
          for (int x = 0; x < 4; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float2 w = cs[16 * x + 4 * gq + r];
              const float u0 = v[x][r], v0 = v[x + 4][r];
              v[x][r] = __builtin_fmaf(u0, w.x, -(v0 * w.y));
              v[x + 4][r] = __builtin_fmaf(v0, w.x, u0 * w.y);
            }
        } else {
          // plane j = channels (2j, 2j + 1): registers r and r + 1
#pragma unroll
          for (int x = 0; x < 8; ++x)
#pragma unroll
            for (int r = 0; r < 4; r += 2) {
              const float2 w = cs[(16 * x + 4 * gq + r) >> 1];
              const float u0 = v[x][r], v0 = v[x][r + 1];
              v[x][r] = __builtin_fmaf(u0, w.x, -(v0 * w.y));
              v[x][r + 1] = __builtin_fmaf(v0, w.x, u0 * w.y);
            }
        }
      }
#pragma unroll
      for (int x = 0; x < 8; ++x)
        *reinterpret_cast<uint2*>(out + (int64_t)t * D + 16 * x + 4 * gq) =
            make_uint2(pack2(v[x][0], v[x][1]), pack2(v[x][2], v[x][3]));
    }
  }
}

template <int LAYER>
hipError_t launch_layer(MlpArgs a, int style, hipStream_t stream) {
  using G = MlpTile<LAYER>;
  const int N = LAYER == 3 ? D : a.F;
  a.n_tiles_t = (a.T + G::BM - 1) / G::BM;
  a.n_tiles_n = (N + G::BN - 1) / G::BN;
  const int64_t total = (int64_t)2 * a.H * a.n_tiles_t * a.n_tiles_n;
  if (total > (int64_t)1 << 30) return hipErrorInvalidValue;
  a.tiles_total = (int)total;
  a.tiles_per_xcd = (int)((total + 7) / 8);
  const dim3 grid((unsigned)(8 * a.tiles_per_xcd));
  if (style == 0)
    hipLaunchKernelGGL((mlp_gemm_kernel<LAYER, 0>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((mlp_gemm_kernel<LAYER, 1>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_mlp_layer(const MlpArgs& a, int layer, int style, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  switch (layer) {
    case 1: return launch_layer<1>(a, style, stream);
    case 2: return launch_layer<2>(a, style, stream);
    case 3: return launch_layer<3>(a, style, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kvx
