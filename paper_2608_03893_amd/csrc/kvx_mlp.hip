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
// Tile: 256 tokens x 256 outputs for layers 1 and 2, 512 tokens x 128 outputs
// (the whole head) for layer 3; each of the 4 waves owns 128 x 128 outputs as
// 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.  Within each 32 outputs the weight
// rows are taken in the order that gives a lane 8 consecutive outputs in
// blocks 2u and 2u + 1, so the epilogue writes 16-byte pieces.  64-wide reduction steps in two
// LDS stages with one barrier per step, loaded by buffer loads straight into
// LDS (the schedule of the cross-head product); one persistent workgroup per
// CU walks a range of tiles.
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

// Persistent: the workgroups of an XCD walk its contiguous range of tiles
// (output tiles fastest, then token tiles, then networks) together, workgroup
// q taking tiles q, q + n, q + 2n, ... of the range (n workgroups per XCD), so
// the tiles in flight at any time are neighbours that share token rows and
// weight rows in the XCD's L2.  The first two steps of the
// next tile are loaded during the last two steps of the current one, and the
// next tile's first fragments are read before the current tile's epilogue, so
// only the epilogue itself sits between the matrix instructions of two tiles.
// A tile's row offsets live in its buffer descriptors (base and range), so the
// per-lane offsets are the same for every tile.
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

  const int xcd = blockIdx.x & 7, qx = blockIdx.x >> 3;
  const int stride = (int)(gridDim.x >> 3);   // workgroups per XCD
  const int xbeg = xcd * a.tiles_per_xcd;
  const int xend = xbeg + a.tiles_per_xcd < a.tiles_total ? xbeg + a.tiles_per_xcd : a.tiles_total;
  const int first = xbeg + qx;
  if (first >= xend) return;

  const int T = a.T, F = a.F;
  const int N = LAYER == 3 ? D : F;            // outputs
  const int KR = LAYER == 1 ? a.k * D : F;     // reduction length
  const int nsteps = KR / 64;
  const uint32_t row_bytes = (uint32_t)(LAYER == 1 ? D * 2 : F * 2);

  // layer 1: the selected source layers (the same for every network of the launch)
  const uint32_t tab = lds0 + 2 * STAGE;
  if constexpr (LAYER == 1) {
    if (threadIdx.x < a.k) reinterpret_cast<uint32_t*>(smem + 2 * STAGE)[threadIdx.x] = (uint32_t)a.src_l[threadIdx.x];
    __syncthreads();
  }

  struct Tile {
    int kv, h, g, t0, n0;
  };
  auto decode = [&](int id) __attribute__((always_inline)) {
    Tile tl;
    const int ntile = id % a.n_tiles_n;
    const int rest = id / a.n_tiles_n;
    tl.g = rest / a.n_tiles_t;   // network of this layer: kv * H + h
    tl.t0 = (rest - tl.g * a.n_tiles_t) * BM;
    tl.n0 = ntile * BN;
    tl.kv = tl.g / a.H;
    tl.h = tl.g - tl.kv * a.H;
    return tl;
  };
  // token rows of the tile's step s (layer 1: source layer sl of step s), and
  // the tile's weight rows
  auto a_rsrc = [&](const Tile& tl, uint32_t sl) __attribute__((always_inline)) {
    const uint16_t* base;
    if constexpr (LAYER == 1) {
      const int64_t pl = tl.kv ? ((int64_t)sl * 2 + 1) * a.H + tl.h : (int64_t)sl * a.H + tl.h;
      base = (tl.kv ? a.src : a.xs) + pl * T * D + (int64_t)tl.t0 * D;
    } else {
      base = a.act_in + ((int64_t)tl.g * T + tl.t0) * F;
    }
    return make_rsrc(base, (uint32_t)(T - tl.t0) * row_bytes);
  };
  auto w_rsrc = [&](const Tile& tl) __attribute__((always_inline)) {
    const int64_t net = (int64_t)a.l * a.H + tl.h;
    return make_rsrc(a.w[tl.kv] + (net * N + tl.n0) * KR, (uint32_t)((int64_t)(N - tl.n0) * KR * 2));
  };
  auto so_t_of = [&](int s) __attribute__((always_inline)) {
    return (uint32_t)(LAYER == 1 ? (s & 1) * 128 : s * 128);
  };

  // buffer loads: lane -> row 8j + (lane >> 3) of a 1 KB piece, chunk
  // (lane & 7) ^ (lane >> 3) of the 64-wide step, stored at chunk lane & 7;
  // rows past the tile's range read as zero
  // (load j of a step adds 8 j rows to the lane's base offset)
  const int r8 = lane >> 3, gch = (lane & 7) ^ r8;
  const uint32_t vt0 = (uint32_t)((BM / 4) * wave + r8) * row_bytes + 16u * gch;
  const uint32_t vn0 = (uint32_t)((BN / 4) * wave + r8) * (uint32_t)KR * 2u + 16u * gch;
  const uint32_t vt_step = 8u * row_bytes, vn_step = 8u * (uint32_t)KR * 2u;

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
  // Weight block i = 2u + b: matrix row m is weight row 32 u + 8 (m / 4) +
  // 4 b + m % 4 of the wave's 128, so that lane group gq (rows 4 gq .. 4 gq + 3
  // of each block) holds outputs 32 u + 8 gq .. 32 u + 8 gq + 7 in blocks 2u
  // and 2u + 1.  32 u adds a multiple of 8 rows: the chunk swizzle is that of
  // the row within its 32.
  const int fr_row = lane & 15, fr_q = lane >> 4;
  uint32_t rd_t[2], rd_n[2][2];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const uint32_t ch = (uint32_t)(((4 * hh + fr_q) ^ (fr_row & 7)) * 16);
    rd_t[hh] = lds0 + (uint32_t)((128 * wt + fr_row) * 128) + ch;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int wr = 8 * (fr_row >> 2) + 4 * b + (fr_row & 3);
      const uint32_t chn = (uint32_t)(((4 * hh + fr_q) ^ (wr & 7)) * 16);
      rd_n[hh][b] = lds0 + (uint32_t)(BM * 128 + (128 * wn + wr) * 128) + chn;
    }
  }
  u32x4_t f0[16], f1[16];   // 0..7 token blocks, 8..15 weight blocks
  auto read_frag = [&](u32x4_t* f, int i, uint32_t stage_off, int hh) __attribute__((always_inline)) {
    if (i < 8) lds_read<0>(f[i], rd_t[hh] + stage_off + (uint32_t)(2048 * i));
    else lds_read<0>(f[i], rd_n[hh][i & 1] + stage_off + (uint32_t)(4096 * ((i - 8) >> 1)));
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

  Tile cur = decode(first);
  // prologue: steps 0 and 1 of the first tile into stages 0 and 1, half-0
  // fragments of step 0
  {
    const uint32_t sl0 = LAYER == 1 ? (uint32_t)a.src_l[0] : 0u;
    const i32x4_t rt = a_rsrc(cur, sl0), rw = w_rsrc(cur);
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const uint32_t so_t = __builtin_amdgcn_readfirstlane(so_t_of(st));
      const uint32_t so_n = (uint32_t)(st * 128);
      const uint32_t base = lds0 + (uint32_t)(st * STAGE);
#pragma unroll
      for (int j = 0; j < NT; ++j)
        dma16(base + (uint32_t)(32 * BM * wave + 1024 * j), vt0 + (uint32_t)j * vt_step, rt, so_t);
#pragma unroll
      for (int j = 0; j < NW; ++j)
        dma16(base + (uint32_t)(BM * 128 + 32 * BN * wave + 1024 * j), vn0 + (uint32_t)j * vn_step, rw, so_n);
      if (st == 0) {
        vm_wait<0>();
        __syncthreads();
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) read_frag(f0, i, 0u, 0);

  for (int id = first; id < xend; id += stride) {
    const bool has_next = id + stride < xend;
    const Tile nxt = decode(has_next ? id + stride : id);
    const i32x4_t rw_cur = w_rsrc(cur), rw_nxt = w_rsrc(nxt);

    // One reduction step s of the current tile.  rd: read the next step's
    // half-0 fragments (the next tile's step 0 after the last step); ld: load
    // step s + 2, of this tile or (s + 2 >= nsteps) of the next.  ZERO: the
    // tile's first step starts every accumulator from zero.
    auto step = [&](int s, bool rd, bool ld, auto ZERO) __attribute__((always_inline)) {
      const uint32_t cst = (uint32_t)((s & 1) * STAGE), nst = (uint32_t)(((s + 1) & 1) * STAGE);
      wait_all(f0);
      const int s2 = s + 2 < nsteps ? s + 2 : s + 2 - nsteps;   // step to load, in its tile
      const bool in_cur = s + 2 < nsteps;
      uint32_t sl = 0;   // layer 1: source layer of step s2, read now, used after the barrier
      if constexpr (LAYER == 1)
        asm volatile("ds_read_b32 %0, %1" : "=v"(sl) : "v"(tab + 4u * (uint32_t)(s2 >> 1)));
#pragma unroll
      for (int m = 0; m < 64; ++m) {
        if constexpr (decltype(ZERO)::value)
          asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0"
                       : "=&a"(acc[m >> 3][m & 7]) : "v"(f0[8 + (m >> 3)]), "v"(f0[m & 7]));
        else
          asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                       : "+a"(acc[m >> 3][m & 7]) : "v"(f0[8 + (m >> 3)]), "v"(f0[m & 7]));
        if (m % 2 == 0 && m < 32) read_frag(f1, m / 2, cst, 1);
      }
      wait_all(f1);   // also covers the source-layer read
      asm volatile("" : "+v"(sl));
      vm_wait<0>();
      __syncthreads();
      i32x4_t rt2 = rw_cur, rw2 = rw_cur;
      uint32_t so_t2 = 0, so_n2 = 0;
      // opaque copies: the offsets of the step's loads are formed at each load
      // rather than all kept live across the loop
      uint32_t vt = vt0, vn = vn0;
      asm volatile("" : "+v"(vt), "+v"(vn));
      if (ld) {
        const Tile& tl = in_cur ? cur : nxt;
        rt2 = a_rsrc(tl, LAYER == 1 ? (uint32_t)__builtin_amdgcn_readfirstlane(sl) : 0u);
        rw2 = in_cur ? rw_cur : rw_nxt;
        so_t2 = __builtin_amdgcn_readfirstlane(so_t_of(s2));
        so_n2 = __builtin_amdgcn_readfirstlane((uint32_t)(s2 * 128));
        // five wait states between these scalar operands and the loads below
        asm volatile("s_nop 4" : : "s"(rt2), "s"(rw2), "s"(so_t2), "s"(so_n2));
      }
#pragma unroll
      for (int m = 0; m < 64; ++m) {
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                     : "+a"(acc[m >> 3][m & 7]) : "v"(f1[8 + (m >> 3)]), "v"(f1[m & 7]));
        if (rd && m % 4 == 0) read_frag(f0, m / 4, nst, 0);
        // the step's NL loads spread over the half: one per EVERY matrix
        // instructions (a wave stalls less on each than when they are bunched)
        constexpr int EVERY = NL <= 16 ? 4 : 3;
        static_assert(NL * EVERY <= 64, "loads of a step must fit in half a step");
        if (ld && m % EVERY == 1) {
          const int j = m / EVERY;
          if (j < NT)
            dma16_near(lds0 + cst + (uint32_t)(32 * BM * wave + 1024 * j),
                       vt + (uint32_t)j * vt_step, rt2, so_t2);
          else if (j < NL)
            dma16_near(lds0 + cst + (uint32_t)(BM * 128 + 32 * BN * wave + 1024 * (j - NT)),
                       vn + (uint32_t)(j - NT) * vn_step, rw2, so_n2);
        }
      }
    };
    step(0, true, 2 < nsteps || has_next, std::true_type{});
    for (int s = 1; s < nsteps; ++s)
      step(s, s + 1 < nsteps || has_next, s + 2 < nsteps || has_next, std::false_type{});

    // wait states after the last matrix instruction, tied to every accumulator
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]),
                   "+a"(acc[0][4]), "+a"(acc[0][5]), "+a"(acc[0][6]), "+a"(acc[0][7]));
#pragma unroll
    for (int x = 1; x < 8; ++x)
      asm volatile("" : "+a"(acc[x][0]), "+a"(acc[x][1]), "+a"(acc[x][2]), "+a"(acc[x][3]),
                   "+a"(acc[x][4]), "+a"(acc[x][5]), "+a"(acc[x][6]), "+a"(acc[x][7]));

    // Epilogue.  Block (x, y) of a wave: lane holds outputs 32 (x / 2) + 8 gq +
    // 4 (x % 2) + r (r = 0..3) of its 128 for token 16 y + (lane & 15) of its 128.
    const int gq = lane >> 4;
    const int64_t net = (int64_t)a.l * a.H + cur.h;
    const uint16_t* bias = a.b[cur.kv];
    uint2 bw[8];   // the lane's biases, bf16, unpacked where used
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const int n = cur.n0 + 128 * wn + 32 * (x >> 1) + 8 * gq + 4 * (x & 1);
      bw[x] = bias != nullptr && n < N ? *reinterpret_cast<const uint2*>(bias + net * N + n)
                                       : make_uint2(0u, 0u);
    }
    if constexpr (LAYER < 3) {
      uint16_t* out = a.act_out + (int64_t)cur.g * T * F;
#pragma unroll
      for (int y = 0; y < 8; ++y) {
        const int t = cur.t0 + 128 * wt + 16 * y + (lane & 15);
        if (t >= T) continue;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int n = cur.n0 + 128 * wn + 32 * u + 8 * gq;
          float b0[4], b1[4], v0[4], v1[4];
          unpack4(bw[2 * u], b0);
          unpack4(bw[2 * u + 1], b1);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v0[r] = fmaxf(acc[2 * u][y][r] + b0[r], 0.f);
            v1[r] = fmaxf(acc[2 * u + 1][y][r] + b1[r], 0.f);
          }
          *reinterpret_cast<uint4*>(out + (int64_t)t * F + n) =
              make_uint4(pack2(v0[0], v0[1]), pack2(v0[2], v0[3]), pack2(v1[0], v1[1]), pack2(v1[2], v1[3]));
        }
      }
    } else {
      // the whole head: outputs = channels 0 .. 127 (wn == 0, n0 == 0)
      uint16_t* out = a.tgt + (((int64_t)a.l * 2 + cur.kv) * a.H + cur.h) * T * D;
#pragma unroll
      for (int y = 0; y < 8; ++y) {
        const int t = cur.t0 + 128 * wt + 16 * y + (lane & 15);
        if (t >= T) continue;
        const float2* cs = a.cs_tgt + (int64_t)t * (D / 2);
        uint16_t* orow = out + (int64_t)t * D + 8 * gq;
        // blocks 2u, 2u + 1 hold channels 32 u + 8 gq .. + 7 of the first half;
        // blocks 2u + 4, 2u + 5 their half-split RoPE partners 64 channels on
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          float p[2][4], q[2][4];   // p: first-half channels, q: their partners
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            const int x = 2 * u + b;
            float b0[4], b1[4];
            unpack4(bw[x], b0);
            unpack4(bw[x + 4], b1);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              p[b][r] = acc[x][y][r] + b0[r];
              q[b][r] = acc[x + 4][y][r] + b1[r];
            }
            if (cur.kv == 0) {
              const int c0 = 32 * u + 8 * gq + 4 * b;   // channel of register 0
              if (STYLE == 0) {
                // plane j = channel j of the first half
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                  const float2 c = cs[c0 + r];
                  const float u0 = p[b][r], v0 = q[b][r];
                  p[b][r] = __builtin_fmaf(u0, c.x, -(v0 * c.y));
                  q[b][r] = __builtin_fmaf(v0, c.x, u0 * c.y);
                }
              } else {
                // plane j = channels (2j, 2j + 1): registers r and r + 1
#pragma unroll
                for (int r = 0; r < 4; r += 2) {
                  const float2 e0 = cs[(c0 + r) >> 1];
                  const float2 e1 = cs[(c0 + 64 + r) >> 1];
                  const float u0 = p[b][r], u1 = p[b][r + 1], w0 = q[b][r], w1 = q[b][r + 1];
                  p[b][r] = __builtin_fmaf(u0, e0.x, -(u1 * e0.y));
                  p[b][r + 1] = __builtin_fmaf(u1, e0.x, u0 * e0.y);
                  q[b][r] = __builtin_fmaf(w0, e1.x, -(w1 * e1.y));
                  q[b][r + 1] = __builtin_fmaf(w1, e1.x, w0 * e1.y);
                }
              }
            }
          }
          *reinterpret_cast<uint4*>(orow + 32 * u) =
              make_uint4(pack2(p[0][0], p[0][1]), pack2(p[0][2], p[0][3]), pack2(p[1][0], p[1][1]), pack2(p[1][2], p[1][3]));
          *reinterpret_cast<uint4*>(orow + 64 + 32 * u) =
              make_uint4(pack2(q[0][0], q[0][1]), pack2(q[0][2], q[0][3]), pack2(q[1][0], q[1][1]), pack2(q[1][2], q[1][3]));
        }
      }
    }
    cur = nxt;
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
  // one persistent workgroup per CU (32 per XCD), fewer for small launches
  const dim3 grid((unsigned)(8 * (a.tiles_per_xcd < 32 ? a.tiles_per_xcd : 32)));
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
