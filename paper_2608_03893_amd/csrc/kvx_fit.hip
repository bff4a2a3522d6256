// Fitting side of the mapper: the whole per-head ridge fit (Sec. 3.1, Eq.
// Wstar with centring, from two models' caches of the same calibration
// tokens, Sec. 3.3 for the keys) and the single-source linear probe that
// chooses the source layers (Sec. 2.3, Eq. single_source_ols; Sec. 3.2).
//
// Both reduce to Gram matrices of per-token head features, then small SPD
// solves:
//   fit_prep_kernel   per (layer, K|V, head) plane of either cache and
//                     8192-token chunk: strip the RoPE from keys (fp32
//                     coefficients) and keep each stripped key as a bf16 pair
//                     hi + lo (the lo planes follow the planes), write the
//                     plane token-tiled (each 16-token step of a plane is one
//                     contiguous 4 KB slab: 128 channel rows of 16 tokens),
//                     and sum every channel and its square (fp64) for the
//                     centring; fit_sums_kernel adds the chunks' sums;
//   fit_plan_kernel   (fit) from the index table: the distinct Gram blocks
//                     (a source-pair block is shared by every target layer
//                     whose list holds the pair) and the jobs that compute
//                     them;
//   gram_kernel       batched 128 x 128 blocks P_a^T P_b of those planes on the
//                     matrix cores (bf16 operands, fp32 accumulation), one job
//                     = up to four blocks (one per wave) over at most four
//                     planes, which stream through an LDS ring of slabs; the
//                     fit's key blocks add hi.hi + hi.lo + lo.hi in the same
//                     sweep (the probe's take hi.hi only);
//   fit_solve_kernel  per (target layer, head, K|V): the centred design Gram
//                     plus lambda I, Cholesky in fp64 (32-column panels in
//                     LDS), forward and backward substitution for the
//                     centred cross Gram, the bias from the means;
//   probe_kernel      per (source layer, head, K|V) and half of the target
//                     layers: Cholesky and inverse of the centred Gram of
//                     that plane in LDS, then for every target layer the
//                     explained sum of squares ||L^-1 X_c^T Y_c||_F^2 over
//                     the total sum of squares;
//   topk_kernel       per target layer: the top-k source layers by R2
//                     averaged over heads and over keys and values.
#include <type_traits>

#include "kvx_bf16.h"
#include "kvx_fitplan.h"
#include "kvx_internal.h"

namespace kvx {
namespace {

constexpr int D = 128;        // head dimension of every fit kernel
constexpr int NB = 32;        // panel width of the Cholesky
constexpr int TS = 16;        // tokens per Gram step (the reduction of one matrix instruction)
constexpr int SLAB = D * TS * 2;   // bytes of one plane's step: 4 KB
constexpr int RING = 128 * 1024;   // LDS ring of the Gram kernel
constexpr int TP = D + 8;     // row stride (elements) of the prep kernel's LDS tiles

// Within a slab, channel row r (32 bytes) holds 16 tokens as two 8-token
// chunks; chunk c is stored at position c ^ swz(r), so that the fragment
// reads of 8 (and of 16) consecutive lanes, one row each, hit distinct banks.
__device__ __forceinline__ int swz(int r) { return ((r >> 2) ^ (r >> 3)) & 1; }

typedef __bf16 bf16x8_t_ __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef int i32x4_t_ __attribute__((ext_vector_type(4)));

__device__ __forceinline__ i32x4_t_ rsrc(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  i32x4_t_ r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// The rounding residual of key plane pid is stored as plane P + lo_slot(pid):
// one per (layer of either cache, head).
__device__ __forceinline__ int lo_slot(const FitArgs& a, int pid) {
  return (pid / (2 * a.H)) * a.H + pid % a.H;
}

// ------------------------------------------------------------------ fit plan
//
// A fit task (target layer l, head h, K|V) needs the blocks P_a^T P_b of every
// pair of its source planes (a <= b in list order) and the cross blocks
// P_a^T Q_l with its target plane.  The Gram of two source planes does not
// depend on the target layer, so each distinct pair of source layers is
// computed once per (head, K|V), by its owner: the first target layer whose
// list holds the pair (target layers in order, within a list the pairs (i, j),
// i <= j, in that order).  The items of target layer l are the cross blocks of
// its distinct source layers, then the pairs it owns; they take consecutive
// block slots, and they are packed first-fit into jobs of at most four blocks
// over at most four distinct planes.  Every table follows from the index
// table alone: the host runs plan_layer for the counts, and fit_plan_kernel
// writes the tables that the Gram and solve kernels read.
constexpr uint32_t kNoItem = 0xffffffffu;   // an idle wave
constexpr uint32_t kCross = 0x80000000u;    // item kCross | l << 8 | a: P_a^T Q_l
constexpr uint32_t kTransposed = 0x80000000u;   // solve table: the slot holds the transpose
constexpr int kMaxItems = 14;               // k(k + 3) / 2 for k = 4
constexpr int kEnt = 25;                    // solve table entries per target layer

// Items of one target layer; a pair item is b << 8 | a, the block P_a^T P_b.
struct LayerRec {
  uint32_t item[kMaxItems];
  uint8_t job[kMaxItems];      // job of each item, counted within the layer
  uint16_t unused0;
  int32_t n_items, n_cross, n_jobs, slot_base, job_base;
  int32_t unused1;
};
static_assert(sizeof(LayerRec) == 96, "plan record layout");

struct FitPlan {
  LayerRec* lay;     // [L_t]
  uint32_t* jobs;    // [n_jobs][4 waves][item, slot]
  uint32_t* stab;    // [L_t][5 x 5]: entry (x, y), x <= y < k: block of list
                     // positions x and y; (x, 4): the cross block of position
                     // x.  Value: slot | transposed << 31
  int32_t nj, nu;    // jobs and slots per (head, K|V)
};

__host__ __device__ __forceinline__ bool list_holds(const uint8_t* s, int k, int a, int b) {
  bool fa = false, fb = false;
  for (int i = 0; i < k; ++i) {
    fa |= s[i] == a;
    fb |= s[i] == b;
  }
  return fa && fb;
}

// The items of target layer l and their packing; returns the layer's jobs.
__host__ __device__ __forceinline__ int plan_layer(const uint8_t* idx, int k, int l, LayerRec& r) {
  const uint8_t* s = idx + l * k;
  int n = 0;
  for (int i = 0; i < k; ++i) {
    bool dup = false;
    for (int i2 = 0; i2 < i; ++i2) dup |= s[i2] == s[i];
    if (!dup) r.item[n++] = kCross | (uint32_t)l << 8 | s[i];
  }
  r.n_cross = n;
  for (int i = 0; i < k; ++i)
    for (int j = i; j < k; ++j) {
      const int a = s[i], b = s[j];
      bool seen = false;
      for (int l2 = 0; l2 < l && !seen; ++l2) seen = list_holds(idx + l2 * k, k, a, b);
      for (int i2 = 0; i2 <= i && !seen; ++i2)
        for (int j2 = i2; j2 < k; ++j2) {
          if (i2 == i && j2 >= j) break;   // (i2, j2) comes before (i, j)
          if ((s[i2] == a && s[j2] == b) || (s[i2] == b && s[j2] == a)) seen = true;
        }
      if (!seen) r.item[n++] = (uint32_t)b << 8 | a;
    }
  r.n_items = n;
  for (int t = 0; t < n; ++t) r.job[t] = 0xff;
  int nj = 0;
  for (int done = 0; done < n; ++nj) {
    int pl[4], np = 0, cnt = 0;
    for (int t = 0; t < n && cnt < 4; ++t) {
      if (r.job[t] != 0xff) continue;
      const uint32_t it = r.item[t];
      const int pa = (int)(it & 255u), pb = (it & kCross) ? 256 : (int)((it >> 8) & 255u);
      bool ha = false, hb = pb == pa;
      for (int q = 0; q < np; ++q) {
        ha |= pl[q] == pa;
        hb |= pl[q] == pb;
      }
      if (np + (ha ? 0 : 1) + (hb ? 0 : 1) > 4) continue;
      if (!ha) pl[np++] = pa;
      if (!hb) pl[np++] = pb;
      r.job[t] = (uint8_t)nj;
      ++cnt;
      ++done;
    }
  }
  r.n_jobs = nj;
  return nj;
}

// One workgroup: the layer records, their slot and job offsets, the jobs and
// the solve table.  Run by fit_plan_kernel, or by one extra workgroup of the
// prep kernel, which needs none of it, so that the plan is made while the
// planes are written.
__device__ void fit_plan_body(const FitArgs& a, const FitPlan& p) {
  const int k = a.k;
  for (int l = threadIdx.x; l < a.L_t; l += 256) plan_layer(a.idx, k, l, p.lay[l]);
  __syncthreads();
  if (threadIdx.x == 0) {
    int sb = 0, jb = 0;
    for (int l = 0; l < a.L_t; ++l) {
      p.lay[l].slot_base = sb;
      p.lay[l].job_base = jb;
      sb += p.lay[l].n_items;
      jb += p.lay[l].n_jobs;
    }
  }
  __syncthreads();
  for (int l = threadIdx.x; l < a.L_t; l += 256) {
    const LayerRec& r = p.lay[l];
    for (int j = 0; j < r.n_jobs; ++j) {
      uint32_t* o = p.jobs + (int64_t)(r.job_base + j) * 8;
      int w = 0;
      for (int t = 0; t < r.n_items; ++t)
        if (r.job[t] == j) {
          o[2 * w] = r.item[t];
          o[2 * w + 1] = (uint32_t)(r.slot_base + t);
          ++w;
        }
      for (; w < 4; ++w) {
        o[2 * w] = kNoItem;
        o[2 * w + 1] = 0u;
      }
    }
    const uint8_t* s = a.idx + l * k;
    uint32_t* st = p.stab + (int64_t)l * kEnt;
    for (int e = 0; e < kEnt; ++e) {
      const int x = e / 5, y = e % 5;
      uint32_t v = 0u;   // entries the solve does not use point at slot 0
      if (x < k && y == 4) {
        for (int t = 0; t < r.n_cross; ++t)
          if ((r.item[t] & 255u) == s[x]) v = (uint32_t)(r.slot_base + t);
      } else if (x <= y && y < k) {
        const int xa = s[x], yb = s[y];
        int l0 = 0;
        while (!list_holds(a.idx + l0 * k, k, xa, yb)) ++l0;   // ends at l at the latest
        const LayerRec& r0 = p.lay[l0];
        for (int t = r0.n_cross; t < r0.n_items; ++t) {
          const int ia = (int)(r0.item[t] & 255u), ib = (int)((r0.item[t] >> 8) & 255u);
          if (ia == xa && ib == yb) v = (uint32_t)(r0.slot_base + t);
          else if (ia == yb && ib == xa) v = (uint32_t)(r0.slot_base + t) | kTransposed;
        }
      }
      st[e] = v;
    }
  }
}

__global__ __launch_bounds__(256) void fit_plan_kernel(const FitArgs a, const FitPlan p) {
  fit_plan_body(a, p);
}

// ------------------------------------------------------------------ prep

// One (plane, token chunk) of the prep kernel: KEYS planes are stripped of the
// RoPE rotation and also get the rounding residual.  The body is one template
// per plane kind so that the loop has no branch around its loads: the rows of
// the next 64 tokens (and, for keys, their RoPE coefficients) are loaded
// before the current tokens are written out and stay untouched until the next
// pass, so they fly during the write phase.  The last pass loads one more
// (clamped) row group that nothing uses.  Tokens past N load the last token's
// row and are replaced by zeros where the pass takes them up.
template <bool KEYS>
__device__ __forceinline__ void prep_chunk(const FitArgs& a, int pid, int ch, const uint16_t* plane,
                                           const float2* cs, uint16_t* out, uint16_t* out_lo,
                                           uint16_t* tile, uint16_t* tile_lo, double (*red)[4][D]) {
  const int t_lo = ch * kPrepChunk, t_hi = min(a.Npad, t_lo + kPrepChunk);
  const int t = threadIdx.x;
  const int g = t & 7;         // channels 8g .. 8g+7 and 64+8g .. 64+8g+7
  const int tk = t >> 3;       // token within half a pass
  // channel sums of the values the Gram sees (hi + lo; lo is zero for
  // values), taken from the tile in the write phase: lane pair (2j, 2j + 1)
  // of every wave holds channels j, 32 + j, 64 + j, 96 + j
  double s1[4], s2[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) s1[e] = s2[e] = 0.0;
  // coefficient float4s of the row's planes: style 0 planes 8g .. 8g+7;
  // style 1 planes 4g .. 4g+3 and 32+4g .. 32+4g+3
  const int c0 = a.style == 0 ? 4 * g : 2 * g;
  const int c2 = a.style == 0 ? 4 * g + 2 : 16 + 2 * g;
  uint4 rx[2], ry[2];
  float4 rc[2][4];
  auto load = [&](int t0) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int tok = t0 + tk + 32 * it;
      const int64_t tc = tok < a.N ? tok : a.N - 1;
      rx[it] = *reinterpret_cast<const uint4*>(plane + tc * D + 8 * g);
      ry[it] = *reinterpret_cast<const uint4*>(plane + tc * D + 64 + 8 * g);
      if constexpr (KEYS) {
        const float4* c4 = reinterpret_cast<const float4*>(cs + tc * (D / 2));
        rc[it][0] = c4[c0];
        rc[it][1] = c4[c0 + 1];
        rc[it][2] = c4[c2];
        rc[it][3] = c4[c2 + 1];
      }
    }
  };
  load(t_lo);
  // vmcnt(0): the first pass needs these rows anyway, and with nothing in
  // flight at the loop's entry the pass waits at its top only for the rows,
  // not for the previous pass's stores that went out after them
  __builtin_amdgcn_s_waitcnt(0x0f70);
  for (int t0 = t_lo; t0 < t_hi; t0 += 64) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int row = tk + 32 * it;
      const uint4 z = make_uint4(0u, 0u, 0u, 0u);
      const bool ok = t0 + row < a.N;
      uint4 x = ok ? rx[it] : z, y = ok ? ry[it] : z, xl = z, yl = z;
      if constexpr (KEYS) {
        uint32_t* px = reinterpret_cast<uint32_t*>(&x);
        uint32_t* py = reinterpret_cast<uint32_t*>(&y);
        const float* cf = reinterpret_cast<const float*>(&rc[it][0]);   // 16 floats: (cos, sin) x 8
        if (a.style == 0) {
          // plane j = (channel j, channel j + 64): x holds the first members
          // of planes 8g .. 8g+7, y the second ones
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            float u0 = lo_bf16(px[w]), u1 = hi_bf16(px[w]);
            float v0 = lo_bf16(py[w]), v1 = hi_bf16(py[w]);
            const float c0x = cf[4 * w], c0y = cf[4 * w + 1], c1x = cf[4 * w + 2], c1y = cf[4 * w + 3];
            const float nu0 = u0 * c0x + v0 * c0y, nv0 = v0 * c0x - u0 * c0y;
            const float nu1 = u1 * c1x + v1 * c1y, nv1 = v1 * c1x - u1 * c1y;
            px[w] = pack2(nu0, nu1);
            py[w] = pack2(nv0, nv1);
            reinterpret_cast<uint32_t*>(&xl)[w] =
                pack2(nu0 - lo_bf16(px[w]), nu1 - hi_bf16(px[w]));
            reinterpret_cast<uint32_t*>(&yl)[w] =
                pack2(nv0 - lo_bf16(py[w]), nv1 - hi_bf16(py[w]));
          }
        } else {
          // plane j = (channel 2j, channel 2j + 1): the four words of x hold
          // planes 4g .. 4g+3, those of y planes 32+4g .. 32+4g+3
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const float cxx = cf[2 * w], cxy = cf[2 * w + 1];
            const float cyx = cf[8 + 2 * w], cyy = cf[8 + 2 * w + 1];
            float u = lo_bf16(px[w]), v = hi_bf16(px[w]);
            float nu = u * cxx + v * cxy, nv = v * cxx - u * cxy;
            px[w] = pack2(nu, nv);
            reinterpret_cast<uint32_t*>(&xl)[w] = pack2(nu - lo_bf16(px[w]), nv - hi_bf16(px[w]));
            u = lo_bf16(py[w]);
            v = hi_bf16(py[w]);
            nu = u * cyx + v * cyy;
            nv = v * cyx - u * cyy;
            py[w] = pack2(nu, nv);
            reinterpret_cast<uint32_t*>(&yl)[w] = pack2(nu - lo_bf16(py[w]), nv - hi_bf16(py[w]));
          }
        }
      }
      *reinterpret_cast<uint4*>(tile + row * TP + 8 * g) = x;
      *reinterpret_cast<uint4*>(tile + row * TP + 64 + 8 * g) = y;
      if constexpr (KEYS) {
        *reinterpret_cast<uint4*>(tile_lo + row * TP + 8 * g) = xl;
        *reinterpret_cast<uint4*>(tile_lo + row * TP + 64 + 8 * g) = yl;
      }
    }
    __syncthreads();
    load(t0 + 64);
    // token-tiled write: the 64 tokens are 4 slabs; wave q writes slab q (4 KB
    // contiguous), store i the 16-byte pieces m = 64 i + lane (1 KB
    // contiguous); piece m = (row r = m / 2, position m % 2) holds token chunk
    // (m % 2) ^ swz(r)
    {
      const int q = t >> 6, lane = t & 63;
      const int64_t so = (int64_t)(t0 / TS + q) * (D * TS);   // element offset of the slab
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 64 * i + lane, r = m >> 1, c = (m & 1) ^ swz(r);
        const int tok = TS * q + 8 * c;
        uint32_t w[4], wl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = (uint32_t)tile[(tok + 2 * e) * TP + r] | ((uint32_t)tile[(tok + 2 * e + 1) * TP + r] << 16);
        *reinterpret_cast<uint4*>(out + so + 8 * m) = make_uint4(w[0], w[1], w[2], w[3]);
        if constexpr (KEYS) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            wl[e] = (uint32_t)tile_lo[(tok + 2 * e) * TP + r] |
                    ((uint32_t)tile_lo[(tok + 2 * e + 1) * TP + r] << 16);
          *reinterpret_cast<uint4*>(out_lo + so + 8 * m) = make_uint4(wl[0], wl[1], wl[2], wl[3]);
        }
        // channel r of these 8 tokens: piece i of every pass is channel
        // 32 i + lane / 2
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          double u = lo_bf16(w[e]), v = hi_bf16(w[e]);
          if constexpr (KEYS) {
            u += lo_bf16(wl[e]);
            v += hi_bf16(wl[e]);
          }
          s1[i] += u + v;
          s2[i] = fma(u, u, fma(v, v, s2[i]));
        }
      }
    }
    __syncthreads();
  }
  // channel sums: the two lanes of a pair, then the four waves
  const int wave = t >> 6, lane = t & 63;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s1[i] += __shfl_xor(s1[i], 1);
    s2[i] += __shfl_xor(s2[i], 1);
    if ((lane & 1) == 0) {
      red[0][wave][32 * i + (lane >> 1)] = s1[i];
      red[1][wave][32 * i + (lane >> 1)] = s2[i];
    }
  }
  __syncthreads();
  if (t < D) {
    const int64_t o = ((int64_t)ch * a.P + pid) * D + t;   // this chunk's partial sums
    a.sums[o] = red[0][0][t] + red[0][1][t] + red[0][2][t] + red[0][3][t];
    a.sumsq[o] = red[1][0][t] + red[1][1][t] + red[1][2][t] + red[1][3][t];
  }
}

// Work item (plane, token chunk).  Block b runs on XCD b % 8; the H heads of
// one (cache, layer, K|V) and chunk take consecutive blocks of one XCD, so
// their key planes read each token's RoPE coefficients through that XCD's L2
// together.  Blocks past the last item exit at once, except block plan_block
// (if not -1, the last one of the grid), which makes the fit's plan.
__global__ __launch_bounds__(256) void fit_prep_kernel(const FitArgs a, const FitPlan pl, int plan_block) {
  if ((int)blockIdx.x == plan_block) {
    fit_plan_body(a, pl);
    return;
  }
  __shared__ __attribute__((aligned(16))) uint16_t tile[64 * TP];     // [token][channel]
  __shared__ __attribute__((aligned(16))) uint16_t tile_lo[64 * TP];
  __shared__ double red[2][4][D];
  const int n_ch = prep_chunks(a.Npad);
  const int units = (a.P / a.H) * n_ch;       // (cache, layer, K|V) x chunk
  const int r_ = (int)(blockIdx.x >> 3), unit = (r_ / a.H) * 8 + (int)(blockIdx.x & 7);
  if (unit >= units) return;
  const int ch = unit % n_ch;
  const int pid = (unit / n_ch) * a.H + r_ % a.H;
  const int nsrc = a.L_s * 2 * a.H;
  const bool is_src = pid < nsrc;
  const int q = is_src ? pid : pid - nsrc;                 // plane within its cache
  const uint16_t* plane = (is_src ? a.src : a.tgt) + (int64_t)q * a.N * D;
  uint16_t* out = a.planes + (int64_t)pid * fit_plane_stride(a.Npad);
  if (((q / a.H) & 1) == 0) {
    // keys also get the rounding residual: plane hi + lo carries the
    // stripped key to about 16 significant bits
    uint16_t* out_lo = a.planes + (int64_t)(a.P + lo_slot(a, pid)) * fit_plane_stride(a.Npad);
    prep_chunk<true>(a, pid, ch, plane, is_src ? a.cs_src : a.cs_tgt, out, out_lo, tile, tile_lo, red);
  } else {
    prep_chunk<false>(a, pid, ch, plane, nullptr, out, nullptr, tile, tile_lo, red);
  }
}

// The channel sums of every plane: the chunks' partial sums added in chunk
// order into the first chunk's slot, which the later kernels read.
__global__ __launch_bounds__(256) void fit_sums_kernel(const FitArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x, n = (int64_t)a.P * D;
  if (i >= n) return;
  const int n_ch = prep_chunks(a.Npad);
  double s1 = a.sums[i], s2 = a.sumsq[i];
  for (int c = 1; c < n_ch; ++c) {
    s1 += a.sums[c * n + i];
    s2 += a.sumsq[c * n + i];
  }
  a.sums[i] = s1;
  a.sumsq[i] = s2;
}

// ------------------------------------------------------------------ Gram

// Jobs.  The fit's jobs are the plan's jobs of every (head h, K|V): job
// (2 h + kv) * nj + j, so each XCD's contiguous job range holds one head's key
// and value blocks.  A probe group (head h, K|V) needs P_s^T P_s and P_s^T Q_l for
// every source layer s and target layer l: its jobs are 2 x 2 tiles (source
// pair) x (target pair), ordered in blocks of 4 source pairs so that 32
// consecutive jobs (the CUs of an XCD) share 8 source and 16 target planes,
// then the self blocks four at a time.
struct GJob {
  int np;              // distinct planes (<= 4)
  int keys;            // key planes: hi and lo slabs per plane
  int pid[4];          // their plane ids
  int sa, sb;          // this wave's A and B plane (index into pid), sa < 0: idle
  int64_t out;         // this wave's output block
};

__device__ __forceinline__ int add_plane(GJob& j, int p) {
  int f = -1;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (i < j.np && j.pid[i] == p) f = i;
  if (f >= 0) return f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (i == j.np) j.pid[i] = p;
  return j.np++;
}

__device__ __forceinline__ int probe_jobs_per_group(const FitArgs& a) {
  const int n_sp = (a.L_s + 1) / 2, n_lp = (a.L_t + 1) / 2;
  return n_sp * n_lp + (a.L_s + 3) / 4;
}

__device__ __forceinline__ GJob decode_job(const FitArgs& a, const FitPlan& p, int job, int wave) {
  GJob j;
  j.np = 0;
  j.sa = j.sb = -1;
  j.out = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) j.pid[i] = 0;
  const int nsrc = a.L_s * 2 * a.H;
  if (a.mode == 0) {
    const int hk = job / p.nj, jj = job - hk * p.nj, kv = hk & 1, h = hk >> 1;
    j.keys = kv == 0;
    const uint32_t* o = p.jobs + (int64_t)jj * 8;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t it = o[2 * w];
      if (it == kNoItem) continue;
      const int pa = ((int)(it & 255u) * 2 + kv) * a.H + h;
      const int pb = (it & kCross) ? nsrc + ((int)((it >> 8) & 0xffffu) * 2 + kv) * a.H + h
                                   : ((int)((it >> 8) & 255u) * 2 + kv) * a.H + h;
      const int sa = add_plane(j, pa), sb = add_plane(j, pb);
      if (w == wave) {
        j.sa = sa;
        j.sb = sb;
        j.out = (int64_t)hk * p.nu + o[2 * w + 1];
      }
    }
  } else {
    const int per = probe_jobs_per_group(a);
    const int grp = job / per, c = job - grp * per;
    const int h = grp >> 1, kv = grp & 1;
    // the probe's key Grams take the stripped keys rounded once to bf16 (the
    // hi planes): one product, as for values
    j.keys = 0;
    const int n_sp = (a.L_s + 1) / 2, n_lp = (a.L_t + 1) / 2;
    const int base_task = a.L_s * (2 * h + kv);   // probe task of source s: base_task + s
    if (c < n_sp * n_lp) {
      const int fb = n_sp / 4;
      int sbk, rem, rows;
      if (c < fb * 4 * n_lp) {
        sbk = c / (4 * n_lp);
        rem = c - sbk * 4 * n_lp;
        rows = 4;
      } else {
        sbk = fb;
        rem = c - fb * 4 * n_lp;
        rows = n_sp - fb * 4;
      }
      const int lp = rem / rows, sp = sbk * 4 + (rem - lp * rows);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int sl = 2 * sp + (w >> 1), l = 2 * lp + (w & 1);
        if (sl >= a.L_s || l >= a.L_t) continue;
        const int sa = add_plane(j, (sl * 2 + kv) * a.H + h);
        const int sb = add_plane(j, nsrc + (l * 2 + kv) * a.H + h);
        if (w == wave) {
          j.sa = sa;
          j.sb = sb;
          j.out = (int64_t)(base_task + sl) * (a.L_t + 1) + 1 + l;
        }
      }
    } else {
      const int c2 = c - n_sp * n_lp;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int sl = 4 * c2 + w;
        if (sl >= a.L_s) continue;
        const int sa = add_plane(j, (sl * 2 + kv) * a.H + h);
        if (w == wave) {
          j.sa = j.sb = sa;
          j.out = (int64_t)(base_task + sl) * (a.L_t + 1);
        }
      }
    }
  }
  return j;
}

template <int N>
__device__ __forceinline__ void vm_wait_n() { asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory"); }

// f(integral_constant<int, I>) for I = B .. E - 1, in order
template <int B, int E, typename Fn>
__device__ __forceinline__ void static_for(Fn&& fn) {
  if constexpr (B < E) {
    fn(std::integral_constant<int, B>{});
    static_for<B + 1, E>(fn);
  }
}

// One job: four waves, one 128 x 128 block each (4 x 4 accumulators of
// v_mfma_f32_32x32x16_bf16, 256 AGPRs), over all tokens in 16-token steps.
// A stage of the LDS ring holds the step's slab of every plane of the job
// (and of its residual plane for keys): 8 slabs (keys, 4 stages) or 4
// (values, 8 stages).  Each wave loads one 1 KB quarter of every slab straight
// into LDS.  Step s: wait for this wave's loads of step s + 1 and for the
// fragments it read during step s - 1, barrier (step s + 1 landed for every
// wave; the stage of step s - 1 was last read during step s - 2), then run
// step s's matrix instructions on those fragments while reading step s + 1's
// fragments and loading step s + NST - 1 into the stage of step s - 1.  In
// the steady state the reads and loads go out between the matrix
// instructions, so that the matrix pipe starts at the barrier.  Key blocks
// add hi.hi + hi.lo + lo.hi in the same step.
template <bool KEYS, int NP>
__device__ __forceinline__ void gram_job(const FitArgs& a, const GJob& jb, uint32_t lds0, int lane,
                                         int wave) {
  constexpr int NSL = KEYS ? 8 : 4;            // slab slots per stage
  constexpr int SBY = NSL * SLAB;              // stage bytes
  constexpr int NST = RING / SBY;              // stages: 4 or 8
  constexpr int NF = KEYS ? 16 : 8;            // fragments per step
  constexpr int nsl = KEYS ? 2 * NP : NP;      // slabs this job loads per step
  const int total = a.Npad / TS;
  const uint32_t plane_bytes = (uint32_t)(D * a.Npad * 2);

  // slab i of a step: keys: plane pid[i / 2] (i even) or its residual (i odd);
  // values: plane pid[i]
  i32x4_t_ rs[nsl];
#pragma unroll
  for (int i = 0; i < nsl; ++i) {
    int p = jb.pid[KEYS ? (i >> 1) : i];
    if (KEYS && (i & 1)) p = a.P + lo_slot(a, p);
    rs[i] = rsrc(a.planes + (int64_t)p * fit_plane_stride(a.Npad), plane_bytes);
  }
  auto issue = [&](int st) __attribute__((always_inline)) {
    const uint32_t base = lds0 + (uint32_t)((st % NST) * SBY + wave * 1024);
    const uint32_t vo = (uint32_t)st * SLAB + (uint32_t)(wave * 1024 + lane * 16);
#pragma unroll
    for (int i = 0; i < nsl; ++i)
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   :
                   : "s"(base + (uint32_t)(i * SLAB)), "v"(vo), "s"(rs[i])
                   : "memory");
  };

  f32x16_t acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    acc[i] = (f32x16_t){0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    asm volatile("" : "+a"(acc[i]));
  }
  const bool active = jb.sa >= 0;
  const int sa = active ? jb.sa : 0, sb = active ? jb.sb : 0;
  // fragment i of a plane: row r = 32 i + lane % 32, token chunk lane / 32
  const int fr = lane & 31;
  const uint32_t fo = (uint32_t)(fr * 32 + 16 * ((lane >> 5) ^ swz(fr)));
  // this wave's operands within a stage: A hi, B hi (and A lo, B lo)
  const uint32_t oah = (uint32_t)((KEYS ? 2 * sa : sa) * SLAB) + fo;
  const uint32_t obh = (uint32_t)((KEYS ? 2 * sb : sb) * SLAB) + fo;
  // fragments: A hi 0..3, B hi 4..7, A lo 8..11, B lo 12..15, read by inline
  // assembly (fragment f at the A or B base plus a constant offset); every
  // step starts with a wait for the fragments read during the step before
  auto read_frag = [&](auto fc, uint32_t sbase, bf16x8_t_* f) __attribute__((always_inline)) {
    constexpr int fi = decltype(fc)::value;
    constexpr int off = (fi & 3) * 1024 + (fi >= 8 ? SLAB : 0);
    const uint32_t addr = sbase + ((fi & 4) ? obh : oah);
    bf16x8_t_& v = f[fi];
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(off));
  };
  auto read_step = [&](int st, bf16x8_t_* f) __attribute__((always_inline)) {
    const uint32_t sbase = lds0 + (uint32_t)((st % NST) * SBY);
    static_for<0, NF>([&](auto fc) __attribute__((always_inline)) { read_frag(fc, sbase, f); });
  };
  auto wait_frags = [&](bf16x8_t_* g) __attribute__((always_inline)) {
    if constexpr (KEYS)
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(g[0]), "+v"(g[1]), "+v"(g[2]), "+v"(g[3]), "+v"(g[4]), "+v"(g[5]),
                     "+v"(g[6]), "+v"(g[7]), "+v"(g[8]), "+v"(g[9]), "+v"(g[10]), "+v"(g[11]),
                     "+v"(g[12]), "+v"(g[13]), "+v"(g[14]), "+v"(g[15]));
    else
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(g[0]), "+v"(g[1]), "+v"(g[2]), "+v"(g[3]), "+v"(g[4]), "+v"(g[5]),
                     "+v"(g[6]), "+v"(g[7]));
  };
  // matrix instruction m of a step: (A, B) = (i, 4 + jx) for hi.hi, then
  // (i, 12 + jx) for hi.lo and (8 + i, 4 + jx) for lo.hi (keys)
  constexpr int NM = KEYS ? 48 : 16;
  auto mfma_one = [&](auto mc, const bf16x8_t_* g) __attribute__((always_inline)) {
    constexpr int m = decltype(mc)::value;
    constexpr int i = (m & 15) >> 2, jx = m & 3, part = m >> 4;
    constexpr int fa_ = (part == 2 ? 8 : 0) + i, fb_ = (part == 1 ? 12 : 4) + jx;
    f32x16_t& c = acc[4 * i + jx];   // (asm operands alone do not capture)
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(g[fa_]), "v"(g[fb_]));
  };
  auto mfma_step = [&](const bf16x8_t_* g) __attribute__((always_inline)) {
    static_for<0, NM>([&](auto mc) __attribute__((always_inline)) { mfma_one(mc, g); });
  };
  bf16x8_t_ fa[NF], fb[NF];
  auto step = [&](int s, bf16x8_t_* cur, bf16x8_t_* nxt) __attribute__((always_inline)) {
    // step s + 1 landed: in steady state the loads of steps s + 2 .. s + NST - 2
    // may stay in flight; near the end wait for all
    if (s + NST - 1 <= total) vm_wait_n<nsl * (NST - 3)>();
    else vm_wait_n<0>();
    if (active) wait_frags(cur);
    __syncthreads();
    if (s + NST - 1 < total) issue(s + NST - 1);
    if (active) {
      if (s + 1 < total) read_step(s + 1, nxt);
      mfma_step(cur);
    }
  };
  // a step of an active wave with both a load and a read ahead: the matrix
  // pipe starts right after the barrier, and the fragment reads (after the
  // first NF matrix instructions) and the loads (after every other one from
  // then on) go out between the matrix instructions
  auto step_steady = [&](int s, bf16x8_t_* cur, bf16x8_t_* nxt) __attribute__((always_inline)) {
    vm_wait_n<nsl * (NST - 3)>();
    wait_frags(cur);
    __syncthreads();
    const int st = s + NST - 1;
    const uint32_t lbase = lds0 + (uint32_t)((st % NST) * SBY + wave * 1024);
    const uint32_t vo = (uint32_t)st * SLAB + (uint32_t)(wave * 1024 + lane * 16);
    const uint32_t sbase = lds0 + (uint32_t)(((s + 1) % NST) * SBY);
    static_for<0, NM>([&](auto mc) __attribute__((always_inline)) {
      constexpr int m = decltype(mc)::value;
      mfma_one(mc, cur);
      if constexpr (m < NF) read_frag(std::integral_constant<int, m>{}, sbase, nxt);
      if constexpr (m >= NF && (m - NF) % 2 == 0 && (m - NF) / 2 < nsl) {
        constexpr int i = (m - NF) / 2;
        const uint32_t lb = lbase + (uint32_t)(i * SLAB), v = vo;
        const i32x4_t_ r = rs[i];
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                     :
                     : "s"(lb), "v"(v), "s"(r)
                     : "memory");
      }
    });
  };

  // prologue: steps 0 .. NST - 2 in flight; step 0 landed everywhere
  for (int st = 0; st < NST - 1 && st < total; ++st) issue(st);
  if (total >= NST - 1) vm_wait_n<nsl * (NST - 2)>();
  else vm_wait_n<0>();
  __syncthreads();
  if (active) read_step(0, fa);
  int s = 0;
  if (active)
    for (; s + 1 < total - NST + 1; s += 2) {
      step_steady(s, fa, fb);
      step_steady(s + 1, fb, fa);
    }
  for (; s + 1 < total; s += 2) {
    step(s, fa, fb);
    step(s + 1, fb, fa);
  }
  if (s < total) step(s, fa, fb);
  if (!active) return;
  // the matrix results are readable 18 wait states after the last matrix
  // instruction (the compiler does not see inside the assembly above)
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3"
               : "+a"(acc[0]), "+a"(acc[1]), "+a"(acc[2]), "+a"(acc[3]), "+a"(acc[4]),
                 "+a"(acc[5]), "+a"(acc[6]), "+a"(acc[7]), "+a"(acc[8]), "+a"(acc[9]),
                 "+a"(acc[10]), "+a"(acc[11]), "+a"(acc[12]), "+a"(acc[13]), "+a"(acc[14]),
                 "+a"(acc[15]));
  // block (32 i + row, 32 jx + col): accumulator register rr of lane L holds
  // row 8 (rr / 4) + 4 (L / 32) + rr % 4, column L % 32
  const int fh = lane >> 5;
  float* G = a.G + jb.out * (int64_t)(D * D);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jx = 0; jx < 4; ++jx) {
      const f32x16_t v = acc[4 * i + jx];
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int row = 32 * i + 8 * (rr >> 2) + 4 * fh + (rr & 3);
        G[row * D + 32 * jx + fr] = v[rr];
      }
    }
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gram_kernel(const FitArgs a, const FitPlan p) {
  __shared__ __attribute__((aligned(256))) char smem[RING];
  const int xcd = blockIdx.x & 7, qx = blockIdx.x >> 3;
  const int job = xcd * a.jobs_per_xcd + qx;   // an XCD takes a contiguous range of jobs
  if (job >= a.n_jobs) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const GJob jb = decode_job(a, p, job, wave);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)smem;
  switch (jb.keys * 4 + jb.np) {
    case 1: gram_job<false, 1>(a, jb, lds0, lane, wave); break;
    case 2: gram_job<false, 2>(a, jb, lds0, lane, wave); break;
    case 3: gram_job<false, 3>(a, jb, lds0, lane, wave); break;
    case 4: gram_job<false, 4>(a, jb, lds0, lane, wave); break;
    case 5: gram_job<true, 1>(a, jb, lds0, lane, wave); break;
    case 6: gram_job<true, 2>(a, jb, lds0, lane, wave); break;
    case 7: gram_job<true, 3>(a, jb, lds0, lane, wave); break;
    default: gram_job<true, 4>(a, jb, lds0, lane, wave); break;
  }
}

// ------------------------------------------------------------ fit solve

// The fp64 SPD solve of one fit task, blocked in 32-column panels.  The
// p x p matrix is kept as its lower triangle in column-major order, A[j * p +
// i] = A(i, j) for i >= j, so every panel, tile and row block below is read
// from global memory in contiguous pieces.  A panel of p - J rows is held in
// LDS transposed, PT[c][r] = A(J + r, J + c), so that 8 consecutive rows of
// one column are one 64-byte read; updates run as 8 x 8 register tiles
// (8 + 8 fp64 reads from LDS per 64 FMAs).  Copies between global memory and
// LDS keep 8 loads per thread in flight.
constexpr int PLD = 520;   // PT row stride (doubles): >= 512 + 8, even

// PT[c][r] = A(J + r, J + c) for c < 32, r < R (R <= 512)
__device__ __forceinline__ void load_panel(const double* A, int p, int J, int R, double* PT) {
  const int t = threadIdx.x;
#pragma unroll
  for (int c0 = 0; c0 < NB; c0 += 8) {
    double v[8][2];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = t + 256 * h < R ? t + 256 * h : R - 1;   // loads stay in range
        v[u][h] = A[(int64_t)(J + c0 + u) * p + J + r];
      }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = t + 256 * h;
        if (r < R) PT[(c0 + u) * PLD + r] = v[u][h];
      }
  }
}

// A(J + .., J + ..) -= L21 L21^T below the panel (lower triangle), L21 = PT rows 32 ..
__device__ void syrk_update(double* A, int p, int J, const double* PT) {
  const int R2 = p - J - NB;
  const int n8 = (R2 + 7) / 8;
  const int ntile = n8 * (n8 + 1) / 2;
  for (int tile = threadIdx.x; tile < ntile; tile += 256) {
    // u = ntile - 1 - tile enumerates the triangle row by row as (ui, uj),
    // uj <= ui; (bi, bj) = (n8 - 1 - uj, n8 - 1 - ui) then runs down the
    // columns, so that consecutive threads take consecutive row blocks of one
    // column block (neighbouring addresses in the column-major matrix)
    const int u = ntile - 1 - tile;
    int ui = (int)((sqrtf(8.0f * (float)u + 1.0f) - 1.0f) * 0.5f);
    while (ui * (ui + 1) / 2 > u) --ui;
    while ((ui + 1) * (ui + 2) / 2 <= u) ++ui;
    const int uj = u - ui * (ui + 1) / 2;
    const int bi = n8 - 1 - uj, bj = n8 - 1 - ui;
    // every tile lies inside the matrix (p - J - 32 is a multiple of 32); the
    // diagonal tiles also update the unused upper triangle, which nothing
    // reads.  The tile's old values are read first, so that their latency
    // passes under the products.
    double* At = A + (int64_t)(J + NB + 8 * bj) * p + J + NB + 8 * bi;
    double acc[8][8];
#pragma unroll
    for (int y = 0; y < 8; ++y)
#pragma unroll
      for (int x = 0; x < 8; ++x) acc[x][y] = At[(int64_t)y * p + x];
    for (int c = 0; c < NB; ++c) {
      double li[8], lj[8];
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        li[x] = PT[c * PLD + NB + 8 * bi + x];
        lj[x] = PT[c * PLD + NB + 8 * bj + x];
      }
#pragma unroll
      for (int x = 0; x < 8; ++x)
#pragma unroll
        for (int y = 0; y < 8; ++y) acc[x][y] = fma(-li[x], lj[y], acc[x][y]);
    }
#pragma unroll
    for (int y = 0; y < 8; ++y)
#pragma unroll
      for (int x = 0; x < 8; ++x) At[(int64_t)y * p + x] = acc[x][y];
  }
}

// The value of v in lane `lane` (a constant), through scalar registers.
__device__ __forceinline__ double lane_value(double v, int lane) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
  return __hiloint2double(hi, lo);
}

// Cholesky of the p x p matrix A (lower triangle, column-major, fp64, global
// memory) in place.
__device__ void chol_panels(double* A, int p, double* PT) {
  const int t = threadIdx.x;
  for (int J = 0; J < p; J += NB) {
    const int R = p - J;
    load_panel(A, p, J, R, PT);
    __syncthreads();
    // the panel's top 32 x 32 block, by wave 0: lane r < 32 holds row r; the
    // diagonal and the column below it are read from their lanes into scalar
    // registers (readlane: no LDS round trip in the dependent chain)
    if (t < 64) {
      double row[NB];
#pragma unroll
      for (int c = 0; c < NB; ++c) row[c] = t < NB ? PT[c * PLD + t] : 0.0;
      double rdg = 0.0;   // 1 / l(t, t) (the array is never indexed by t:
                          // that would put it in scratch memory)
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        const double dg = sqrt(lane_value(row[c], c));
        const double rd = 1.0 / dg;
        const double lrc = t == c ? dg : row[c] * rd;   // l(t, c) for t >= c
        rdg = t == c ? rd : rdg;
        row[c] = lrc;
#pragma unroll
        for (int c2 = c + 1; c2 < NB; ++c2) row[c2] -= lrc * lane_value(lrc, c2);
      }
      if (t < NB) {
#pragma unroll
        for (int c = 0; c < NB; ++c) PT[c * PLD + t] = row[c];   // upper part unused
        // past the last row of column t (PLD >= 512 + 8)
        PT[t * PLD + PLD - 1] = rdg;
      }
    }
    __syncthreads();
    // rows 32 .. R-1: L21 = A21 L11^-T, one row per thread, in registers
    for (int r = NB + t; r < R; r += 256) {
      double x[NB];
#pragma unroll
      for (int c = 0; c < NB; ++c) x[c] = PT[c * PLD + r];
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        double v = x[c];
#pragma unroll
        for (int q = 0; q < c; ++q) v = fma(-x[q], PT[q * PLD + c], v);
        x[c] = v * PT[c * PLD + PLD - 1];
      }
#pragma unroll
      for (int c = 0; c < NB; ++c) PT[c * PLD + r] = x[c];
    }
    __syncthreads();
    for (int c = 0; c < NB; ++c)
      for (int r = c + t; r < R; r += 256) A[(int64_t)(J + c) * p + J + r] = PT[c * PLD + r];
    syrk_update(A, p, J, PT);
    __syncthreads();
  }
}

// B = L^-T L^-1 B in place (B [p][128] row-major), L in the lower triangle of
// A (column-major), all 128 right-hand sides at once in blocks of 64 rows:
//   forward   Z_i = L_ii^-1 (B_i - sum_{j < i} L_ij Z_j),
//   backward  W_i = L_ii^-T (Z_i - sum_{j > i} L_ji^T W_j).
// A block's right-hand sides stay in registers (thread (tr, tc): rows 8 tr ..
// 8 tr + 7, columns tc + 32 y) while the factor's row block and the solved
// rows stream through LDS in double-buffered chunks of 16; the block is then
// multiplied by the inverse of its 64 x 64 diagonal block of L (or its
// transpose), the eight inverses formed once for both sweeps.  The
// right-hand sides are read and written once per block instead of after
// every panel.
constexpr int SQ = 64;           // rows per block
constexpr int SK = 16;           // reduction chunk
constexpr int SBS = D + 1;       // row stride of the staged block (doubles)
constexpr int SLD = SQ + 1;      // row stride of the staged diagonal block
// LDS: chunk buffers [2][SK][SQ] of the factor and [2][SK][D] of solved rows,
// the staged block [SQ][SBS] and diagonal block [SQ][SLD]
constexpr int S_LC = 0, S_ZC = S_LC + 2 * SK * SQ, S_BS = S_ZC + 2 * SK * D,
              S_LD = S_BS + SQ * SBS, S_END = S_LD + SQ * SLD;

template <bool BWD>
__device__ void solve_sweep(const double* A, double* B, int p, double* sm) {
  const int t = threadIdx.x;
  const int tr = t >> 5, tc = t & 31;
  const int nb = p / SQ;
  double* Lc = sm + S_LC;
  double* Zc = sm + S_ZC;
  double* Bs = sm + S_BS;
  double* Ld = sm + S_LD;
  for (int n = 0; n < nb; ++n) {
    const int i = BWD ? nb - 1 - n : n;
    const int r0 = SQ * i;
    // the block's right-hand sides
    double acc[8][4];
#pragma unroll
    for (int x = 0; x < 8; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) acc[x][y] = B[(int64_t)(r0 + 8 * tr + x) * D + tc + 32 * y];
    // solved rows that enter: forward rows 0 .. r0 - 1, backward r0 + 64 .. p - 1
    const int k0 = BWD ? r0 + SQ : 0;
    const int nch = (BWD ? p - r0 - SQ : r0) / SK;
    double pl[4], pz[8];
    // chunk c: Lc[k][r] = L(r0 + r, k0 + 16 c + k) (forward) or
    // L(k0 + 16 c + k, r0 + r) (backward); Zc[k][col] = B row k0 + 16 c + k
    auto fetch = [&](int c) __attribute__((always_inline)) {
      const int kb = k0 + SK * c;
      if (BWD) {
        const int r = t >> 2, k = 4 * (t & 3);   // column r0 + r of A holds L(kb + k .., r0 + r)
#pragma unroll
        for (int u = 0; u < 4; ++u) pl[u] = A[(int64_t)(r0 + r) * p + kb + k + u];
      } else {
        const int k = t >> 4, r = 4 * (t & 15);  // column kb + k of A holds L(r0 + r .., kb + k)
#pragma unroll
        for (int u = 0; u < 4; ++u) pl[u] = A[(int64_t)(kb + k) * p + r0 + r + u];
      }
      const int k = t >> 4, col = 8 * (t & 15);
#pragma unroll
      for (int u = 0; u < 8; ++u) pz[u] = B[(int64_t)(kb + k) * D + col + u];
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
      double* lc = Lc + buf * SK * SQ;
      double* zc = Zc + buf * SK * D;
      if (BWD) {
        const int r = t >> 2, k = 4 * (t & 3);
#pragma unroll
        for (int u = 0; u < 4; ++u) lc[(k + u) * SQ + r] = pl[u];
      } else {
        const int k = t >> 4, r = 4 * (t & 15);
#pragma unroll
        for (int u = 0; u < 4; ++u) lc[k * SQ + r + u] = pl[u];
      }
      const int k = t >> 4, col = 8 * (t & 15);
#pragma unroll
      for (int u = 0; u < 8; ++u) zc[k * D + col + u] = pz[u];
    };
    if (nch > 0) {
      fetch(0);
      stash(0);
    }
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      if (c + 1 < nch) fetch(c + 1);
      const double* lc = Lc + (c & 1) * SK * SQ;
      const double* zc = Zc + (c & 1) * SK * D;
#pragma unroll 4
      for (int k = 0; k < SK; ++k) {
        double l[8], z[4];
#pragma unroll
        for (int x = 0; x < 8; ++x) l[x] = lc[k * SQ + 8 * tr + x];
#pragma unroll
        for (int y = 0; y < 4; ++y) z[y] = zc[k * D + tc + 32 * y];
#pragma unroll
        for (int x = 0; x < 8; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) acc[x][y] = fma(-l[x], z[y], acc[x][y]);
      }
      if (c + 1 < nch) stash((c + 1) & 1);
      __syncthreads();
    }
    // the diagonal block: the updated right-hand sides go to LDS, and the
    // block's inverse M = L_ii^-1 (forward) or its transpose (backward),
    // stored transposed in the block's upper triangle, with the diagonal
    // 1 / L(r, r)
#pragma unroll
    for (int x = 0; x < 8; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) Bs[(8 * tr + x) * SBS + tc + 32 * y] = acc[x][y];
    for (int e = t; e < SQ * SQ; e += 256) {
      const int c = e >> 6, r = e & 63;   // Ld[r][c] = G(r, c): the factor applied to row c of Bs
      double v = 0.0;
      if (r == c) v = 1.0 / A[(int64_t)(r0 + r) * p + r0 + r];
      else if (!BWD && r > c) v = A[(int64_t)(r0 + r) * p + r0 + c];   // M(r, c)
      else if (BWD && r < c) v = A[(int64_t)(r0 + c) * p + r0 + r];    // M(c, r)
      Ld[r * SLD + c] = v;
    }
    __syncthreads();
    // rows 8 tr .. 8 tr + 7 of G Bs; G is lower (forward) or upper (backward)
    // triangular, so the sum runs over k <= 8 tr + 7 or k >= 8 tr
    {
      double out[8][4];
#pragma unroll
      for (int x = 0; x < 8; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) out[x][y] = 0.0;
      const int ka = BWD ? 8 * tr : 0, kz = BWD ? SQ : 8 * tr + 8;
#pragma unroll 4
      for (int k = ka; k < kz; ++k) {
        double g[8], z[4];
#pragma unroll
        for (int x = 0; x < 8; ++x) g[x] = Ld[(8 * tr + x) * SLD + k];
#pragma unroll
        for (int y = 0; y < 4; ++y) z[y] = Bs[k * SBS + tc + 32 * y];
#pragma unroll
        for (int x = 0; x < 8; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) out[x][y] = fma(g[x], z[y], out[x][y]);
      }
#pragma unroll
      for (int x = 0; x < 8; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) B[(int64_t)(r0 + 8 * tr + x) * D + tc + 32 * y] = out[x][y];
    }
    __syncthreads();
  }
}

// The inverses M_b = L_bb^-1 of the 64 x 64 diagonal blocks of the factor,
// four blocks at a time in LDS, one column per thread (forward
// substitution); M_b(r, c), r > c, is stored at A[(r0 + r) p + r0 + c] (the
// block's unused upper triangle), its diagonal is 1 / L(r, r).
__device__ void invert_diag_blocks(double* A, int p, double* sm) {
  const int t = threadIdx.x;
  const int nb = p / SQ;
  constexpr int LS = SQ + 1;   // row stride of a staged block
  for (int b0 = 0; b0 < nb; b0 += 4) {
    const int nbb = nb - b0 < 4 ? nb - b0 : 4;
    for (int e = t; e < nbb * SQ * SQ; e += 256) {
      const int bb = e / (SQ * SQ), rem = e - bb * SQ * SQ, c = rem >> 6, r = rem & 63;
      const int r0 = SQ * (b0 + bb);
      sm[bb * SQ * LS + r * LS + c] = r >= c ? A[(int64_t)(r0 + c) * p + r0 + r] : 0.0;
    }
    __syncthreads();
    // thread (bb, j): column j of block bb; M(i, j) for i > j goes to the
    // staged block's upper triangle at [j][i]
    const int bb = t >> 6, j = t & 63;
    if (bb < nbb) {
      double* L = sm + bb * SQ * LS;
      const double mjj = 1.0 / L[j * LS + j];
      for (int i = j + 1; i < SQ; ++i) {
        double v = L[i * LS + j] * mjj;
        for (int q = j + 1; q < i; ++q) v = fma(L[i * LS + q], L[j * LS + q], v);
        L[j * LS + i] = -v / L[i * LS + i];
      }
    }
    __syncthreads();
    for (int e = t; e < nbb * SQ * SQ; e += 256) {
      const int bb2 = e / (SQ * SQ), rem = e - bb2 * SQ * SQ, r = rem >> 6, c = rem & 63;   // M(c, r), c > r
      const int r0 = SQ * (b0 + bb2);
      if (c > r) A[(int64_t)(r0 + c) * p + r0 + r] = sm[bb2 * SQ * LS + r * LS + c];
    }
    __syncthreads();
  }
}

__device__ void chol_solve(double* A, double* B, int p, double* sm) {
  invert_diag_blocks(A, p, sm);
  solve_sweep<false>(A, B, p, sm);
  solve_sweep<true>(A, B, p, sm);
}

__global__ __launch_bounds__(256) void fit_solve_kernel(const FitArgs a, const FitPlan pl) {
  // one array for the factorization's transposed panel (133 KB) and, after
  // it, the substitutions' buffers (145 KB)
  __shared__ double PT[S_END > NB * PLD ? S_END : NB * PLD];
  const int task = blockIdx.x;
  const int k = a.k, p = k * D;
  const int l = task % a.L_t, hk = task / a.L_t, kv = hk & 1, h = hk >> 1;
  __shared__ uint32_t st[kEnt];     // this task's slots (plan solve table)
  __shared__ double SX[4 * D];      // channel sums of the k source planes
  const int t = threadIdx.x;
  if (t < kEnt) st[t] = pl.stab[(int64_t)l * kEnt + t];
  for (int e = t; e < p; e += 256) {
    const int ai = e / D;
    SX[e] = a.sums[(int64_t)(((int)a.idx[l * k + ai] * 2 + kv) * a.H + h) * D + e % D];
  }
  __syncthreads();
  const int nsrc = a.L_s * 2 * a.H;
  const float* G = a.G + (int64_t)hk * pl.nu * D * D;
  double* A = a.Ascr + (int64_t)task * p * p;
  double* B = a.Bscr + (int64_t)task * p * D;
  const double N = (double)a.N;
  const int qp = nsrc + (l * 2 + kv) * a.H + h;     // target plane
  const double* T = a.sums + (int64_t)qp * D;
  // centred design Gram + lambda I: A(i, j), i >= j, at A[j * p + i]; the
  // block of list positions (jr / D, i / D) holds it at row jr % D, column
  // i % D (at row i % D, column jr % D when the plan stores its transpose).
  // A pass takes 16 columns jr = jb + 2 u + t / 128 (u < 8) and, per 128-row
  // block q of i, row i = 128 q + t % 128; blocks above the diagonal are
  // skipped.
  {
    const int c_ = t & 127, jh = t >> 7;
#pragma unroll 1
    for (int jb = 0; jb < p; jb += 16)
#pragma unroll 1
      for (int q = jb >> 7; q < k; ++q) {
        const int i = 128 * q + c_;
        float g[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int jr = jb + 2 * u + jh, r = jr & 127;
          const uint32_t v = st[(jr >> 7) * 5 + q];
          const int64_t off = (v & kTransposed) ? c_ * D + r : r * D + c_;
          g[u] = G[(int64_t)(v & ~kTransposed) * D * D + off];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int jr = jb + 2 * u + jh;
          if (i >= jr)
            A[(int64_t)jr * p + i] = (double)g[u] - SX[i] * SX[jr] / N + (i == jr ? a.lam : 0.0);
        }
      }
  }
  // centred cross Gram B [p][128]: the cross block of list position i / D
  // holds row i % D, column c
  for (int e0 = t; e0 < p * D; e0 += 256 * 8) {
    float g[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + 256 * u, i = e / D, c = e % D;
      g[u] = G[(int64_t)st[(i / D) * 5 + 4] * D * D + (i % D) * D + c];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + 256 * u, i = e / D, c = e % D;
      B[e] = (double)g[u] - SX[i] * T[c] / N;
    }
  }
  __syncthreads();
  chol_panels(A, p, PT);
  chol_solve(A, B, p, PT);
  // outputs: W rows = input features; b = mean(Y) - mean(X) W
  float* Wo = (kv == 0 ? a.W_K : a.W_V) + ((int64_t)l * a.H + h) * p * D;
  for (int e = t; e < p * D; e += 256) Wo[e] = (float)B[e];
  if (t < D) {
    const int c = t;
    double v = T[c] / N;
    for (int i0 = 0; i0 < p; i0 += 8) {
      double w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) w[u] = B[(int64_t)(i0 + u) * D + c];
#pragma unroll
      for (int u = 0; u < 8; ++u) v -= SX[i0 + u] / N * w[u];
    }
    (kv == 0 ? a.b_K : a.b_V)[((int64_t)l * a.H + h) * D + c] = (float)v;
  }
}

// ------------------------------------------------------------------ probe

// Two workgroups per (source layer s, head, K|V), each for half of the target
// layers.  LDS holds one 128 x 128 fp64 array: the centred Gram, factored in
// place (Cholesky, lower triangle), then M = L^-1 stored transposed in the
// upper triangle and the lower triangle cleared, so that row j holds M[.][j].
// For every target layer the centred cross Gram X_c^T Y_c = X^T Y - S T^T / N
// (S, T the channel sums; X^T Y the fp32 Gram output) enters Z = M X_c^T Y_c
// on the fp64 matrix cores, and the explained sum of squares ||Z||_F^2 over
// the target's total sum of squares is the R2.
typedef double f64x4_t __attribute__((ext_vector_type(4)));
constexpr int PR_ROWS = 16;   // cross-block rows per stage of the probe's ring
constexpr int PR_NST = 3;     // stages

__global__ __launch_bounds__(256) void probe_kernel(const FitArgs a) {
  __shared__ double A[D * D];
  __shared__ double S[D], Md[D];
  __shared__ double red[8];
  __shared__ __attribute__((aligned(16))) float ring[PR_NST * PR_ROWS * D];
  const int task = blockIdx.x >> 1, half = blockIdx.x & 1;
  const int s = task % a.L_s, hk = task / a.L_s, kv = hk & 1, h = hk >> 1;
  const int nsrc = a.L_s * 2 * a.H;
  const int ps = (s * 2 + kv) * a.H + h;
  const int nbl = a.L_t + 1;
  const float* G = a.G + (int64_t)task * nbl * D * D;
  const double N = (double)a.N;
  const int t = threadIdx.x;
  if (t < D) S[t] = a.sums[(int64_t)ps * D + t];
  __syncthreads();
  for (int e = t; e < D * D; e += 256) {
    const int i = e / D, j = e - i * D;
    A[e] = j <= i ? (double)G[e] - S[i] * S[j] / N : 0.0;
  }
  __syncthreads();
  // Cholesky, right-looking, column by column, on the unscaled columns:
  // step j subtracts a_ij a_cj / a_jj from every a_ic (j < c <= i), one
  // barrier per step; a last pass scales column j by 1 / sqrt(a_jj).  Thread
  // (ty, tx) takes rows j + 1 + ty + 16 a and columns j + 1 + tx + 16 b.
  {
    const int ty = t >> 4, tx = t & 15;
    for (int j = 0; j < D - 1; ++j) {
      const double inv = 1.0 / A[j * D + j];
      for (int i = j + 1 + ty; i < D; i += 16) {
        const double li = A[i * D + j] * inv;
        for (int c = j + 1 + tx; c <= i; c += 16) A[i * D + c] = fma(-li, A[c * D + j], A[i * D + c]);
      }
      __syncthreads();
    }
    if (t < D) {
      const double rs = 1.0 / sqrt(A[t * D + t]);
      for (int i = t + 1; i < D; ++i) A[i * D + t] *= rs;
    }
    __syncthreads();
    if (t < D) A[t * D + t] = sqrt(A[t * D + t]);
    __syncthreads();
  }
  // M = L^-1, column j by thread j: M[i][j] goes to A[j][i] (i > j), the
  // diagonal to Md
  if (t < D) {
    const int j = t;
    const double mjj = 1.0 / A[j * D + j];
    Md[j] = mjj;
    for (int i = j + 1; i < D; ++i) {
      double v = A[i * D + j] * mjj;
      for (int q = j + 1; q < i; ++q) v += A[i * D + q] * A[j * D + q];
      A[j * D + i] = -v / A[i * D + i];
    }
  }
  __syncthreads();
  for (int e = t; e < D * D; e += 256) {
    const int i = e / D, j = e - i * D;
    if (j < i) A[e] = 0.0;
    else if (j == i) A[e] = Md[i];
  }
  __syncthreads();

  // The cross blocks stream through an LDS ring: stage c of this workgroup's
  // row stream holds rows 16 (c % 8) .. + 15 of the cross block of target
  // layer l0 + c / 8, loaded straight into LDS two stages ahead (each wave
  // loads 4 of the 16 rows); one barrier per stage makes them visible and
  // frees the stage loaded next.
  //
  // Z = M C_c runs on the fp64 matrix cores (16 x 16 x 4 steps), with the
  // centred cross Gram C_c = X^T Y - S T^T / N formed in fp64 as the B
  // operand, so that only the sum of squares of the result is needed.  Wave w
  // owns the 16-row blocks w and 7 - w of Z (all 128 columns), so that the
  // triangular M gives every wave the same work: a row block takes the steps
  // whose 4 rows of C meet its nonzero columns of M only.
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int li = lane & 15, lk = lane >> 4;
  const int l0 = half * ((a.L_t + 1) / 2), l1 = half ? a.L_t : (a.L_t + 1) / 2;
  const int n_st = (l1 - l0) * (D / PR_ROWS);
  const i32x4_t_ rs = rsrc(G, (uint32_t)(nbl * D * D * 4));
  const uint32_t ring0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)ring;
  auto issue = [&](int c) __attribute__((always_inline)) {
    if (c >= n_st) return;
    const int l = l0 + c / (D / PR_ROWS), j0 = PR_ROWS * (c % (D / PR_ROWS));
    const uint32_t go = (uint32_t)(((1 + l) * D + j0) * D * 4);   // byte offset of the stage's rows
    const uint32_t lb = ring0 + (uint32_t)((c % PR_NST) * PR_ROWS * D * 4);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t q = (uint32_t)(2 * wave + i) * 1024u;   // two rows per load
      const uint32_t vo = go + q + (uint32_t)lane * 16u;
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   :
                   : "s"(lb + q), "v"(vo), "s"(rs)
                   : "memory");
    }
  };
  issue(0);
  issue(1);
  const int rb[2] = {wave, 7 - wave};
  f64x4_t acc[2][8];
  double w[8];   // T[16 cb + li] / N of the current target layer
  double tq = 0.0;   // thread t < 128: channel t's centred sum of squares of the target
  for (int c = 0; c < n_st; ++c) {
    const int l = l0 + c / (D / PR_ROWS), jb = c % (D / PR_ROWS);
    const int pq = nsrc + (l * 2 + kv) * a.H + h;
    if (jb == 0) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc[u][cb] = f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) w[cb] = a.sums[(int64_t)pq * D + 16 * cb + li] / N;
      if (t < D) {
        const double sc = a.sums[(int64_t)pq * D + t];
        tq = a.sumsq[(int64_t)pq * D + t] - sc * sc / N;
      }
    }
    // this wave's loads of stage c have landed (those of stage c + 1 may
    // still be in flight); after the barrier every wave's have, and every
    // wave is done with stage c - 1, whose slot stage c + 2 takes
    if (c + 1 < n_st) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    issue(c + 2);
    const float* rg = ring + (c % PR_NST) * PR_ROWS * D;
    // the operands of the stage's four steps first, then its matrix
    // instructions back to back (they run while the next stage's operands
    // are read and converted)
    double bv[PR_ROWS / 4][8];   // B operand: C_c[k0 + lk][16 cb + li]
    double av[PR_ROWS / 4][2];   // A operand: M[16 rb + li][k0 + lk], at A[(k0 + lk) D + 16 rb + li]
#pragma unroll
    for (int kq = 0; kq < PR_ROWS / 4; ++kq) {
      const int k0 = PR_ROWS * jb + 4 * kq;   // rows k0 .. k0 + 3 of C
      const double sk = S[k0 + lk];
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) bv[kq][cb] = fma(-sk, w[cb], (double)rg[(4 * kq + lk) * D + 16 * cb + li]);
#pragma unroll
      for (int u = 0; u < 2; ++u) av[kq][u] = A[(k0 + lk) * D + 16 * rb[u] + li];
    }
#pragma unroll
    for (int kq = 0; kq < PR_ROWS / 4; ++kq) {
      const int k0 = PR_ROWS * jb + 4 * kq;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (k0 > 16 * rb[u] + 15) continue;   // M is zero there
#pragma unroll
        for (int cb = 0; cb < 8; ++cb)
          acc[u][cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[kq][u], bv[kq][cb], acc[u][cb], 0, 0, 0);
      }
    }
    if (jb != D / PR_ROWS - 1) continue;
    // the squared norm of Z = M C_c
    double ss = 0.0;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int cb = 0; cb < 8; ++cb)
#pragma unroll
        for (int q = 0; q < 4; ++q) ss = fma(acc[u][cb][q], acc[u][cb][q], ss);
    double tt = tq;   // zero on threads t >= 128
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      ss += __shfl_xor(ss, off);
      tt += __shfl_xor(tt, off);
    }
    if (lane == 0) {
      red[wave] = ss;
      red[4 + wave] = tt;
    }
    __syncthreads();
    if (t == 0) {
      const double reg = red[0] + red[1] + red[2] + red[3];
      const double tot = red[4] + red[5] + red[6] + red[7];
      a.r2[(((int64_t)s * a.L_t + l) * a.H + h) * 2 + kv] = (float)(reg / tot);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ top-k

__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ r2, int L_s, int L_t,
                                                   int H, int k, int32_t* __restrict__ out) {
  const int l = blockIdx.x * blockDim.x + threadIdx.x;
  if (l >= L_t) return;
  int best[32];
  double bs[32];
  int n = 0;
  for (int s = 0; s < L_s; ++s) {
    double v = 0.0;
    for (int h = 0; h < H; ++h)
      for (int kv = 0; kv < 2; ++kv) v += (double)r2[(((int64_t)s * L_t + l) * H + h) * 2 + kv];
    v /= (double)(2 * H);
    // insert into the descending list; an equal score keeps the earlier
    // (lower) source index ahead
    int pos = n;
    while (pos > 0 && bs[pos - 1] < v) --pos;
    if (pos < k) {
      const int last = n < k ? n : k - 1;
      for (int q = last; q > pos; --q) {
        bs[q] = bs[q - 1];
        best[q] = best[q - 1];
      }
      bs[pos] = v;
      best[pos] = s;
      if (n < k) ++n;
    }
  }
  // ascending source order
  for (int i = 1; i < k; ++i)
    for (int q = i; q > 0 && best[q - 1] > best[q]; --q) {
      const int tmp = best[q];
      best[q] = best[q - 1];
      best[q - 1] = tmp;
    }
  for (int i = 0; i < k; ++i) out[(int64_t)l * k + i] = best[i];
}

}  // namespace

size_t fit_plan_bytes(int L_t, int k) {
  const size_t up = 256;
  auto r = [&](size_t n) { return (n + up - 1) / up * up; };
  const size_t items = (size_t)L_t * (size_t)(k * (k + 3) / 2);   // at most one job per item
  return r((size_t)L_t * sizeof(LayerRec)) + r(items * 8 * sizeof(uint32_t)) +
         r((size_t)L_t * kEnt * sizeof(uint32_t));
}

void fit_plan_count(const FitArgs& a, int* n_blocks, int* n_jobs) {
  int nu = 0, nj = 0;
  LayerRec r;
  for (int l = 0; l < a.L_t; ++l) {
    nj += plan_layer(a.idx, a.k, l, r);
    nu += r.n_items;
  }
  *n_blocks = nu;
  *n_jobs = nj;
}

int gram_jobs(const FitArgs& a) {
  if (a.mode == 0) {
    int nu, nj;
    fit_plan_count(a, &nu, &nj);
    return a.H * 2 * nj;
  }
  const int n_sp = (a.L_s + 1) / 2, n_lp = (a.L_t + 1) / 2;
  return a.H * 2 * (n_sp * n_lp + (a.L_s + 3) / 4);
}

hipError_t launch_fit(FitArgs a, void* plan, bool prep, hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  FitPlan p{};
  if (a.mode == 0) {
    if (plan == nullptr) return hipErrorInvalidValue;
    const size_t up = 256;
    auto r = [&](size_t n) { return (n + up - 1) / up * up; };
    const size_t items = (size_t)a.L_t * (size_t)(a.k * (a.k + 3) / 2);
    char* base = static_cast<char*>(plan);
    p.lay = reinterpret_cast<LayerRec*>(base);
    p.jobs = reinterpret_cast<uint32_t*>(base + r((size_t)a.L_t * sizeof(LayerRec)));
    p.stab = reinterpret_cast<uint32_t*>(base + r((size_t)a.L_t * sizeof(LayerRec)) +
                                         r(items * 8 * sizeof(uint32_t)));
    fit_plan_count(a, &p.nu, &p.nj);
    // without a prep the plan takes a launch of its own
    if (!prep) hipLaunchKernelGGL(fit_plan_kernel, dim3(1), dim3(256), 0, stream, a, p);
  }
  if (prep) {
    const int units = (a.P / a.H) * prep_chunks(a.Npad);
    const int blocks = 8 * a.H * ((units + 7) / 8);
    const int plan_block = a.mode == 0 ? blocks : -1;   // one more block for the plan
    hipLaunchKernelGGL(fit_prep_kernel, dim3(blocks + (a.mode == 0 ? 1 : 0)), dim3(256), 0, stream,
                       a, p, plan_block);
    if (prep_chunks(a.Npad) > 1)
      hipLaunchKernelGGL(fit_sums_kernel, dim3((a.P * D + 255) / 256), dim3(256), 0, stream, a);
  }
  a.n_jobs = gram_jobs(a);
  a.jobs_per_xcd = (a.n_jobs + 7) / 8;
  hipLaunchKernelGGL(gram_kernel, dim3(8 * a.jobs_per_xcd), dim3(256), 0, stream, a, p);
  if (a.mode == 0) {
    hipLaunchKernelGGL(fit_solve_kernel, dim3(a.L_t * a.H * 2), dim3(256), 0, stream, a, p);
  } else {
    hipLaunchKernelGGL(probe_kernel, dim3(2 * a.L_s * a.H * 2), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_fit(FitArgs a, bool prep, hipStream_t stream) {
  return launch_fit(a, nullptr, prep, stream);
}

hipError_t launch_topk(const float* r2, int L_s, int L_t, int H, int k, int32_t* out,
                       hipStream_t stream) {
  hipLaunchKernelGGL(topk_kernel, dim3((L_t + 255) / 256), dim3(256), 0, stream, r2, L_s, L_t, H,
                     k, out);
  return hipGetLastError();
}

}  // namespace kvx
