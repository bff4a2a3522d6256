// Fitting side of the mapper: the whole per-head ridge fit (Sec. 3.1, Eq.
// Wstar with centring, from two models' caches of the same calibration
// tokens, Sec. 3.3 for the keys) and the single-source linear probe that
// chooses the source layers (Sec. 2.3, Eq. single_source_ols; Sec. 3.2).
//
// Both reduce to Gram matrices of per-token head features, then small SPD
// solves:
//   fit_prep_kernel   per (layer, K|V, head) plane of either cache: strip the
//                     RoPE from keys (fp32 coefficients) and keep each
//                     stripped key as a bf16 pair hi + lo (the lo planes
//                     follow the planes), write the plane token-tiled (each
//                     16-token step of a plane is one contiguous 4 KB slab:
//                     128 channel rows of 16 tokens), and sum every channel
//                     and its square (fp64) for the centring;
//   gram_kernel       batched 128 x 128 blocks P_a^T P_b of those planes on the
//                     matrix cores (bf16 operands, fp32 accumulation), one job
//                     = up to four blocks (one per wave) over at most four
//                     planes, which stream through an LDS ring of slabs; key
//                     blocks add hi.hi + hi.lo + lo.hi in the same sweep;
//   fit_solve_kernel  per (target layer, head, K|V): the centred design Gram
//                     plus lambda I, Cholesky in fp64 (32-column panels in
//                     LDS), forward and backward substitution for the
//                     centred cross Gram, the bias from the means;
//   probe_kernel      per (source layer, head, K|V): Cholesky and inverse of
//                     the centred Gram of that plane in LDS, then for every
//                     target layer the explained sum of squares
//                     ||L^-1 X_c^T Y_c||_F^2 over the total sum of squares;
//   topk_kernel       per target layer: the top-k source layers by R2
//                     averaged over heads and over keys and values.
#include "kvx_bf16.h"
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

// Order of a fit task's blocks (a, b): b < 4 is source plane P_b of idx[l],
// b == 4 the target plane Q.  Chunks of four are one Gram job each; the order
// keeps every job within five distinct planes in each of the three key
// passes (hi.hi, hi.lo, lo.hi).
__constant__ uint8_t kBlockOrder[4][14] = {
    {0x00, 0x04},
    {0x00, 0x01, 0x04, 0x11, 0x14},
    {0x00, 0x01, 0x02, 0x04, 0x11, 0x12, 0x14, 0x22, 0x24},
    {0x00, 0x01, 0x02, 0x03, 0x11, 0x12, 0x13, 0x14, 0x22, 0x23, 0x24, 0x04, 0x33, 0x34}};

// ------------------------------------------------------------------ prep

__global__ __launch_bounds__(256) void fit_prep_kernel(const FitArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[64 * TP];  // [token][channel]
  __shared__ double red[2][4][D];
  const int pid = blockIdx.x;
  const int nsrc = a.L_s * 2 * a.H;
  const bool is_src = pid < nsrc;
  const int q = is_src ? pid : pid - nsrc;                 // plane within its cache
  const bool keys = ((q / a.H) & 1) == 0;
  const uint16_t* plane = (is_src ? a.src : a.tgt) + (int64_t)q * a.N * D;
  const float2* cs = is_src ? a.cs_src : a.cs_tgt;
  uint16_t* out = a.planes + (int64_t)pid * D * a.Npad;
  // keys also get the rounding residual: plane hi + lo carries the stripped
  // key to about 16 significant bits
  uint16_t* out_lo = a.planes + (int64_t)(a.P + lo_slot(a, pid)) * D * a.Npad;
  __shared__ __attribute__((aligned(16))) uint16_t tile_lo[64 * TP];
  const int t = threadIdx.x;
  const int g = t & 7;         // channels 8g .. 8g+7 and 64+8g .. 64+8g+7
  const int tk = t >> 3;       // token within half a pass
  double s1[16], s2[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) s1[e] = s2[e] = 0.0;
  for (int t0 = 0; t0 < a.Npad; t0 += 64) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int row = tk + 32 * it;
      const int tok = t0 + row;
      uint4 x = make_uint4(0u, 0u, 0u, 0u), y = x, xl = x, yl = x;
      if (tok < a.N) {
        x = *reinterpret_cast<const uint4*>(plane + (int64_t)tok * D + 8 * g);
        y = *reinterpret_cast<const uint4*>(plane + (int64_t)tok * D + 64 + 8 * g);
        if (keys) {
          uint32_t* px = reinterpret_cast<uint32_t*>(&x);
          uint32_t* py = reinterpret_cast<uint32_t*>(&y);
          const float2* c = cs + (int64_t)tok * (D / 2);
          if (a.style == 0) {
            // plane j = (channel j, channel j + 64): x holds the first members
            // of planes 8g .. 8g+7, y the second ones
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              float u0 = lo_bf16(px[w]), u1 = hi_bf16(px[w]);
              float v0 = lo_bf16(py[w]), v1 = hi_bf16(py[w]);
              const float2 c0 = c[8 * g + 2 * w], c1 = c[8 * g + 2 * w + 1];
              const float nu0 = u0 * c0.x + v0 * c0.y, nv0 = v0 * c0.x - u0 * c0.y;
              const float nu1 = u1 * c1.x + v1 * c1.y, nv1 = v1 * c1.x - u1 * c1.y;
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
              const float2 cx = c[4 * g + w], cy = c[32 + 4 * g + w];
              float u = lo_bf16(px[w]), v = hi_bf16(px[w]);
              float nu = u * cx.x + v * cx.y, nv = v * cx.x - u * cx.y;
              px[w] = pack2(nu, nv);
              reinterpret_cast<uint32_t*>(&xl)[w] = pack2(nu - lo_bf16(px[w]), nv - hi_bf16(px[w]));
              u = lo_bf16(py[w]);
              v = hi_bf16(py[w]);
              nu = u * cy.x + v * cy.y;
              nv = v * cy.x - u * cy.y;
              py[w] = pack2(nu, nv);
              reinterpret_cast<uint32_t*>(&yl)[w] = pack2(nu - lo_bf16(py[w]), nv - hi_bf16(py[w]));
            }
          }
        }
      }
      const uint32_t* px = reinterpret_cast<const uint32_t*>(&x);
      const uint32_t* py = reinterpret_cast<const uint32_t*>(&y);
      const uint32_t* pxl = reinterpret_cast<const uint32_t*>(&xl);
      const uint32_t* pyl = reinterpret_cast<const uint32_t*>(&yl);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        // the values the Gram sees: hi + lo (lo is zero for values)
        const double xa = (double)lo_bf16(px[w]) + lo_bf16(pxl[w]);
        const double xb = (double)hi_bf16(px[w]) + hi_bf16(pxl[w]);
        const double ya = (double)lo_bf16(py[w]) + lo_bf16(pyl[w]);
        const double yb = (double)hi_bf16(py[w]) + hi_bf16(pyl[w]);
        s1[2 * w] += xa;  s2[2 * w] += xa * xa;
        s1[2 * w + 1] += xb;  s2[2 * w + 1] += xb * xb;
        s1[8 + 2 * w] += ya;  s2[8 + 2 * w] += ya * ya;
        s1[9 + 2 * w] += yb;  s2[9 + 2 * w] += yb * yb;
      }
      *reinterpret_cast<uint4*>(tile + row * TP + 8 * g) = x;
      *reinterpret_cast<uint4*>(tile + row * TP + 64 + 8 * g) = y;
      if (keys) {
        *reinterpret_cast<uint4*>(tile_lo + row * TP + 8 * g) = xl;
        *reinterpret_cast<uint4*>(tile_lo + row * TP + 64 + 8 * g) = yl;
      }
    }
    __syncthreads();
    // token-tiled write: the 64 tokens are 4 slabs; wave q writes slab q (4 KB
    // contiguous), lane -> 16-byte pieces m = 4 lane .. 4 lane + 3, piece m =
    // (row r = m / 2, position m % 2) holding token chunk (m % 2) ^ swz(r)
    {
      const int q = t >> 6, lane = t & 63;
      const int64_t so = (int64_t)(t0 / TS + q) * (D * TS);   // element offset of the slab
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 4 * lane + i, r = m >> 1, c = (m & 1) ^ swz(r);
        const int tok = TS * q + 8 * c;
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = (uint32_t)tile[(tok + 2 * e) * TP + r] | ((uint32_t)tile[(tok + 2 * e + 1) * TP + r] << 16);
        *reinterpret_cast<uint4*>(out + so + 8 * m) = make_uint4(w[0], w[1], w[2], w[3]);
        if (keys) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            w[e] = (uint32_t)tile_lo[(tok + 2 * e) * TP + r] |
                   ((uint32_t)tile_lo[(tok + 2 * e + 1) * TP + r] << 16);
          *reinterpret_cast<uint4*>(out_lo + so + 8 * m) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
    }
    __syncthreads();
  }
  // channel sums: lanes of a wave with the same g are 8 apart
#pragma unroll
  for (int e = 0; e < 16; ++e) {
#pragma unroll
    for (int off = 8; off < 64; off <<= 1) {
      s1[e] += __shfl_xor(s1[e], off);
      s2[e] += __shfl_xor(s2[e], off);
    }
  }
  const int wave = t >> 6, lane = t & 63;
  if (lane < 8) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int ch = e < 8 ? 8 * lane + e : 64 + 8 * lane + (e - 8);
      red[0][wave][ch] = s1[e];
      red[1][wave][ch] = s2[e];
    }
  }
  __syncthreads();
  if (t < D) {
    a.sums[(int64_t)pid * D + t] = red[0][0][t] + red[0][1][t] + red[0][2][t] + red[0][3][t];
    a.sumsq[(int64_t)pid * D + t] = red[1][0][t] + red[1][1][t] + red[1][2][t] + red[1][3][t];
  }
}

// ------------------------------------------------------------------ Gram

// Jobs.  A fit task (target layer l, head h, K|V) needs the blocks
// kBlockOrder[k-1][e] of its k source planes P_0 .. P_{k-1} (idx[l] order)
// and the target plane Q; chunks of four are one job each, and every chunk
// touches at most four distinct planes.  Tasks run head-major, then K|V, then
// target layer, so each XCD's contiguous job range holds one head's key and
// value tasks.  A probe group (head h, K|V) needs P_s^T P_s and P_s^T Q_l for
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

__device__ __forceinline__ GJob decode_job(const FitArgs& a, int job, int wave) {
  GJob j;
  j.np = 0;
  j.sa = j.sb = -1;
  j.out = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) j.pid[i] = 0;
  const int nsrc = a.L_s * 2 * a.H;
  if (a.mode == 0) {
    const int k = a.k;
    const int nbl = k * (k + 3) / 2;
    const int nch = (nbl + 3) / 4;
    const int task = job / nch, ch = job - task * nch;
    const int l = task % a.L_t, hk = task / a.L_t, kv = hk & 1, h = hk >> 1;
    j.keys = kv == 0;
    const int nblk = nbl - 4 * ch < 4 ? nbl - 4 * ch : 4;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (w >= nblk) continue;
      const int e = 4 * ch + w;
      const int pr = kBlockOrder[k - 1][e], ai = pr >> 4, bi = pr & 15;
      const int pa = ((int)a.idx[l * k + ai] * 2 + kv) * a.H + h;
      const int pb = bi == 4 ? nsrc + (l * 2 + kv) * a.H + h : ((int)a.idx[l * k + bi] * 2 + kv) * a.H + h;
      const int sa = add_plane(j, pa), sb = add_plane(j, pb);
      if (w == wave) {
        j.sa = sa;
        j.sb = sb;
        j.out = (int64_t)task * nbl + e;
      }
    }
  } else {
    const int per = probe_jobs_per_group(a);
    const int grp = job / per, c = job - grp * per;
    const int h = grp >> 1, kv = grp & 1;
    j.keys = kv == 0;
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

// wait until at most n (<= 24) loads of this wave are in flight
__device__ __forceinline__ void vm_wait_upto(int n) {
  switch (n) {
    case 0: vm_wait_n<0>(); break;
    case 1: vm_wait_n<1>(); break;
    case 2: vm_wait_n<2>(); break;
    case 3: vm_wait_n<3>(); break;
    case 4: vm_wait_n<4>(); break;
    case 5: vm_wait_n<5>(); break;
    case 6: vm_wait_n<6>(); break;
    case 7: vm_wait_n<7>(); break;
    case 8: vm_wait_n<8>(); break;
    case 9: vm_wait_n<9>(); break;
    case 10: vm_wait_n<10>(); break;
    case 11: vm_wait_n<11>(); break;
    case 12: vm_wait_n<12>(); break;
    case 13: vm_wait_n<13>(); break;
    case 14: vm_wait_n<14>(); break;
    case 15: vm_wait_n<15>(); break;
    case 16: vm_wait_n<16>(); break;
    case 17: vm_wait_n<17>(); break;
    case 18: vm_wait_n<18>(); break;
    case 19: vm_wait_n<19>(); break;
    case 20: vm_wait_n<20>(); break;
    case 21: vm_wait_n<21>(); break;
    case 22: vm_wait_n<22>(); break;
    case 23: vm_wait_n<23>(); break;
    default: vm_wait_n<24>(); break;
  }
}

// One job: four waves, one 128 x 128 block each (4 x 4 accumulators of
// v_mfma_f32_32x32x16_bf16, 256 AGPRs), over all tokens in 16-token steps.
// A stage of the LDS ring holds the step's slab of every plane of the job
// (and of its residual plane for keys): 8 slabs (keys, 4 stages) or 4
// (values, 8 stages).  Each wave loads one 1 KB quarter of every slab straight
// into LDS.  Step s: wait for this wave's loads of step s + 1, barrier (step
// s + 1 landed for every wave; the stage of step s - 1 was last read during
// step s - 2), load step s + NST - 1 into that stage, read step s + 1's
// fragments and run step s's matrix instructions on the fragments read during
// step s - 1.  Key blocks add hi.hi + hi.lo + lo.hi in the same step.
template <bool KEYS>
__device__ __forceinline__ void gram_job(const FitArgs& a, const GJob& jb, uint32_t lds0, int lane,
                                         int wave) {
  constexpr int NSL = KEYS ? 8 : 4;            // slab slots per stage
  constexpr int SBY = NSL * SLAB;              // stage bytes
  constexpr int NST = RING / SBY;              // stages: 4 or 8
  constexpr int NF = KEYS ? 16 : 8;            // fragments per step
  const int nsl = KEYS ? 2 * jb.np : jb.np;    // slabs this job loads per step
  const int total = a.Npad / TS;
  const uint32_t plane_bytes = (uint32_t)(D * a.Npad * 2);

  // slab i of a step: keys: plane pid[i / 2] (i even) or its residual (i odd);
  // values: plane pid[i]
  i32x4_t_ rs[NSL];
#pragma unroll
  for (int i = 0; i < NSL; ++i) {
    int p = jb.pid[KEYS ? (i >> 1) : i];
    if (KEYS && (i & 1)) p = a.P + lo_slot(a, p);
    rs[i] = rsrc(a.planes + (int64_t)p * D * a.Npad, plane_bytes);
  }
  auto issue = [&](int st) __attribute__((always_inline)) {
    const uint32_t base = lds0 + (uint32_t)((st % NST) * SBY + wave * 1024);
    const uint32_t vo = (uint32_t)st * SLAB + (uint32_t)(wave * 1024 + lane * 16);
#pragma unroll
    for (int i = 0; i < NSL; ++i)
      if (i < nsl)
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
  typedef const __attribute__((address_space(3))) bf16x8_t_* lp_t;
  // fragments: A hi 0..3, B hi 4..7, A lo 8..11, B lo 12..15
  auto read_step = [&](int st, bf16x8_t_* f) __attribute__((always_inline)) {
    const uint32_t sbase = lds0 + (uint32_t)((st % NST) * SBY);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[i] = *reinterpret_cast<lp_t>((uintptr_t)(sbase + oah + 1024 * i));
      f[4 + i] = *reinterpret_cast<lp_t>((uintptr_t)(sbase + obh + 1024 * i));
      if (KEYS) {
        f[8 + i] = *reinterpret_cast<lp_t>((uintptr_t)(sbase + oah + SLAB + 1024 * i));
        f[12 + i] = *reinterpret_cast<lp_t>((uintptr_t)(sbase + obh + SLAB + 1024 * i));
      }
    }
  };
  auto mfma_step = [&](const bf16x8_t_* g) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jx = 0; jx < 4; ++jx)
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc[4 * i + jx]) : "v"(g[i]), "v"(g[4 + jx]));
    if (KEYS) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jx = 0; jx < 4; ++jx)
          asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc[4 * i + jx]) : "v"(g[i]), "v"(g[12 + jx]));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jx = 0; jx < 4; ++jx)
          asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc[4 * i + jx]) : "v"(g[8 + i]), "v"(g[4 + jx]));
    }
  };
  bf16x8_t_ fa[NF], fb[NF];
  auto step = [&](int s, bf16x8_t_* cur, bf16x8_t_* nxt) __attribute__((always_inline)) {
    if (s + 1 < total) {
      int later = total - 2 - s;
      if (later > NST - 3) later = NST - 3;
      vm_wait_upto(nsl * later);
    }
    __syncthreads();
    if (s + NST - 1 < total) issue(s + NST - 1);
    if (active) {
      if (s + 1 < total) read_step(s + 1, nxt);
      mfma_step(cur);
    }
  };

  // prologue: steps 0 .. NST - 2 in flight; step 0 landed everywhere
  for (int st = 0; st < NST - 1 && st < total; ++st) issue(st);
  vm_wait_upto(nsl * (NST - 2 < total - 1 ? NST - 2 : total - 1));
  __syncthreads();
  if (active) read_step(0, fa);
  int s = 0;
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
void gram_kernel(const FitArgs a) {
  __shared__ __attribute__((aligned(256))) char smem[RING];
  const int xcd = blockIdx.x & 7, qx = blockIdx.x >> 3;
  const int job = xcd * a.jobs_per_xcd + qx;   // an XCD takes a contiguous range of jobs
  if (job >= a.n_jobs) return;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const GJob jb = decode_job(a, job, wave);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)smem;
  if (jb.keys) gram_job<true>(a, jb, lds0, lane, wave);
  else gram_job<false>(a, jb, lds0, lane, wave);
}

// ------------------------------------------------------------ fit solve

// Cholesky of the p x p matrix A (lower triangle, row-major, fp64, in global
// memory) in place, in 32-column panels held in LDS.
__device__ void chol_panels(double* A, int p, double* P /* LDS [512][NB + 1] */) {
  const int t = threadIdx.x;
  constexpr int LD = NB + 1;
  for (int J = 0; J < p; J += NB) {
    const int R = p - J;
    for (int e = t; e < R * NB; e += 256) {
      const int r = e / NB, c = e - r * NB;
      P[r * LD + c] = A[(int64_t)(J + r) * p + J + c];
    }
    __syncthreads();
    for (int c = 0; c < NB; ++c) {
      const double dg = sqrt(P[c * LD + c]);
      for (int r = c + 1 + t; r < R; r += 256) P[r * LD + c] /= dg;
      __syncthreads();
      if (t == 0) P[c * LD + c] = dg;
      // the panel's later columns
      const int nc = NB - 1 - c;
      for (int e = t; e < (R - c - 1) * nc; e += 256) {
        const int r = c + 1 + e / nc, c2 = c + 1 + e % nc;
        if (r >= c2) P[r * LD + c2] -= P[r * LD + c] * P[c2 * LD + c];
      }
      __syncthreads();
    }
    for (int e = t; e < R * NB; e += 256) {
      const int r = e / NB, c = e - r * NB;
      if (r >= c) A[(int64_t)(J + r) * p + J + c] = P[r * LD + c];
    }
    // trailing update of rows and columns J + NB .. p - 1 (lower triangle),
    // 4 x 4 tiles per thread
    const int R2 = R - NB;
    const int nbk = (R2 + 3) / 4;
    for (int tile = t; tile < nbk * nbk; tile += 256) {
      const int bi = tile / nbk, bj = tile - bi * nbk;
      if (bj > bi) continue;
      double s[4][4];
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) s[x][y] = 0.0;
      for (int c = 0; c < NB; ++c) {
        double li[4], lj[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const int ri = NB + 4 * bi + x, rj = NB + 4 * bj + x;
          li[x] = ri < R ? P[ri * LD + c] : 0.0;
          lj[x] = rj < R ? P[rj * LD + c] : 0.0;
        }
#pragma unroll
        for (int x = 0; x < 4; ++x)
#pragma unroll
          for (int y = 0; y < 4; ++y) s[x][y] += li[x] * lj[y];
      }
#pragma unroll
      for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 4; ++y) {
          const int i = J + NB + 4 * bi + x, j = J + NB + 4 * bj + y;
          if (i < p && j <= i) A[(int64_t)i * p + j] -= s[x][y];
        }
    }
    __syncthreads();
  }
}

// Z = L^-1 B (forward), then W = L^-T Z (backward), in place in B [p][128],
// L in the lower triangle of A.  Thread t owns column t % 128; the two
// threads of a column split the update rows.
__device__ void chol_solve(const double* A, double* B, int p, double* P /* LDS */) {
  const int t = threadIdx.x, c = t & 127, half = t >> 7;
  constexpr int LD = NB + 1;
  double z[NB];
  for (int J = 0; J < p; J += NB) {
    const int R = p - J;
    for (int e = t; e < R * NB; e += 256) {
      const int r = e / NB, cc = e - r * NB;
      P[r * LD + cc] = A[(int64_t)(J + r) * p + J + cc];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < NB; ++r) {
      double v = B[(int64_t)(J + r) * D + c];
#pragma unroll
      for (int r2 = 0; r2 < r; ++r2) v -= P[r * LD + r2] * z[r2];
      z[r] = v / P[r * LD + r];
    }
    __syncthreads();
    if (half == 0)
#pragma unroll
      for (int r = 0; r < NB; ++r) B[(int64_t)(J + r) * D + c] = z[r];
    for (int i = J + NB + half; i < p; i += 2) {
      double v = B[(int64_t)i * D + c];
#pragma unroll
      for (int r = 0; r < NB; ++r) v -= P[(i - J) * LD + r] * z[r];
      B[(int64_t)i * D + c] = v;
    }
    __syncthreads();
  }
  // backward: block row J (rows J .. J+NB-1, columns 0 .. J+NB-1) in LDS
  for (int J = p - NB; J >= 0; J -= NB) {
    const int W = J + NB;
    for (int e = t; e < NB * W; e += 256) {
      const int r = e / W, cc = e - r * W;
      P[r * 513 + cc] = A[(int64_t)(J + r) * p + cc];
    }
    __syncthreads();
#pragma unroll
    for (int r = NB - 1; r >= 0; --r) {
      double v = B[(int64_t)(J + r) * D + c];
#pragma unroll
      for (int r2 = r + 1; r2 < NB; ++r2) v -= P[r2 * 513 + J + r] * z[r2];
      z[r] = v / P[r * 513 + J + r];
    }
    __syncthreads();
    if (half == 0)
#pragma unroll
      for (int r = 0; r < NB; ++r) B[(int64_t)(J + r) * D + c] = z[r];
    for (int i = half; i < J; i += 2) {
      double v = B[(int64_t)i * D + c];
#pragma unroll
      for (int r = 0; r < NB; ++r) v -= P[r * 513 + i] * z[r];
      B[(int64_t)i * D + c] = v;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void fit_solve_kernel(const FitArgs a) {
  __shared__ double P[512 * (NB + 1)];   // 132 KB: a 512 x 33 panel or a 32 x 513 block row
  const int task = blockIdx.x;
  const int k = a.k, p = k * D;
  const int l = task % a.L_t, hk = task / a.L_t, kv = hk & 1, h = hk >> 1;
  const int nbl = k * (k + 3) / 2;
  // position of pair (a, b) (b == 4: the target plane) in the block order
  __shared__ int8_t pos[4][5];
  if (threadIdx.x < 20) pos[threadIdx.x / 5][threadIdx.x % 5] = -1;
  __syncthreads();
  if (threadIdx.x < nbl) {
    const int pr = kBlockOrder[k - 1][threadIdx.x];
    pos[pr >> 4][pr & 15] = (int8_t)threadIdx.x;
  }
  __syncthreads();
  const int nsrc = a.L_s * 2 * a.H;
  const float* G = a.G + (int64_t)task * nbl * D * D;
  double* A = a.Ascr + (int64_t)task * p * p;
  double* B = a.Bscr + (int64_t)task * p * D;
  const double N = (double)a.N;
  const int qp = nsrc + (l * 2 + kv) * a.H + h;     // target plane
  const double* T = a.sums + (int64_t)qp * D;
  // centred design Gram + lambda I (lower triangle) and centred cross Gram
  for (int e = threadIdx.x; e < p * p; e += 256) {
    const int i = e / p, j = e - i * p;
    if (j > i) continue;
    const int ai = i / D, bj = j / D, ii = i % D, jj = j % D;
    // block (bj, ai) = P_bj^T P_ai holds entry [jj][ii] (bj <= ai)
    const int eb = pos[bj][ai];
    const double g = G[(int64_t)eb * D * D + jj * D + ii];
    const double si = a.sums[(int64_t)(((int)a.idx[l * k + ai] * 2 + kv) * a.H + h) * D + ii];
    const double sj = a.sums[(int64_t)(((int)a.idx[l * k + bj] * 2 + kv) * a.H + h) * D + jj];
    A[(int64_t)i * p + j] = g - si * sj / N + (i == j ? a.lam : 0.0);
  }
  for (int e = threadIdx.x; e < p * D; e += 256) {
    const int i = e / D, c = e - i * D;
    const int ai = i / D, ii = i % D;
    const double g = G[(int64_t)pos[ai][4] * D * D + ii * D + c];
    const double si = a.sums[(int64_t)(((int)a.idx[l * k + ai] * 2 + kv) * a.H + h) * D + ii];
    B[e] = g - si * T[c] / N;
  }
  __syncthreads();
  chol_panels(A, p, P);
  chol_solve(A, B, p, P);
  // outputs: W rows = input features; b = mean(Y) - mean(X) W
  float* Wo = (kv == 0 ? a.W_K : a.W_V) + ((int64_t)l * a.H + h) * p * D;
  for (int e = threadIdx.x; e < p * D; e += 256) Wo[e] = (float)B[e];
  if (threadIdx.x < D) {
    const int c = threadIdx.x;
    double v = T[c] / N;
    for (int i = 0; i < p; ++i) {
      const int ai = i / D, ii = i % D;
      const double si = a.sums[(int64_t)(((int)a.idx[l * k + ai] * 2 + kv) * a.H + h) * D + ii];
      v -= si / N * B[(int64_t)i * D + c];
    }
    (kv == 0 ? a.b_K : a.b_V)[((int64_t)l * a.H + h) * D + c] = (float)v;
  }
}

// ------------------------------------------------------------------ probe

__device__ __forceinline__ int tri(int i) { return i * (i + 1) / 2; }

__global__ __launch_bounds__(256) void probe_kernel(const FitArgs a) {
  __shared__ double Lp[D * (D + 1) / 2];   // Cholesky factor, packed lower
  __shared__ double Mp[D * (D + 1) / 2];   // its inverse, packed lower
  __shared__ double S[D];
  __shared__ double red[4];
  const int task = blockIdx.x;
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
    if (j <= i) Lp[tri(i) + j] = (double)G[i * D + j] - S[i] * S[j] / N;
  }
  __syncthreads();
  // Cholesky, right-looking
  for (int j = 0; j < D; ++j) {
    const double dg = sqrt(Lp[tri(j) + j]);
    __syncthreads();
    for (int i = j + 1 + t; i < D; i += 256) Lp[tri(i) + j] /= dg;
    if (t == 0) Lp[tri(j) + j] = dg;
    __syncthreads();
    const int n = D - 1 - j;
    for (int e = t; e < n * n; e += 256) {
      const int i = j + 1 + e / n, c = j + 1 + e % n;
      if (c <= i) Lp[tri(i) + c] -= Lp[tri(i) + j] * Lp[tri(c) + j];
    }
    __syncthreads();
  }
  // M = L^-1, column j by thread j
  if (t < D) {
    const int j = t;
    Mp[tri(j) + j] = 1.0 / Lp[tri(j) + j];
    for (int i = j + 1; i < D; ++i) {
      double v = 0.0;
      for (int q = j; q < i; ++q) v += Lp[tri(i) + q] * Mp[tri(q) + j];
      Mp[tri(i) + j] = -v / Lp[tri(i) + i];
    }
  }
  __syncthreads();
  // every target layer: Z = M (X_c^T Y_c); thread -> column c, rows of its half
  const int c = t & 127, half = t >> 7;
  const int i0 = half * 64;
  for (int l = 0; l < a.L_t; ++l) {
    const int pq = nsrc + (l * 2 + kv) * a.H + h;
    const double Tc = a.sums[(int64_t)pq * D + c];
    const float* Gb = G + (int64_t)(1 + l) * D * D;
    double z[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) z[i] = 0.0;
    for (int jq = 0; jq < i0 + 64; ++jq) {
      const double b = (double)Gb[jq * D + c] - S[jq] * Tc / N;
#pragma unroll
      for (int i = 0; i < 64; ++i)
        if (i0 + i >= jq) z[i] += Mp[tri(i0 + i) + jq] * b;
    }
    double ss = 0.0;
#pragma unroll
    for (int i = 0; i < 64; ++i) ss += z[i] * z[i];
    // sum over the 256 threads
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) ss += __shfl_xor(ss, off);
    if ((t & 63) == 0) red[t >> 6] = ss;
    __syncthreads();
    if (t == 0) {
      const double reg = red[0] + red[1] + red[2] + red[3];
      double tot = 0.0;
      for (int cc = 0; cc < D; ++cc) {
        const double sc = a.sums[(int64_t)pq * D + cc];
        tot += a.sumsq[(int64_t)pq * D + cc] - sc * sc / N;
      }
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

int gram_jobs(const FitArgs& a) {
  if (a.mode == 0) {
    const int nbl = a.k * (a.k + 3) / 2;
    return a.L_t * a.H * 2 * ((nbl + 3) / 4);
  }
  const int n_sp = (a.L_s + 1) / 2, n_lp = (a.L_t + 1) / 2;
  return a.H * 2 * (n_sp * n_lp + (a.L_s + 3) / 4);
}

hipError_t launch_fit(FitArgs a, bool prep, hipStream_t stream) {
  if (a.N == 0) return hipSuccess;
  if (prep) hipLaunchKernelGGL(fit_prep_kernel, dim3(a.P), dim3(256), 0, stream, a);
  a.n_jobs = gram_jobs(a);
  a.jobs_per_xcd = (a.n_jobs + 7) / 8;
  hipLaunchKernelGGL(gram_kernel, dim3(8 * a.jobs_per_xcd), dim3(256), 0, stream, a);
  if (a.mode == 0)
    hipLaunchKernelGGL(fit_solve_kernel, dim3(a.L_t * a.H * 2), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(probe_kernel, dim3(a.L_s * a.H * 2), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_topk(const float* r2, int L_s, int L_t, int H, int k, int32_t* out,
                       hipStream_t stream) {
  hipLaunchKernelGGL(topk_kernel, dim3((L_t + 255) / 256), dim3(256), 0, stream, r2, L_s, L_t, H,
                     k, out);
  return hipGetLastError();
}

}  // namespace kvx
