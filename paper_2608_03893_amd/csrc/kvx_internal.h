// Internal interface between the host API (kvx_api.hip) and the kernels
// (kvx_kernels.hip).  Not installed; the public ABI is include/kvx.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvx.h"

namespace kvx {

// Records the text of a non-OK status for kvx_last_error() on the calling
// thread and returns the status (printf-style message).
kvx_status set_error(kvx_status st, const char* fmt, ...);

constexpr int kMaxIdx = 2048;   // L_t * k entries carried in the kernel arguments
constexpr int kMaxHalf = 64;    // d / 2 for the largest supported head dimension

// Plane frequencies of one RoPE, computed on the host in float64.
struct InvFreq {
  double w[kMaxHalf];
};

// Arguments of one map launch.  The source-layer index table travels by value
// (one byte per entry) so a launch needs no host-to-device copy.
struct MapArgs {
  const void* src;        // [L_s, 2, H, T, d]
  const void* wk;         // [L_t, H, k*d, d]
  const void* wv;
  const void* bk;         // [L_t, H, d] or nullptr
  const void* bv;
  const float2* cs_src;   // [T, d/2] (cos, sin) of the source RoPE
  const float2* cs_tgt;   // [T, d/2] (cos, sin) of the target RoPE
  const void* cs16;       // [T, d/2] (cos, sin) of the source RoPE as fp16 pairs
  const void* cs16_tgt;   // [T, d/2] (cos, sin) of the target RoPE as fp16 pairs
  const void* wpack;      // packed map images [L_t, H, 2, d, k*d] (W-stationary kernel)
  void* tgt;              // [L_t, 2, H, rows, d]
  const int32_t* slots;   // [T] or nullptr (dense)
  int64_t tgt_rows;       // T (dense) or num_slots (slot-addressed)
  int32_t H, T, k;
  int32_t l0;             // first target layer of this launch
  int32_t nl;             // number of target layers in this launch
  int32_t range_len;      // tokens per workgroup (W-stationary kernel)
  int32_t wave_tokens;    // tokens per wave per tile, 32 or 64 (W-stationary kernel)
  uint8_t idx[kMaxIdx];   // idx[(l - l0) * k + i]
};

// Fills cs_src and (unless same) cs_tgt with float32 (cos, sin) pairs, and
// cs16 / (unless same) cs16_tgt with the same pairs rounded to fp16.
hipError_t launch_rope_tables(const int32_t* positions, int T, int d,
                              const InvFreq& src, const InvFreq& tgt,
                              bool same, float2* cs_src, float2* cs_tgt,
                              void* cs16, void* cs16_tgt, hipStream_t stream);

// dtype: 0 = bf16, 1 = f32.  Returns hipErrorInvalidValue for a
// combination that is not instantiated (never reached after validation).
hipError_t launch_map(const MapArgs& a, int dtype, int d, int style,
                      hipStream_t stream);

// W-stationary kernel (bf16, d = 128, k <= 4); needs a.cs16, a.cs16_tgt and
// a.range_len.
bool map_w_supported(int dtype, int d, int k);
hipError_t launch_map_w(const MapArgs& a, int style, hipStream_t stream);
// Bytes of the packed map images of all L_t target layers, and the kernel that
// writes the images of layers a.l0 .. a.l0+a.nl-1 from W_K / W_V.
size_t packed_w_bytes(int L_t, int H, int k);
hipError_t launch_pack_w(const MapArgs& a, void* wp, hipStream_t stream);

// Layer-sweep kernel (bf16, d = 128, k <= 4): one workgroup per CU.  The
// target layers of a launch are cut into groups of 64 and then groups whose
// sizes are the powers of two of the remainder (80 = 64 + 16, 36 = 32 + 4),
// so that every group's layer pairs times token parts fill the 32 CUs of an
// XCD exactly; a unit of work is (group, head, K|V).
struct SweepPlan {
  int32_t n_units;       // n_groups * H * 2
  int32_t n_groups;      // full_groups + n_rest
  int32_t full_groups;   // leading groups of 64 layers
  int32_t n_rest;        // remainder groups, at most 6
  int32_t rest_len[6];   // their sizes (descending powers of two)
};
SweepPlan plan_sweep(int nl, int H, int64_t T);
hipError_t launch_map_sweep(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream);

// K-split layer-sweep kernels (bf16, d = 128, same plan): the two waves of a
// target layer split the reduction (k <= 4); the second variant keeps the
// matrix pipe busy across tiles (k = 2 or 4).
bool map_ks_supported(int k, int64_t T, int64_t tgt_rows, bool slots, bool tgt_rope);
hipError_t launch_map_ks(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream);
bool map_ks2_supported(int k, int64_t T, int64_t tgt_rows, bool slots, bool tgt_rope);
hipError_t launch_map_ks2(const MapArgs& a, const SweepPlan& p, int style, hipStream_t stream);

// Cross-head map (bf16, d = 64 or 128): strip pass, map packing and the
// matrix-core product (kvx_xhead.hip).
struct XArgs {
  const uint16_t* src;     // [L_s, 2, H_s, T, d]
  const uint16_t* xs;      // stripped keys [L_s, H_s, T, d] (workspace)
  const uint16_t* wp;      // packed maps [L_t, 2, H_t*d, k*H_s*d] (workspace)
  const uint16_t* bk;      // [L_t, H_t, d] or nullptr
  const uint16_t* bv;
  const float2* cs_tgt;    // [T, d/2] (cos, sin) of the target RoPE
  uint16_t* tgt;           // [L_t, 2, H_t, tgt_rows, d]
  const int32_t* slots;    // [T] or nullptr (dense: row t of a plane is token t)
  int64_t tgt_rows;        // T (dense) or num_slots (slot-addressed)
  int32_t L_s, L_t, H_s, H_t, T, k;
  int32_t l0, nl;          // target layers l0 .. l0 + nl - 1 in this launch
  int32_t n_tiles_t, n_tiles_n, tiles_total, tiles_per_xcd;   // set by launch_xhead
  uint8_t idx[kMaxIdx];    // idx[(l - l0) * k + i]
};
size_t xhead_strip_bytes(int L_s, int H_s, int T, int d);
size_t xhead_packed_bytes(int L_t, int H_s, int H_t, int k, int d);
// Strips the keys when strip is set (cs_src: float32 source table), packs
// W_K / W_V into a.wp when pack is set, and runs the product.
hipError_t launch_xhead(XArgs& a, int d, int style, bool strip, bool pack, const void* wk,
                        const void* wv, const float2* cs_src, hipStream_t stream);

// Key strip of every source layer and head into xs [L_s, H, T, d] (the
// cross-head form's strip pass; cs: float32 source table).
hipError_t launch_strip_keys(const uint16_t* src, const float2* cs, uint16_t* xs, int L_s, int H,
                             int T, int d, int style, hipStream_t stream);

// MLP mapper (kvx_mlp.hip): bf16, head dimension 128.  One launch per network
// layer (1, 2, 3) of target layer l covers the 2H networks of that layer.
constexpr int kMaxMlpK = 8;
struct MlpArgs {
  const uint16_t* src;      // [L_s, 2, H, T, 128]
  const uint16_t* xs;       // stripped keys [L_s, H, T, 128] (workspace)
  const uint16_t* act_in;   // layers 2, 3: activations [2H, T, F] (workspace)
  uint16_t* act_out;        // layers 1, 2: activations [2H, T, F] (workspace)
  const uint16_t* w[2];     // this network layer's weights, K and V: [L_t, H, out, in]
  const uint16_t* b[2];     // [L_t, H, out] or nullptr
  const float2* cs_tgt;     // [T, 64] (cos, sin) of the target RoPE
  uint16_t* tgt;            // [L_t, 2, H, T, 128]
  int32_t T, H, k, F, l;
  int32_t n_tiles_t, n_tiles_n, tiles_total, tiles_per_xcd;   // set by launch_mlp_layer
  int32_t src_l[kMaxMlpK];  // idx[l][i]
};
hipError_t launch_mlp_layer(const MlpArgs& a, int layer, int style, hipStream_t stream);

// Fit and probe (kvx_fit.hip): calibration caches with head dimension 128.
// The fit's prep kernel splits each plane into chunks of this many tokens;
// the channel sums hold one partial per chunk until they are added up.
constexpr int kPrepChunk = 8192;
__host__ __device__ inline int prep_chunks(int Npad) { return (Npad + kPrepChunk - 1) / kPrepChunk; }

struct FitArgs {
  const uint16_t* src;     // [L_s, 2, H, N, 128] bf16
  const uint16_t* tgt;     // [L_t, 2, H, N, 128] bf16
  const float2* cs_src;    // [N, 64] (cos, sin) of the source RoPE
  const float2* cs_tgt;    // [N, 64] of the target RoPE
  uint16_t* planes;        // [P + P/2][Npad/16][128][16] token-tiled planes (bf16)
  double* sums;            // [chunks][P][128] channel sums (chunk 0: the totals)
  double* sumsq;           // [chunks][P][128] channel sums of squares
  float* G;                // [blocks][128][128] Gram blocks
  double* Ascr;            // fit: [L_t * H * 2][p][p] design Gram, Cholesky factor
  double* Bscr;            // fit: [L_t * H * 2][p][128] cross Gram, solution
  float* W_K;              // fit outputs [L_t, H, k*128, 128] and [L_t, H, 128]
  float* W_V;
  float* b_K;
  float* b_V;
  float* r2;               // probe output [L_s, L_t, H, 2]
  double lam;
  int32_t L_s, L_t, H, N, Npad, k, style;
  int32_t P;               // planes of both caches: (L_s + L_t) * 2 * H; key planes'
                           // rounding residuals follow at P + layer * H + head
  int32_t mode;            // 0 = fit, 1 = probe
  int32_t n_jobs, jobs_per_xcd;   // set by launch_fit
  uint8_t idx[kMaxIdx];    // fit: idx[l * k + i]
};
// Gram jobs of a fit or probe launch (host and device agree on the order).
int gram_jobs(const FitArgs& a);
// prep (when prep is set), Gram and solve (fit) or probe kernels; the RoPE
// tables must be built.
hipError_t launch_fit(FitArgs a, bool prep, hipStream_t stream);
hipError_t launch_topk(const float* r2, int L_s, int L_t, int H, int k, int32_t* out,
                       hipStream_t stream);

}  // namespace kvx
