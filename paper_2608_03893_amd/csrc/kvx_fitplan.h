// Launch interface of the fit with its block plan (host only), and the
// workspace layout of its token-tiled planes.  The plan lives in the fit's
// workspace; kvx_fit.hip documents what it holds.
#pragma once

#include <stddef.h>

#include "kvx_internal.h"

namespace kvx {

// Elements from one token-tiled plane to the next: the plane (128 x Npad
// bf16) and a pad of 4352 bytes, so that the planes a Gram job streams
// together do not start at the same offset modulo large powers of two.
constexpr int64_t kPlanePadElems = 2176;
__host__ __device__ inline int64_t fit_plane_stride(int64_t Npad) { return 128 * Npad + kPlanePadElems; }

// Bytes of workspace the block plan of a fit with L_t target layers and k
// source layers per list takes (a multiple of 256).
size_t fit_plan_bytes(int L_t, int k);

// Distinct Gram blocks per (head, K|V) and Gram jobs per (head, K|V) of the
// fit whose index table a.idx holds (a.mode == 0).
void fit_plan_count(const FitArgs& a, int* n_blocks, int* n_jobs);

// prep (when prep is set), Gram and solve (fit, a.mode == 0) or probe kernels.
// The fit needs `plan`: fit_plan_bytes(a.L_t, a.k) bytes of device memory,
// 256-byte aligned, that no other argument overlaps; the probe ignores it.
hipError_t launch_fit(FitArgs a, void* plan, bool prep, hipStream_t stream);

}  // namespace kvx
