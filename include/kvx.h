/*
 * kvx.h -- C ABI of the MI355X (gfx950) cross-model KV cache mapper.
 *
 * The library applies a fitted per-head linear mapper to a source model's
 * prefilled KV cache and writes the target model's KV cache (paper: "Cross-
 * Model KV Cache Transfer in LLM Families: A Closed-Form Linear Mapping for
 * Prefill Reuse").  For every target layer l, KV head h and token t:
 *
 *   x_K = [ R_src(p_t)^-1 K_src[idx[l][0], h, t] | ... | R_src(p_t)^-1 K_src[idx[l][k-1], h, t] ]
 *   x_V = [ V_src[idx[l][0], h, t] | ... | V_src[idx[l][k-1], h, t] ]
 *   K_tgt[l, h, t] = R_tgt(p_t) ( x_K W_K[l][h] + b_K[l][h] )
 *   V_tgt[l, h, t] =              x_V W_V[l][h] + b_V[l][h]
 *
 * (Sec. 2.1 problem statement, Eq. ridge_kv of Sec. 3.1, the concatenation of
 * the k selected source layers of Sec. 3.2, the RoPE factoring of Sec. 3.3.)
 * kvx_map_cache, kvx_map_layer and kvx_map_cache_slots apply the per-head
 * form: each row block of W sees one source head, so W is [k*d, d], and source
 * and target have matched KV (same head count H and head dimension d,
 * Sec. 2.1).  kvx_map_cache_xhead applies the cross-head form of Sec. 3.2
 * (every source head feeds every target head; head counts may differ).  Both
 * need the same token count on both sides (shared tokenizer).
 *
 * Conventions shared by every entry point:
 *   - Tensor pointers are DEVICE pointers to dense row-major arrays of the
 *     element type given by `dtype` (src, W, b and target all share it).
 *     Every device pointer must be 16-byte aligned.  The caller owns all
 *     memory; the library never allocates or frees.
 *   - `src_idx` is a HOST pointer to int32 [L_t, k], 0-based source layer
 *     indices.  Row l lists the selected source layers of target layer l;
 *     its order is the order of W's row blocks (block i <-> idx[l][i]).
 *     Repeated indices are allowed.  The table is read during the call and
 *     may be freed when the call returns.
 *   - Calls are asynchronous: work is enqueued on `stream` (a hipStream_t;
 *     NULL is the default stream) and the call returns without waiting.
 *   - Every argument is validated on the host before anything is enqueued.
 *     On any status other than KVX_OK nothing was enqueued and the target
 *     is untouched; kvx_last_error() describes the failure.
 *   - Rounding: keys are stripped with fp32 arithmetic and rounded once to
 *     the element type before the contraction; the contraction accumulates in
 *     fp32 and the result is rounded once (round-to-nearest-even) on store.
 *     The rotation coefficients (cos, sin) come from angles reduced in fp64;
 *     the fp32 path uses them as fp32, the per-head bf16 path as fp16 pairs
 *     (11 significant bits, an eighth of a bf16 rounding step), and the
 *     cross-head bf16 path as fp32.
 *   - Thread safety: calls on different streams may run concurrently.  Calls
 *     that share a workspace must be ordered by the caller.
 */
#ifndef KVX_H
#define KVX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kvx_status {
  KVX_OK = 0,
  KVX_ERR_NULL = 1,        /* a required pointer is NULL                         */
  KVX_ERR_SHAPE = 2,       /* a dimension is negative, zero where it may not be,
                              odd where it must be even, or sizes overflow       */
  KVX_ERR_INDEX = 3,       /* a source index is outside [0, L_s), or l_t is
                              outside [0, L_t)                                   */
  KVX_ERR_DTYPE = 4,       /* unknown element type                              */
  KVX_ERR_UNSUPPORTED = 5, /* well-formed but not built: head dimension other
                              than 64 or 128, L_s > 256, L_t*k > 2048, a pointer
                              that is not 16-byte aligned                        */
  KVX_ERR_ALIAS = 6,       /* the target overlaps an input or the workspace, or
                              the workspace overlaps an input                    */
  KVX_ERR_WORKSPACE = 7,   /* workspace NULL, smaller than the bytes that
                              kvx_workspace_bytes() reports,
                              or not 256-byte aligned                            */
  KVX_ERR_HIP = 8,         /* the HIP runtime rejected a launch                 */
  KVX_ERR_ROPE = 9         /* RoPE parameters out of range                       */
} kvx_status;

typedef enum kvx_dtype { KVX_BF16 = 0, KVX_F32 = 1 } kvx_dtype;

/* RoPE of one model (Sec. 3.3).  Plane j rotates by angle p * w_j with
 * w_j = theta^(-2j/d), j = 0 .. d/2-1, over the full head dimension.
 *   style 0: plane j is channels (j, j + d/2)   (rotate-half layout)
 *   style 1: plane j is channels (2j, 2j + 1)   (interleaved layout)
 * factor == 1 leaves w_j unchanged.  factor > 1 applies the Llama 3.1
 * rescaling: with wavelength L = 2*pi/w_j and C = original_max_pos, w_j is kept
 * when L < C/high_freq_factor, divided by factor when L > C/low_freq_factor,
 * and blended linearly in C/L in between.  Valid: theta > 1, finite;
 * factor >= 1; when factor > 1, 0 < low_freq_factor < high_freq_factor and
 * original_max_pos > 0. */
typedef struct kvx_rope {
  double theta;
  int32_t style;
  int32_t original_max_pos;
  double factor;
  double low_freq_factor;
  double high_freq_factor;
} kvx_rope;

/* Problem sizes.  L_s source layers, L_t target layers, H KV heads on both
 * sides, T tokens (T == 0 is a valid empty call), d head dimension (64 or
 * 128), k selected source layers per target layer (k >= 1). */
typedef struct kvx_dims {
  int32_t L_s, L_t, H, T, d, k;
} kvx_dims;

/* Flag for the map entry points: the workspace already holds the RoPE
 * tables that kvx_rope_prepare (or an earlier map call) built for the same
 * T, d, positions and RoPE parameters, so they are not rebuilt. */
#define KVX_FLAG_TABLES_READY 1u
/* Flag for the map entry points: the workspace already holds the packed maps
 * that an earlier call wrote from the same W_K / W_V (for the same target
 * layers), so they are not packed again.  Only used for head dimension 128,
 * k <= 4 and bf16; ignored otherwise. */
#define KVX_FLAG_WEIGHTS_PACKED 2u
/* Flag for kvx_map_cache_xhead only: the workspace already holds the stripped
 * source keys that an earlier call wrote from the same src_kv, positions and
 * source RoPE, so the strip pass is skipped.  Ignored by the other entry
 * points. */
#define KVX_FLAG_KEYS_STRIPPED 4u

/* Bytes of device workspace a call with these sizes and element type needs:
 * 0 when T == 0 (an empty call touches no workspace); otherwise the cos/sin
 * tables of both RoPEs as float32 [2][T][d/2][2] and as fp16 [2][T][d/2][2]
 * (12*T*d bytes, rounded up to 256), plus, for bf16 with d == 128 and k <= 4,
 * the maps re-packed into the matrix-core operand layout (2*L_t*H*k*d*d*2
 * bytes, the size of W_K and W_V in bf16).  Returns 0 when dims is NULL or
 * inconsistent, or dtype is unknown. */
size_t kvx_workspace_bytes(const kvx_dims* dims, kvx_dtype dtype);

/* Build the cos/sin tables of rope_src and rope_tgt for the given positions
 * in the workspace (Sec. 3.3; angles reduced in float64, stored as float32
 * and as fp16 pairs in the first 12*T*d bytes, rounded up to 256).
 * positions: device int32 [T].  Used to share tables across several
 * kvx_map_layer calls with KVX_FLAG_TABLES_READY. */
kvx_status kvx_rope_prepare(const kvx_dims* dims, const kvx_rope* rope_src,
                            const kvx_rope* rope_tgt, const int32_t* positions,
                            void* workspace, size_t workspace_bytes,
                            void* stream);

/* Map the whole cache: every target layer, head, K and V.
 *   src_kv     device [L_s, 2, H, T, d]   source cache, keys carry the source RoPE
 *   src_idx    HOST int32 [L_t, k]        selected source layers (see above)
 *   W_K, W_V   device [L_t, H, k*d, d]    per-head maps, rows = input features
 *   b_K, b_V   device [L_t, H, d] or NULL (NULL = zero bias), content space
 *   rope_src, rope_tgt                    RoPE of the source and of the target
 *   positions  device int32 [T]           position of each token (strip and
 *                                         re-apply use the same position)
 *   tgt_kv     device [L_t, 2, H, T, d]   written completely
 *   workspace  device, >= kvx_workspace_bytes(dims, dtype), 256-byte
 *              aligned; it must not overlap any input or the target
 *   flags      0, or KVX_FLAG_TABLES_READY and/or KVX_FLAG_WEIGHTS_PACKED  */
kvx_status kvx_map_cache(const kvx_dims* dims, kvx_dtype dtype,
                         const void* src_kv, const int32_t* src_idx,
                         const void* W_K, const void* W_V,
                         const void* b_K, const void* b_V,
                         const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                         const int32_t* positions, void* tgt_kv,
                         void* workspace, size_t workspace_bytes,
                         uint32_t flags, void* stream);

/* Map one target layer l_t (0 <= l_t < L_t).  Arguments are those of
 * kvx_map_cache with the full [L_t, ...] arrays; only idx[l_t], W[l_t],
 * b[l_t] are read and only tgt_kv[l_t] is written (the layer-by-layer
 * batched matmul of Sec. 4.7 / Appendix D). */
kvx_status kvx_map_layer(const kvx_dims* dims, kvx_dtype dtype, int32_t l_t,
                         const void* src_kv, const int32_t* src_idx,
                         const void* W_K, const void* W_V,
                         const void* b_K, const void* b_V,
                         const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                         const int32_t* positions, void* tgt_kv,
                         void* workspace, size_t workspace_bytes,
                         uint32_t flags, void* stream);

/* Map packed new-turn tokens into a slot-addressed (paged) target pool: the
 * incremental multi-turn handoff of Sec. 4.6.  dims.T is the number of packed
 * source rows; src_kv is [L_s, 2, H, T, d] and positions [T] as above.
 *   slot_mapping  device int32 [T]: row t is written to slot slot_mapping[t]
 *                 of every (layer, K|V, head) plane of the pool; a row whose
 *                 slot is negative or >= num_slots is skipped (padding).
 *                 Slots must be distinct within one call (otherwise which
 *                 row wins is unspecified).
 *   num_slots     rows per plane of the pool (>= 1, < 2^31)
 *   tgt_pool      device [L_t, 2, H, num_slots, d]; slots not named by
 *                 slot_mapping are never written.                           */
kvx_status kvx_map_cache_slots(const kvx_dims* dims, kvx_dtype dtype,
                               const void* src_kv, const int32_t* src_idx,
                               const void* W_K, const void* W_V,
                               const void* b_K, const void* b_V,
                               const kvx_rope* rope_src,
                               const kvx_rope* rope_tgt,
                               const int32_t* positions,
                               const int32_t* slot_mapping, int64_t num_slots,
                               void* tgt_pool, void* workspace,
                               size_t workspace_bytes, uint32_t flags,
                               void* stream);

/* Sizes of the cross-head form (Sec. 3.2, Eq. ridge_kv): L_s source layers
 * with H_s KV heads, L_t target layers with H_t KV heads, head dimension d on
 * both sides (64 or 128), T tokens (T == 0 is a valid empty call), k selected
 * source layers per target layer (k >= 1). */
typedef struct kvx_xdims {
  int32_t L_s, L_t, H_s, H_t, T, d, k;
} kvx_xdims;

/* Bytes of device workspace kvx_map_cache_xhead needs: the RoPE tables
 * (12*T*d bytes, rounded up to 256), the stripped source keys in bf16
 * (L_s*H_s*T*d*2, rounded up to 256) and the packed maps
 * (2*L_t*H_t*d*k*H_s*d*2, the size of W_K and W_V).  0 when dims is NULL or
 * inconsistent. */
size_t kvx_xhead_workspace_bytes(const kvx_xdims* dims);

/* Map the whole cache with the cross-head map: the input of every target head
 * concatenates, for each selected source layer in list order, the features of
 * ALL source KV heads (head 0 first), so for target layer l, head h, token t:
 *
 *   x_K = [ R_src(p_t)^-1 K_src[idx[l][i], g, t] for i = 0..k-1, g = 0..H_s-1 ]
 *   K_tgt[l, h, t] = R_tgt(p_t) ( x_K W_K[l][h] + b_K[l][h] ),  and V alike
 *
 * (Eq. ridge_kv with the features of Sec. 3.2; RoPE factoring of Sec. 3.3.)
 *   src_kv     device [L_s, 2, H_s, T, d]
 *   src_idx    HOST int32 [L_t, k]
 *   W_K, W_V   device [L_t, H_t, k*H_s*d, d]; row (i*H_s + g)*d + c multiplies
 *              channel c of source head g of layer src_idx[l][i]
 *   b_K, b_V   device [L_t, H_t, d] or NULL (zero)
 *   positions  device int32 [T]
 *   tgt_kv     device [L_t, 2, H_t, T, d], written completely
 *   workspace  device, >= kvx_xhead_workspace_bytes(dims), 256-byte aligned;
 *              it must not overlap any input or the target
 *   flags      any of KVX_FLAG_TABLES_READY (tables of an earlier call with
 *              the same T, d, positions and RoPEs), KVX_FLAG_WEIGHTS_PACKED
 *              (maps packed by an earlier call from the same W_K / W_V) and
 *              KVX_FLAG_KEYS_STRIPPED (keys stripped by an earlier call from
 *              the same src_kv, positions and source RoPE)
 * Only bf16 is built (KVX_F32 -> KVX_ERR_UNSUPPORTED).  Also unsupported: byte
 * offsets of a source plane ((T + 256)*d*2) or of a packed map
 * ((H_t*d + 256)*k*H_s*d*2) reaching 2^32, L_s > 256, L_t*k > 2048.
 * Rounding: keys stripped with fp32 coefficients and arithmetic and rounded
 * once to bf16, fp32 accumulation, one RNE of each output. */
kvx_status kvx_map_cache_xhead(const kvx_xdims* dims, kvx_dtype dtype,
                               const void* src_kv, const int32_t* src_idx,
                               const void* W_K, const void* W_V,
                               const void* b_K, const void* b_V,
                               const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                               const int32_t* positions, void* tgt_kv,
                               void* workspace, size_t workspace_bytes,
                               uint32_t flags, void* stream);

/* Cross-head map of one target layer l_t (0 <= l_t < L_t; KVX_ERR_INDEX
 * otherwise): arguments as for kvx_map_cache_xhead with the full arrays; only
 * idx[l_t], W[l_t], b[l_t] are read and only tgt_kv[l_t] is written (the
 * layer-by-layer serving of Sec. 4.7).  KVX_FLAG_WEIGHTS_PACKED refers to the
 * maps of this layer. */
kvx_status kvx_map_layer_xhead(const kvx_xdims* dims, kvx_dtype dtype, int32_t l_t,
                               const void* src_kv, const int32_t* src_idx,
                               const void* W_K, const void* W_V,
                               const void* b_K, const void* b_V,
                               const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                               const int32_t* positions, void* tgt_kv,
                               void* workspace, size_t workspace_bytes,
                               uint32_t flags, void* stream);

/* Cross-head map of packed new-turn tokens into a slot-addressed target pool
 * (the multi-turn handoff of Sec. 4.6): dims.T packed source rows, row t
 * written to slot slot_mapping[t] of every (layer, K|V, head) plane of
 * tgt_pool [L_t, 2, H_t, num_slots, d]; rows with a slot outside
 * [0, num_slots) are skipped, slots not named are never written, slots must
 * be distinct within a call.  Other arguments as for kvx_map_cache_xhead. */
kvx_status kvx_map_cache_slots_xhead(const kvx_xdims* dims, kvx_dtype dtype,
                                     const void* src_kv, const int32_t* src_idx,
                                     const void* W_K, const void* W_V,
                                     const void* b_K, const void* b_V,
                                     const kvx_rope* rope_src,
                                     const kvx_rope* rope_tgt,
                                     const int32_t* positions,
                                     const int32_t* slot_mapping, int64_t num_slots,
                                     void* tgt_pool, void* workspace,
                                     size_t workspace_bytes, uint32_t flags,
                                     void* stream);

/* ---- Fitting the mapper (the step before the map) ----------------------
 *
 * Both calls take the source and the target model's KV caches of the same N
 * calibration tokens (dims.T = N), laid out like the map's source:
 *   src_kv  device bf16 [L_s, 2, H, N, 128]   keys carry the source RoPE
 *   tgt_kv  device bf16 [L_t, 2, H, N, 128]   keys carry the target RoPE
 *   positions device int32 [N]
 * Keys of both sides are stripped of their own RoPE (fp32 coefficients,
 * rounded once to bf16) before any statistic is formed (Sec. 3.3).  The Gram
 * matrices are accumulated in fp32 on the matrix cores from bf16 operands
 * (the paper fits with bf16 features and an fp32 covariance); centring, the
 * ridge term and every solve run in fp64.  Only bf16 caches with head
 * dimension 128 are built (others: KVX_ERR_UNSUPPORTED).  The workspace must
 * not overlap any input or output.  flags: 0, or KVX_FLAG_PLANES_READY when the
 * workspace already holds the stripped token-tiled planes and channel sums
 * that an earlier fit or probe call built from the same caches, positions and
 * RoPEs (the call then starts at the Gram matrices). */
#define KVX_FLAG_PLANES_READY 8u

/* Bytes of workspace kvx_fit_cache needs (0 for T == 0 or invalid dims):
 * the RoPE tables (12*N*128), token-tiled copies of every plane of both
 * caches ((L_s + L_t)*2*H planes of 128*roundup(N, 64)*2 bytes plus a
 * 4352-byte pad, and half as many again for the keys' rounding residuals),
 * their channel sums and sums of squares (fp64, one partial per 8192
 * tokens), the Gram blocks (L_t*H*2*k(k+3)/2 blocks of 128 x 128 fp32, an
 * upper bound: a block of two source layers is computed once for every
 * target layer whose list holds the pair), fp64 scratch for the solves
 * (L_t*H*2*(p*p + p*128)*8, p = k*128) and the block plan
 * (L_t*96 + L_t*k(k+3)/2*32 + L_t*100), each rounded up to 256 bytes. */
size_t kvx_fit_workspace_bytes(const kvx_dims* dims);

/* Fit the whole per-head mapper (Sec. 3.1, Fitting: Eq. Wstar on centred data
 * with the bias recovered as mean(Y) - mean(X) W): for every target layer l,
 * head h and K|V, the design concatenates the selected source layers'
 * stripped keys (values) of head h in the order of src_idx[l], the response
 * is the target's stripped keys (values) of layer l, head h, and
 *   W = (Xc^T Xc + lambda I)^-1 Xc^T Yc,   b = mean(Y) - mean(X) W.
 *   src_idx  HOST int32 [L_t, k], 1 <= k <= 4 (as for kvx_map_cache)
 *   lambda   ridge term, finite, >= 0 (the paper uses 0.01); with lambda = 0
 *            the design Gram must be positive definite (N > k*128 and no
 *            exactly collinear features), or the results are not finite
 *   W_K, W_V device fp32 [L_t, H, k*128, 128] (rows = input features: the
 *            layout kvx_map_cache takes, after rounding to bf16)
 *   b_K, b_V device fp32 [L_t, H, 128]
 * Asynchronous on `stream`; all-or-nothing validation as for the map.  The
 * fit and the probe lay out their workspace alike up to the Gram blocks, so
 * KVX_FLAG_PLANES_READY holds across them for the same dims.T. */
kvx_status kvx_fit_cache(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                         const int32_t* src_idx, const void* tgt_kv,
                         const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                         const int32_t* positions, double lambda, float* W_K, float* W_V,
                         float* b_K, float* b_V, void* workspace, size_t workspace_bytes,
                         uint32_t flags, void* stream);

/* Bytes of workspace kvx_probe_r2 needs (dims.k is ignored): the tables,
 * plane copies and sums as for the fit, and L_s*H*2*(L_t + 1) Gram blocks. */
size_t kvx_probe_workspace_bytes(const kvx_dims* dims);

/* The single-source linear probe (Sec. 2.3, Eq. single_source_ols): for
 * every source layer l', target layer l and head h, the ordinary least-squares
 * fit with intercept of the target's per-token head features on the
 * source's, for stripped keys (c = 0) and values (c = 1), and its coefficient
 * of determination pooled over the 128 output channels:
 *   R2 = ||L^-1 Xc^T Yc||_F^2 / ||Yc||_F^2,  Xc^T Xc = L L^T (Cholesky, fp64).
 *   r2  device fp32 [L_s, L_t, H, 2]
 * The centred source Gram must be positive definite (N > 128). */
kvx_status kvx_probe_r2(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                        const void* tgt_kv, const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                        const int32_t* positions, float* r2, void* workspace,
                        size_t workspace_bytes, uint32_t flags, void* stream);

/* Cross-layer source selection (Sec. 3.2): for each target layer, the k
 * source layers with the largest R2 averaged over heads and over stripped
 * keys and values (r2 as kvx_probe_r2 writes it); an equal average goes to
 * the lower source index; each row is written in ascending order.
 *   r2       device fp32 [L_s, L_t, H, 2]
 *   src_idx  device int32 [L_t, k] (1 <= k <= min(L_s, 32)) */
kvx_status kvx_select_topk(int32_t L_s, int32_t L_t, int32_t H, int32_t k, const float* r2,
                           int32_t* src_idx, void* stream);

/* ---- MLP mapper (the nonlinear variant, Sec. 4.4) ----------------------
 *
 * The ridge map's features feed, per target layer l, head h and K|V, a
 * three-layer network (hidden width F; F = 1024 in the paper's appendix):
 *   y = W3 ReLU(W2 ReLU(W1 x + b1) + b2) + b3,   K_tgt = R_tgt(p_t) y_K,
 *   V_tgt = y_V,
 * with x = x_K or x_V exactly as in kvx_map_cache (stripped keys / values of
 * the selected source layers of head h, in src_idx order).  Weights are
 * given in the layout of torch.nn.Linear, [out, in], per (l, h):
 *   W1 [L_t, H, F, k*d]   b1 [L_t, H, F] or NULL (zeros)
 *   W2 [L_t, H, F, F]     b2 [L_t, H, F] or NULL
 *   W3 [L_t, H, d, F]     b3 [L_t, H, d] or NULL
 * one kvx_mlp for the key networks and one for the value networks.
 * Only bf16 with d == 128, 1 <= k <= 8 and F a multiple of 256 is built
 * (KVX_ERR_UNSUPPORTED otherwise); (T + 512) * F * 2 must stay below 2^32.
 * Rounding: keys are stripped with fp32 coefficients and rounded once to bf16
 * (as the cross-head map does); each layer accumulates in fp32, adds its
 * bias in fp32, applies ReLU and rounds to bf16 (round-to-nearest-even), as a
 * bf16 network evaluates it; the last layer's output gets the target RoPE in
 * fp32 before its rounding. */
typedef struct kvx_mlp {
  const void* W1;
  const void* b1;
  const void* W2;
  const void* b2;
  const void* W3;
  const void* b3;
} kvx_mlp;

/* Bytes of workspace kvx_mlp_map_cache needs (0 for T == 0, invalid dims or
 * F < 1): the RoPE tables (12*T*d), the stripped source keys
 * (L_s*H*T*d*2) and the two hidden activations of the 2H networks of one
 * target layer (2 * 2H*T*F*2), each rounded up to 256 bytes. */
size_t kvx_mlp_workspace_bytes(const kvx_dims* dims, int32_t F);

/* Map the whole cache with the MLP mapper into tgt_kv [L_t, 2, H, T, d]
 * (dense).  src_kv, src_idx, ropes, positions and flags as for kvx_map_cache
 * (KVX_FLAG_TABLES_READY; KVX_FLAG_KEYS_STRIPPED when the workspace already
 * holds the stripped keys of the same src_kv, positions and source RoPE).
 * The workspace must not overlap any input or the target.  All-or-nothing
 * validation; asynchronous on `stream`; the target layers are computed one
 * after another (three launches each), so calls sharing a workspace must be
 * ordered by the caller. */
kvx_status kvx_mlp_map_cache(const kvx_dims* dims, kvx_dtype dtype, int32_t F,
                             const void* src_kv, const int32_t* src_idx,
                             const kvx_mlp* mlp_K, const kvx_mlp* mlp_V,
                             const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                             const int32_t* positions, void* tgt_kv, void* workspace,
                             size_t workspace_bytes, uint32_t flags, void* stream);

/* The same for target layer l_t only (writes tgt_kv[l_t]; other layers are
 * untouched). */
kvx_status kvx_mlp_map_layer(const kvx_dims* dims, kvx_dtype dtype, int32_t F, int32_t l_t,
                             const void* src_kv, const int32_t* src_idx,
                             const kvx_mlp* mlp_K, const kvx_mlp* mlp_V,
                             const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                             const int32_t* positions, void* tgt_kv, void* workspace,
                             size_t workspace_bytes, uint32_t flags, void* stream);

/* Size of the device scratch that kvx_map_cache_noalloc uses as its
 * workspace (256 MiB; every workload up to the Llama-3.1-8B -> 70B shape at
 * T = 65536 fits). */
#define KVX_SCRATCH_MAX_BYTES ((size_t)256 << 20)

/* kvx_map_cache for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * The arguments are those of kvx_map_cache without the workspace: the
 * library uses a static device array of KVX_SCRATCH_MAX_BYTES bytes instead,
 * one per device (the device of `stream`; the current device for the NULL
 * stream), held until the process ends.  The call allocates nothing and
 * calls no allocating routine.
 *   - A call whose kvx_workspace_bytes(dims, dtype) exceeds
 *     KVX_SCRATCH_MAX_BYTES returns KVX_ERR_WORKSPACE before any HIP call.
 *   - Every call on one device shares that device's array and leaves its
 *     contents (RoPE tables, packed maps) for the next call; nothing in it
 *     needs to start at zero.  KVX_FLAG_TABLES_READY / KVX_FLAG_WEIGHTS_PACKED
 *     may be passed only when the previous call on that device built the
 *     same tables / packed the same maps.
 *   - Calls that overlap on one device (different streams, or threads
 *     without ordering) race on the array: the caller must order them.
 * Results are identical to kvx_map_cache's for the same inputs. */
kvx_status kvx_map_cache_noalloc(const kvx_dims* dims, kvx_dtype dtype,
                                 const void* src_kv, const int32_t* src_idx,
                                 const void* W_K, const void* W_V,
                                 const void* b_K, const void* b_V,
                                 const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                                 const int32_t* positions, void* tgt_kv,
                                 uint32_t flags, void* stream);

/* Text for the last non-OK status returned on the calling thread ("" if
 * none).  The pointer stays valid until the next kvx call on that thread. */
const char* kvx_last_error(void);

/* Library version as 10000*major + 100*minor + patch. */
int32_t kvx_version(void);

/* Name of the kernel that kvx_map_cache / kvx_map_cache_slots (n_layers =
 * L_t) or kvx_map_layer (n_layers = 1) would launch for these sizes and
 * element type: with bf16, d == 128, k <= 4, H a multiple of 8 and at least 16
 * target layers, one of the layer-sweep kernels "map_ks2_kernel" (k = 2, 4),
 * "map_ks_kernel" (k = 1, 3) or "map_sweep_kernel" (when neither fits);
 * "map_w_kernel" for the other bf16 cases with d == 128, k <= 4; "map_kernel"
 * for everything else.  The environment variable KVX_KERNEL can override the
 * choice (tuning).  For profiling and benchmarks; a static string, NULL for
 * invalid arguments. */
const char* kvx_map_kernel_name(const kvx_dims* dims, kvx_dtype dtype, int32_t n_layers);

#ifdef __cplusplus
}
#endif

#endif /* KVX_H */
