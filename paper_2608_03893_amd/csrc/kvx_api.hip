// Host side of the C ABI declared in include/kvx.h: argument validation,
// RoPE frequency set-up, workspace layout and kernel launch.
//
// Every check runs before the first HIP call, so a rejected call enqueues
// nothing and leaves the target untouched; the checks need no GPU.
#include "kvx.h"
#include "kvx_fitplan.h"
#include "kvx_internal.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>

namespace {

thread_local char g_err[512] = "";

kvx_status fail(kvx_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

kvx_status ok() {
  g_err[0] = '\0';
  return KVX_OK;
}

bool overlap(const void* a, uint64_t abytes, const void* b, uint64_t bbytes) {
  if (a == nullptr || b == nullptr || abytes == 0 || bbytes == 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

bool aligned(const void* p, uintptr_t n) { return ((uintptr_t)p % n) == 0; }

// Plane frequencies (Sec. 3.3): w_j = theta^(-2j/d), with the optional
// Llama 3.1 rescaling by wavelength band.
void inv_freq(const kvx_rope& r, int d, kvx::InvFreq& out) {
  const int half = d / 2;
  const double two_pi = 6.283185307179586476925286766559;
  for (int j = 0; j < half; ++j) {
    const double w = std::pow(r.theta, -2.0 * (double)j / (double)d);
    double v = w;
    if (r.factor != 1.0) {
      const double wavelen = two_pi / w;
      const double ctx = (double)r.original_max_pos;
      if (wavelen < ctx / r.high_freq_factor) {
        v = w;
      } else if (wavelen > ctx / r.low_freq_factor) {
        v = w / r.factor;
      } else {
        const double sm = (ctx / wavelen - r.low_freq_factor) /
                          (r.high_freq_factor - r.low_freq_factor);
        v = (1.0 - sm) * w / r.factor + sm * w;
      }
    }
    out.w[j] = v;
  }
  for (int j = half; j < kvx::kMaxHalf; ++j) out.w[j] = 0.0;
}

kvx_status check_rope(const kvx_rope* r, const char* which) {
  if (r == nullptr) return fail(KVX_ERR_NULL, "%s RoPE parameters are NULL", which);
  if (!std::isfinite(r->theta) || !(r->theta > 1.0))
    return fail(KVX_ERR_ROPE, "%s RoPE theta must be finite and > 1 (got %g)", which, r->theta);
  if (r->style != 0 && r->style != 1)
    return fail(KVX_ERR_ROPE, "%s RoPE style must be 0 (half-split) or 1 (interleaved), got %d",
                which, r->style);
  if (!std::isfinite(r->factor) || !(r->factor >= 1.0))
    return fail(KVX_ERR_ROPE, "%s RoPE factor must be >= 1 (got %g)", which, r->factor);
  if (r->factor != 1.0) {
    if (!(r->low_freq_factor > 0.0) || !(r->high_freq_factor > r->low_freq_factor) ||
        !std::isfinite(r->high_freq_factor))
      return fail(KVX_ERR_ROPE,
                  "%s RoPE needs 0 < low_freq_factor < high_freq_factor (got %g, %g)", which,
                  r->low_freq_factor, r->high_freq_factor);
    if (r->original_max_pos <= 0)
      return fail(KVX_ERR_ROPE, "%s RoPE original_max_pos must be > 0 (got %d)", which,
                  r->original_max_pos);
  }
  return KVX_OK;
}

bool same_rope(const kvx_rope& a, const kvx_rope& b) {
  if (a.theta != b.theta || a.factor != b.factor) return false;
  if (a.factor == 1.0) return true;  // style does not change the frequencies
  return a.low_freq_factor == b.low_freq_factor && a.high_freq_factor == b.high_freq_factor &&
         a.original_max_pos == b.original_max_pos;
}

kvx_status check_dims(const kvx_dims* dims) {
  if (dims == nullptr) return fail(KVX_ERR_NULL, "dims is NULL");
  const kvx_dims& m = *dims;
  if (m.L_s < 1 || m.L_t < 1 || m.H < 1 || m.T < 0 || m.k < 1 || m.d < 2)
    return fail(KVX_ERR_SHAPE,
                "dims out of range: L_s=%d L_t=%d H=%d T=%d d=%d k=%d (need L_s,L_t,H,k >= 1, "
                "T >= 0, d >= 2)", m.L_s, m.L_t, m.H, m.T, m.d, m.k);
  if (m.d % 2) return fail(KVX_ERR_SHAPE, "head dimension d=%d must be even", m.d);
  if (m.d != 64 && m.d != 128)
    return fail(KVX_ERR_UNSUPPORTED, "head dimension d=%d is not built (64 or 128)", m.d);
  if (m.L_s > 256)
    return fail(KVX_ERR_UNSUPPORTED, "L_s=%d exceeds 256 source layers", m.L_s);
  if ((int64_t)m.L_t * m.H * 2 > 65535)
    return fail(KVX_ERR_UNSUPPORTED, "L_t*H*2=%lld exceeds 65535 tasks",
                (long long)m.L_t * m.H * 2);
  return KVX_OK;
}

size_t elem_size(kvx_dtype t) { return t == KVX_BF16 ? 2 : 4; }

// Workspace layout: float32 (cos, sin) tables [T][d/2] of the source and of the
// target RoPE, the same two tables as fp16 pairs [T][d/2], then (for head
// dimension 128 and k <= 4) the packed map images of the W-stationary kernel.
size_t tables_bytes(const kvx_dims& m) {
  const size_t n = (size_t)m.T * (size_t)(m.d / 2);
  return (n * 2 * (sizeof(float2) + sizeof(uint32_t)) + 255) / 256 * 256;
}

// The bf16 kernels for head dimension 128 and k <= 4 read the maps from
// packed images in the workspace; the general tile kernel reads W as given.
bool packs_weights(const kvx_dims& m, kvx_dtype dt) {
  return dt == KVX_BF16 && m.d == 128 && m.k >= 1 && m.k <= 4;
}

// An empty call (T == 0) touches no workspace.
size_t ws_bytes(const kvx_dims& m, kvx_dtype dt) {
  if (m.T == 0) return 0;
  return tables_bytes(m) + (packs_weights(m, dt) ? kvx::packed_w_bytes(m.L_t, m.H, m.k) : 0);
}

struct Tables {
  float2* cs_src;
  float2* cs_tgt;
  void* cs16;
  void* cs16_tgt;
};

Tables tables(const kvx_dims& m, void* ws, bool same) {
  const size_t n = (size_t)m.T * (size_t)(m.d / 2);
  Tables t;
  t.cs_src = reinterpret_cast<float2*>(ws);
  t.cs_tgt = same ? t.cs_src : t.cs_src + n;
  uint32_t* h = reinterpret_cast<uint32_t*>(t.cs_src + 2 * n);
  t.cs16 = h;
  t.cs16_tgt = same ? h : h + n;
  return t;
}

// Tokens per workgroup of the W-stationary kernel: long enough to amortise
// staging the map, a multiple of the 256-token tile.  The environment
// variable KVX_TOKENS_PER_WG overrides it (tuning only).
int tokens_per_wg() {
  const char* e = std::getenv("KVX_TOKENS_PER_WG");
  int r = (e != nullptr && std::atoi(e) > 0) ? std::atoi(e) : 4096;
  if (r > (1 << 30)) r = 1 << 30;
  return ((r + 255) / 256) * 256;
}

struct Call {
  kvx_dims m;
  kvx_dtype dtype;
  const void* src;
  const int32_t* idx;
  const void *wk, *wv, *bk, *bv;
  const kvx_rope *rs, *rt;
  const int32_t* pos;
  const int32_t* slots;
  int64_t tgt_rows;
  void* tgt;
  void* ws;
  size_t wsb;
  uint32_t flags;
  hipStream_t stream;
  int l0, nl;
};

kvx_status validate(const Call& c) {
  kvx_status st = check_dims(&c.m);
  if (st != KVX_OK) return st;
  const kvx_dims& m = c.m;
  if (c.dtype != KVX_BF16 && c.dtype != KVX_F32)
    return fail(KVX_ERR_DTYPE, "unknown dtype %d (0 = bf16, 1 = f32)", (int)c.dtype);
  if ((st = check_rope(c.rs, "source")) != KVX_OK) return st;
  if ((st = check_rope(c.rt, "target")) != KVX_OK) return st;
  // The style of each side only changes which channels form a plane; the
  // kernels are built for matching styles.
  if (c.rs->style != c.rt->style)
    return fail(KVX_ERR_UNSUPPORTED, "source and target RoPE styles differ (%d vs %d)",
                c.rs->style, c.rt->style);
  if (c.idx == nullptr) return fail(KVX_ERR_NULL, "src_idx is NULL");
  if (c.wk == nullptr || c.wv == nullptr) return fail(KVX_ERR_NULL, "W_K or W_V is NULL");
  const bool empty = m.T == 0;
  if (!empty) {
    if (c.src == nullptr) return fail(KVX_ERR_NULL, "src_kv is NULL");
    if (c.pos == nullptr) return fail(KVX_ERR_NULL, "positions is NULL");
    if (c.tgt == nullptr) return fail(KVX_ERR_NULL, "target is NULL");
  }
  if ((int64_t)c.nl * m.k > kvx::kMaxIdx)
    return fail(KVX_ERR_UNSUPPORTED, "%d layers x k=%d index entries exceed %d", c.nl, m.k,
                kvx::kMaxIdx);
  for (int l = c.l0; l < c.l0 + c.nl; ++l)
    for (int i = 0; i < m.k; ++i) {
      const int32_t s = c.idx[(int64_t)l * m.k + i];
      if (s < 0 || s >= m.L_s)
        return fail(KVX_ERR_INDEX, "src_idx[%d][%d]=%d is outside [0, %d)", l, i, s, m.L_s);
    }
  const uint64_t es = elem_size(c.dtype);
  const uint64_t src_b = (uint64_t)m.L_s * 2 * m.H * (uint64_t)m.T * m.d * es;
  const uint64_t w_b = (uint64_t)m.L_t * m.H * (uint64_t)m.k * m.d * m.d * es;
  const uint64_t b_b = (uint64_t)m.L_t * m.H * m.d * es;
  const uint64_t pos_b = (uint64_t)m.T * 4;
  const uint64_t tgt_b = (uint64_t)m.L_t * 2 * m.H * (uint64_t)c.tgt_rows * m.d * es;
  const uint64_t limit = (uint64_t)1 << 60;
  if (src_b > limit || tgt_b > limit || w_b > limit)
    return fail(KVX_ERR_SHAPE, "tensor sizes overflow");
  const void* ptrs[] = {c.src, c.wk, c.wv, c.bk, c.bv, c.tgt};
  const char* names[] = {"src_kv", "W_K", "W_V", "b_K", "b_V", "target"};
  for (int n = 0; n < 6; ++n)
    if (ptrs[n] != nullptr && !aligned(ptrs[n], 16))
      return fail(KVX_ERR_UNSUPPORTED, "%s is not 16-byte aligned", names[n]);
  if ((c.pos && !aligned(c.pos, 4)) || (c.slots && !aligned(c.slots, 4)))
    return fail(KVX_ERR_UNSUPPORTED, "positions / slot_mapping must be 4-byte aligned");
  const uint64_t need = ws_bytes(m, c.dtype);
  if (need > 0) {
    if (c.ws == nullptr) return fail(KVX_ERR_WORKSPACE, "workspace is NULL (%llu bytes needed)",
                                     (unsigned long long)need);
    if (c.wsb < need)
      return fail(KVX_ERR_WORKSPACE, "workspace has %llu bytes, %llu needed",
                  (unsigned long long)c.wsb, (unsigned long long)need);
    if (!aligned(c.ws, 256)) return fail(KVX_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  }
  struct In {
    const void* p;
    uint64_t b;
    const char* name;
  } ins[] = {{c.src, src_b, "src_kv"}, {c.wk, w_b, "W_K"}, {c.wv, w_b, "W_V"},
             {c.bk, b_b, "b_K"},       {c.bv, b_b, "b_V"}, {c.pos, pos_b, "positions"},
             {c.slots, pos_b, "slot_mapping"}, {c.ws, need, "workspace"}};
  for (const In& in : ins)
    if (overlap(c.tgt, tgt_b, in.p, in.b))
      return fail(KVX_ERR_ALIAS, "target overlaps %s", in.name);
  // The RoPE tables and packed maps are written into the workspace while the
  // inputs are read, so no input may share its bytes.
  for (int n = 0; n < 7; ++n)
    if (overlap(c.ws, need, ins[n].p, ins[n].b))
      return fail(KVX_ERR_ALIAS, "workspace overlaps %s", ins[n].name);
  return KVX_OK;
}

// Which kernel runs a call: the general tile kernel; the W-stationary kernel
// (bf16, d = 128, k <= 4; one workgroup per task and token range); or one of
// the layer-sweep kernels (same cases; one workgroup per CU, all target layers
// of a head swept together): the k-split kernel with the mid-tile barrier for
// k = 2 and 4, the k-split kernel for k = 1 and 3.  KVX_KERNEL = tile | w |
// sweep | ks | ks2 overrides the choice (tuning and tests).  The
// W-stationary and sweep kernels give bit-identical results; the
// k-split kernels add two partial sums per output and round in another
// order.  All kernels read the same packed maps.
enum class Kernel { Tile, W, Sweep, Ks, Ks2 };

Kernel choose_kernel(int dt, const kvx_dims& m, int nl, int64_t tgt_rows, bool slots,
                     bool tgt_rope) {
  if (!kvx::map_w_supported(dt, m.d, m.k)) return Kernel::Tile;
  const bool ks_ok = kvx::map_ks_supported(m.k, m.T, tgt_rows, slots, tgt_rope);
  const bool ks2_ok = kvx::map_ks2_supported(m.k, m.T, tgt_rows, slots, tgt_rope);
  if (const char* e = std::getenv("KVX_KERNEL")) {
    if (std::strcmp(e, "tile") == 0) return Kernel::Tile;
    if (std::strcmp(e, "w") == 0) return Kernel::W;
    if (std::strcmp(e, "sweep") == 0) return Kernel::Sweep;
    if (std::strcmp(e, "ks") == 0 && ks_ok) return Kernel::Ks;
    if (std::strcmp(e, "ks2") == 0 && ks2_ok) return Kernel::Ks2;
  }
  // The sweep kernels keep every compute unit busy for any layer count (their
  // layer groups fill the 32 CUs of an XCD), but need the heads to spread
  // evenly over the eight XCDs, and enough layers per group to amortise
  // each unit's start (loading the maps, filling the pipeline).
  if (m.H % 8 == 0 && nl >= 16) {
    if (ks2_ok) return Kernel::Ks2;
    if (ks_ok) return Kernel::Ks;
    return Kernel::Sweep;
  }
  return Kernel::W;
}

kvx_status run(const Call& c) {
  kvx_status st = validate(c);
  if (st != KVX_OK) return st;
  const kvx_dims& m = c.m;
  if (m.T == 0) return ok();
  const int dt = c.dtype == KVX_BF16 ? 0 : 1;
  const bool same = same_rope(*c.rs, *c.rt);
  const Kernel kern = choose_kernel(dt, m, c.nl, c.tgt_rows, c.slots != nullptr, !same);
  const bool wpath = kern != Kernel::Tile;
  const Tables tb = tables(m, c.ws, same);
  if (!(c.flags & KVX_FLAG_TABLES_READY)) {
    kvx::InvFreq fs, ft;
    inv_freq(*c.rs, m.d, fs);
    inv_freq(*c.rt, m.d, ft);
    hipError_t e = kvx::launch_rope_tables(c.pos, m.T, m.d, fs, ft, same, tb.cs_src, tb.cs_tgt,
                                           tb.cs16, tb.cs16_tgt, c.stream);
    if (e != hipSuccess) return fail(KVX_ERR_HIP, "RoPE table launch: %s", hipGetErrorString(e));
  }
  kvx::MapArgs a;
  std::memset(&a, 0, sizeof(a));
  a.src = c.src;
  a.wk = c.wk;
  a.wv = c.wv;
  a.bk = c.bk;
  a.bv = c.bv;
  a.cs_src = tb.cs_src;
  a.cs_tgt = tb.cs_tgt;
  a.cs16 = tb.cs16;
  a.cs16_tgt = tb.cs16_tgt;
  a.range_len = tokens_per_wg();
  {
    const char* e = std::getenv("KVX_WAVE_TOKENS");  // tuning only
    a.wave_tokens = (e != nullptr && std::atoi(e) == 64) ? 64 : 32;
  }
  a.tgt = c.tgt;
  a.slots = c.slots;
  a.tgt_rows = c.tgt_rows;
  a.H = m.H;
  a.T = m.T;
  a.k = m.k;
  a.l0 = c.l0;
  a.nl = c.nl;
  for (int l = 0; l < c.nl; ++l)
    for (int i = 0; i < m.k; ++i)
      a.idx[l * m.k + i] = (uint8_t)c.idx[(int64_t)(c.l0 + l) * m.k + i];
  hipError_t e = hipSuccess;
  if (wpath) {
    a.wpack = static_cast<char*>(c.ws) + tables_bytes(m);
    if (!(c.flags & KVX_FLAG_WEIGHTS_PACKED)) {
      e = kvx::launch_pack_w(a, const_cast<void*>(a.wpack), c.stream);
      if (e != hipSuccess) return fail(KVX_ERR_HIP, "weight packing launch: %s", hipGetErrorString(e));
    }
    if (kern == Kernel::Ks)
      e = kvx::launch_map_ks(a, kvx::plan_sweep(c.nl, m.H, m.T), c.rs->style, c.stream);
    else if (kern == Kernel::Ks2)
      e = kvx::launch_map_ks2(a, kvx::plan_sweep(c.nl, m.H, m.T), c.rs->style, c.stream);
    else if (kern == Kernel::Sweep)
      e = kvx::launch_map_sweep(a, kvx::plan_sweep(c.nl, m.H, m.T), c.rs->style, c.stream);
    else
      e = kvx::launch_map_w(a, c.rs->style, c.stream);
  } else {
    e = kvx::launch_map(a, dt, m.d, c.rs->style, c.stream);
  }
  if (e != hipSuccess) return fail(KVX_ERR_HIP, "map launch: %s", hipGetErrorString(e));
  return ok();
}

Call make_call(const kvx_dims* dims, kvx_dtype dtype, const void* src, const int32_t* idx,
               const void* wk, const void* wv, const void* bk, const void* bv,
               const kvx_rope* rs, const kvx_rope* rt, const int32_t* pos, void* tgt,
               void* ws, size_t wsb, uint32_t flags, void* stream) {
  Call c;
  std::memset(&c, 0, sizeof(c));
  if (dims) c.m = *dims;
  c.dtype = dtype;
  c.src = src;
  c.idx = idx;
  c.wk = wk;
  c.wv = wv;
  c.bk = bk;
  c.bv = bv;
  c.rs = rs;
  c.rt = rt;
  c.pos = pos;
  c.tgt = tgt;
  c.tgt_rows = dims ? dims->T : 0;
  c.ws = ws;
  c.wsb = wsb;
  c.flags = flags;
  c.stream = reinterpret_cast<hipStream_t>(stream);
  c.l0 = 0;
  c.nl = dims ? dims->L_t : 0;
  return c;
}

// ---- cross-head form (Sec. 3.2): validation and launch

kvx_status check_xdims(const kvx_xdims* dims) {
  if (dims == nullptr) return fail(KVX_ERR_NULL, "dims is NULL");
  const kvx_xdims& m = *dims;
  if (m.L_s < 1 || m.L_t < 1 || m.H_s < 1 || m.H_t < 1 || m.T < 0 || m.k < 1 || m.d < 2)
    return fail(KVX_ERR_SHAPE,
                "dims out of range: L_s=%d L_t=%d H_s=%d H_t=%d T=%d d=%d k=%d (need L_s, L_t, "
                "H_s, H_t, k >= 1, T >= 0, d >= 2)", m.L_s, m.L_t, m.H_s, m.H_t, m.T, m.d, m.k);
  if (m.d % 2) return fail(KVX_ERR_SHAPE, "head dimension d=%d must be even", m.d);
  if (m.d != 64 && m.d != 128)
    return fail(KVX_ERR_UNSUPPORTED, "head dimension d=%d is not built (64 or 128)", m.d);
  if (m.L_s > 256) return fail(KVX_ERR_UNSUPPORTED, "L_s=%d exceeds 256 source layers", m.L_s);
  if ((int64_t)m.L_s * m.H_s > 65535 || (int64_t)m.L_t * 2 > 65535)
    return fail(KVX_ERR_UNSUPPORTED, "L_s*H_s=%lld or 2*L_t=%lld exceeds 65535",
                (long long)m.L_s * m.H_s, (long long)m.L_t * 2);
  if ((int64_t)m.L_t * m.k > kvx::kMaxIdx)
    return fail(KVX_ERR_UNSUPPORTED, "L_t*k=%lld index entries exceed %d",
                (long long)m.L_t * m.k, kvx::kMaxIdx);
  const uint64_t F = (uint64_t)m.k * m.H_s * m.d, N = (uint64_t)m.H_t * m.d;
  if (((uint64_t)m.T + 256) * m.d * 2 >= ((uint64_t)1 << 32) ||
      (N + 256) * F * 2 >= ((uint64_t)1 << 32) || N / 64 > 65535 || F / 64 > 65535)
    return fail(KVX_ERR_UNSUPPORTED,
                "a source plane ((T+256)*d*2 bytes) or a packed map ((H_t*d+256)*k*H_s*d*2 "
                "bytes) reaches 2^32 (T=%d, H_s=%d, H_t=%d, d=%d, k=%d)", m.T, m.H_s, m.H_t, m.d,
                m.k);
  return KVX_OK;
}

kvx_dims xtables_dims(const kvx_xdims& m) {
  kvx_dims t;
  t.L_s = m.L_s;
  t.L_t = m.L_t;
  t.H = m.H_t;
  t.T = m.T;
  t.d = m.d;
  t.k = m.k;
  return t;
}

size_t xws_bytes(const kvx_xdims& m) {
  return tables_bytes(xtables_dims(m)) + kvx::xhead_strip_bytes(m.L_s, m.H_s, m.T, m.d) +
         kvx::xhead_packed_bytes(m.L_t, m.H_s, m.H_t, m.k, m.d);
}

// l0, nl: the target layers written (all of them for kvx_map_cache_xhead);
// slots / num_slots: slot-addressed target (nullptr: dense, T rows per plane)
kvx_status run_xhead(const kvx_xdims* dims, kvx_dtype dtype, const void* src, const int32_t* idx,
                     const void* wk, const void* wv, const void* bk, const void* bv,
                     const kvx_rope* rs, const kvx_rope* rt, const int32_t* pos, void* tgt,
                     void* ws, size_t wsb, uint32_t flags, void* stream_, int l0, int nl,
                     const int32_t* slots, int64_t num_slots, bool slot_call) {
  kvx_status st = check_xdims(dims);
  if (st != KVX_OK) return st;
  const kvx_xdims& m = *dims;
  if (l0 < 0 || l0 + nl > m.L_t)
    return fail(KVX_ERR_INDEX, "target layer %d is outside [0, %d)", l0, m.L_t);
  if (slot_call && (num_slots < 1 || num_slots >= ((int64_t)1 << 31)))
    return fail(KVX_ERR_SHAPE, "num_slots=%lld must be in [1, 2^31)", (long long)num_slots);
  const int64_t tgt_rows = slot_call ? num_slots : (int64_t)m.T;
  if (dtype != KVX_BF16 && dtype != KVX_F32)
    return fail(KVX_ERR_DTYPE, "unknown dtype %d (0 = bf16, 1 = f32)", (int)dtype);
  if (dtype != KVX_BF16)
    return fail(KVX_ERR_UNSUPPORTED, "the cross-head map is built for bf16 only");
  if ((st = check_rope(rs, "source")) != KVX_OK) return st;
  if ((st = check_rope(rt, "target")) != KVX_OK) return st;
  if (rs->style != rt->style)
    return fail(KVX_ERR_UNSUPPORTED, "source and target RoPE styles differ (%d vs %d)",
                rs->style, rt->style);
  if (idx == nullptr) return fail(KVX_ERR_NULL, "src_idx is NULL");
  if (wk == nullptr || wv == nullptr) return fail(KVX_ERR_NULL, "W_K or W_V is NULL");
  if (m.T > 0) {
    if (src == nullptr) return fail(KVX_ERR_NULL, "src_kv is NULL");
    if (pos == nullptr) return fail(KVX_ERR_NULL, "positions is NULL");
    if (tgt == nullptr) return fail(KVX_ERR_NULL, "target is NULL");
    if (slot_call && slots == nullptr) return fail(KVX_ERR_NULL, "slot_mapping is NULL");
  }
  for (int l = l0; l < l0 + nl; ++l)
    for (int i = 0; i < m.k; ++i) {
      const int32_t s = idx[(int64_t)l * m.k + i];
      if (s < 0 || s >= m.L_s)
        return fail(KVX_ERR_INDEX, "src_idx[%d][%d]=%d is outside [0, %d)", l, i, s, m.L_s);
    }
  const uint64_t F = (uint64_t)m.k * m.H_s * m.d;
  const uint64_t src_b = (uint64_t)m.L_s * 2 * m.H_s * (uint64_t)m.T * m.d * 2;
  const uint64_t w_b = (uint64_t)m.L_t * m.H_t * F * m.d * 2;
  const uint64_t b_b = (uint64_t)m.L_t * m.H_t * m.d * 2;
  const uint64_t pos_b = (uint64_t)m.T * 4;
  const uint64_t tgt_b = (uint64_t)m.L_t * 2 * m.H_t * (uint64_t)tgt_rows * m.d * 2;
  const void* ptrs[] = {src, wk, wv, bk, bv, tgt};
  const char* names[] = {"src_kv", "W_K", "W_V", "b_K", "b_V", "target"};
  for (int n = 0; n < 6; ++n)
    if (ptrs[n] != nullptr && !aligned(ptrs[n], 16))
      return fail(KVX_ERR_UNSUPPORTED, "%s is not 16-byte aligned", names[n]);
  if ((pos && !aligned(pos, 4)) || (slots && !aligned(slots, 4)))
    return fail(KVX_ERR_UNSUPPORTED, "positions / slot_mapping must be 4-byte aligned");
  if (m.T == 0) return ok();   // nothing to map: the workspace is not touched
  const uint64_t need = xws_bytes(m);
  if (ws == nullptr)
    return fail(KVX_ERR_WORKSPACE, "workspace is NULL (%llu bytes needed)", (unsigned long long)need);
  if (wsb < need)
    return fail(KVX_ERR_WORKSPACE, "workspace has %llu bytes, %llu needed",
                (unsigned long long)wsb, (unsigned long long)need);
  if (!aligned(ws, 256)) return fail(KVX_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  struct In {
    const void* p;
    uint64_t b;
    const char* name;
  } ins[] = {{src, src_b, "src_kv"}, {wk, w_b, "W_K"},       {wv, w_b, "W_V"}, {bk, b_b, "b_K"},
             {bv, b_b, "b_V"},       {pos, pos_b, "positions"}, {slots, pos_b, "slot_mapping"}};
  for (const In& in : ins) {
    if (overlap(tgt, tgt_b, in.p, in.b)) return fail(KVX_ERR_ALIAS, "target overlaps %s", in.name);
    if (overlap(ws, need, in.p, in.b)) return fail(KVX_ERR_ALIAS, "workspace overlaps %s", in.name);
  }
  if (overlap(tgt, tgt_b, ws, need)) return fail(KVX_ERR_ALIAS, "target overlaps workspace");

  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  const kvx_dims tm = xtables_dims(m);
  const bool same = same_rope(*rs, *rt);
  const Tables tb = tables(tm, ws, same);
  if (!(flags & KVX_FLAG_TABLES_READY)) {
    kvx::InvFreq fs, ft;
    inv_freq(*rs, m.d, fs);
    inv_freq(*rt, m.d, ft);
    hipError_t e = kvx::launch_rope_tables(pos, m.T, m.d, fs, ft, same, tb.cs_src, tb.cs_tgt,
                                           tb.cs16, tb.cs16_tgt, stream);
    if (e != hipSuccess) return fail(KVX_ERR_HIP, "RoPE table launch: %s", hipGetErrorString(e));
  }
  kvx::XArgs a;
  std::memset(&a, 0, sizeof(a));
  char* wsc = static_cast<char*>(ws);
  a.src = static_cast<const uint16_t*>(src);
  a.xs = reinterpret_cast<const uint16_t*>(wsc + tables_bytes(tm));
  a.wp = reinterpret_cast<const uint16_t*>(wsc + tables_bytes(tm) +
                                           kvx::xhead_strip_bytes(m.L_s, m.H_s, m.T, m.d));
  a.bk = static_cast<const uint16_t*>(bk);
  a.bv = static_cast<const uint16_t*>(bv);
  a.cs_tgt = tb.cs_tgt;
  a.tgt = static_cast<uint16_t*>(tgt);
  a.slots = slots;
  a.tgt_rows = tgt_rows;
  a.l0 = l0;
  a.nl = nl;
  a.L_s = m.L_s;
  a.L_t = m.L_t;
  a.H_s = m.H_s;
  a.H_t = m.H_t;
  a.T = m.T;
  a.k = m.k;
  for (int64_t n = 0; n < (int64_t)nl * m.k; ++n) a.idx[n] = (uint8_t)idx[(int64_t)l0 * m.k + n];
  hipError_t e = kvx::launch_xhead(a, m.d, rs->style, !(flags & KVX_FLAG_KEYS_STRIPPED),
                                   !(flags & KVX_FLAG_WEIGHTS_PACKED), wk, wv, tb.cs_src, stream);
  if (e != hipSuccess) return fail(KVX_ERR_HIP, "cross-head launch: %s", hipGetErrorString(e));
  return ok();
}

// ---- fit and probe (Sec. 3.1 Fitting; Sec. 2.3 / 3.2): validation and layout

struct FitLayout {
  size_t tables, planes, sums, sumsq, G, A, B, plan, total;
  int64_t Npad;
};

size_t up256(size_t n) { return (n + 255) / 256 * 256; }

FitLayout fit_layout(const kvx_dims& m, int mode) {
  FitLayout f;
  f.Npad = ((int64_t)m.T + 63) / 64 * 64;
  const size_t P = (size_t)(m.L_s + m.L_t) * 2 * m.H;
  const size_t tasks = mode == 0 ? (size_t)m.L_t * m.H * 2 : (size_t)m.L_s * m.H * 2;
  const size_t nbl = mode == 0 ? (size_t)m.k * (m.k + 3) / 2 : (size_t)m.L_t + 1;
  const size_t p = (size_t)m.k * 128;
  f.tables = up256((size_t)m.T * 128 * 12);
  f.planes = up256((P + P / 2) * (size_t)kvx::fit_plane_stride(f.Npad) * 2);   // + the keys' residuals
  f.sums = up256((size_t)kvx::prep_chunks((int)f.Npad) * P * 128 * 8);   // a partial per token chunk
  f.sumsq = f.sums;
  f.G = up256(tasks * nbl * 128 * 128 * 4);
  f.A = mode == 0 ? up256(tasks * p * p * 8) : 0;
  f.B = mode == 0 ? up256(tasks * p * 128 * 8) : 0;
  f.plan = mode == 0 ? kvx::fit_plan_bytes(m.L_t, m.k) : 0;
  f.total = f.tables + f.planes + f.sums + f.sumsq + f.G + f.A + f.B + f.plan;
  if (m.T == 0) f.total = 0;
  return f;
}

// mode 0: fit (k selected source layers, 1 <= k <= 4); mode 1: probe (k unused)
kvx_status check_fit_dims(const kvx_dims* dims, int mode) {
  if (dims == nullptr) return fail(KVX_ERR_NULL, "dims is NULL");
  const kvx_dims& m = *dims;
  if (m.L_s < 1 || m.L_t < 1 || m.H < 1 || m.T < 0 || m.d < 2 || (mode == 0 && m.k < 1))
    return fail(KVX_ERR_SHAPE, "dims out of range: L_s=%d L_t=%d H=%d T=%d d=%d k=%d", m.L_s,
                m.L_t, m.H, m.T, m.d, m.k);
  if (m.d % 2) return fail(KVX_ERR_SHAPE, "head dimension d=%d must be even", m.d);
  if (m.d != 128) return fail(KVX_ERR_UNSUPPORTED, "the fit and probe are built for d = 128 (got %d)", m.d);
  if (m.L_s > 256) return fail(KVX_ERR_UNSUPPORTED, "L_s=%d exceeds 256 source layers", m.L_s);
  if (mode == 0 && m.k > 4)
    return fail(KVX_ERR_UNSUPPORTED, "the fit is built for k <= 4 (got %d)", m.k);
  if (mode == 0 && (int64_t)m.L_t * m.k > kvx::kMaxIdx)
    return fail(KVX_ERR_UNSUPPORTED, "L_t*k=%lld index entries exceed %d",
                (long long)m.L_t * m.k, kvx::kMaxIdx);
  const int64_t Npad = ((int64_t)m.T + 63) / 64 * 64;
  if (Npad * 128 * 2 >= ((int64_t)1 << 32))
    return fail(KVX_ERR_UNSUPPORTED, "T=%d: a token-tiled plane reaches 2^32 bytes", m.T);
  if ((int64_t)(m.L_s + m.L_t) * 2 * m.H > 65535 || (int64_t)m.L_t * m.H * 2 > 65535)
    return fail(KVX_ERR_UNSUPPORTED, "too many planes (L_s, L_t, H = %d, %d, %d)", m.L_s, m.L_t, m.H);
  return KVX_OK;
}

kvx_status run_fit(const kvx_dims* dims, kvx_dtype dtype, const void* src, const int32_t* idx,
                   const void* tgt, const kvx_rope* rs, const kvx_rope* rt, const int32_t* pos,
                   double lam, float* wk, float* wv, float* bk, float* bv, float* r2, void* ws,
                   size_t wsb, uint32_t flags, void* stream, int mode) {
  kvx_status st = check_fit_dims(dims, mode);
  if (st != KVX_OK) return st;
  const kvx_dims& m = *dims;
  if (dtype != KVX_BF16 && dtype != KVX_F32)
    return fail(KVX_ERR_DTYPE, "unknown dtype %d (0 = bf16, 1 = f32)", (int)dtype);
  if (dtype != KVX_BF16) return fail(KVX_ERR_UNSUPPORTED, "the fit and probe are built for bf16 caches");
  if ((st = check_rope(rs, "source")) != KVX_OK) return st;
  if ((st = check_rope(rt, "target")) != KVX_OK) return st;
  if (rs->style != rt->style)
    return fail(KVX_ERR_UNSUPPORTED, "source and target RoPE styles differ (%d vs %d)", rs->style,
                rt->style);
  if (mode == 0) {
    if (!std::isfinite(lam) || lam < 0.0)
      return fail(KVX_ERR_SHAPE, "lambda must be finite and >= 0 (got %g)", lam);
    if (idx == nullptr) return fail(KVX_ERR_NULL, "src_idx is NULL");
    for (int l = 0; l < m.L_t; ++l)
      for (int i = 0; i < m.k; ++i) {
        const int32_t s = idx[(int64_t)l * m.k + i];
        if (s < 0 || s >= m.L_s)
          return fail(KVX_ERR_INDEX, "src_idx[%d][%d]=%d is outside [0, %d)", l, i, s, m.L_s);
      }
  }
  if (m.T == 0) return ok();
  if (src == nullptr || tgt == nullptr) return fail(KVX_ERR_NULL, "a calibration cache is NULL");
  if (pos == nullptr) return fail(KVX_ERR_NULL, "positions is NULL");
  if (mode == 0 && (wk == nullptr || wv == nullptr || bk == nullptr || bv == nullptr))
    return fail(KVX_ERR_NULL, "an output (W_K, W_V, b_K, b_V) is NULL");
  if (mode == 1 && r2 == nullptr) return fail(KVX_ERR_NULL, "the R2 output is NULL");
  if (!aligned(src, 16) || !aligned(tgt, 16))
    return fail(KVX_ERR_UNSUPPORTED, "the calibration caches must be 16-byte aligned");
  if (!aligned(pos, 4) || (wk && !aligned(wk, 4)) || (wv && !aligned(wv, 4)) ||
      (bk && !aligned(bk, 4)) || (bv && !aligned(bv, 4)) || (r2 && !aligned(r2, 4)))
    return fail(KVX_ERR_UNSUPPORTED, "positions and outputs must be 4-byte aligned");
  const FitLayout f = fit_layout(m, mode);
  if (ws == nullptr)
    return fail(KVX_ERR_WORKSPACE, "workspace is NULL (%llu bytes needed)", (unsigned long long)f.total);
  if (wsb < f.total)
    return fail(KVX_ERR_WORKSPACE, "workspace has %llu bytes, %llu needed", (unsigned long long)wsb,
                (unsigned long long)f.total);
  if (!aligned(ws, 256)) return fail(KVX_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  const uint64_t src_b = (uint64_t)m.L_s * 2 * m.H * (uint64_t)m.T * 128 * 2;
  const uint64_t tgt_b = (uint64_t)m.L_t * 2 * m.H * (uint64_t)m.T * 128 * 2;
  const uint64_t pos_b = (uint64_t)m.T * 4;
  const uint64_t w_b = (uint64_t)m.L_t * m.H * (uint64_t)m.k * 128 * 128 * 4;
  const uint64_t b_b = (uint64_t)m.L_t * m.H * 128 * 4;
  const uint64_t r2_b = (uint64_t)m.L_s * m.L_t * m.H * 2 * 4;
  struct Ref {
    const void* p;
    uint64_t b;
    const char* name;
  };
  const Ref ins[] = {{src, src_b, "source cache"}, {tgt, tgt_b, "target cache"}, {pos, pos_b, "positions"}};
  const Ref outs[] = {{wk, mode == 0 ? w_b : 0, "W_K"}, {wv, mode == 0 ? w_b : 0, "W_V"},
                      {bk, mode == 0 ? b_b : 0, "b_K"}, {bv, mode == 0 ? b_b : 0, "b_V"},
                      {r2, mode == 1 ? r2_b : 0, "R2"}, {ws, f.total, "workspace"}};
  for (const Ref& o : outs) {
    for (const Ref& i : ins)
      if (overlap(o.p, o.b, i.p, i.b)) return fail(KVX_ERR_ALIAS, "%s overlaps the %s", o.name, i.name);
    for (const Ref& o2 : outs)
      if (&o2 != &o && overlap(o.p, o.b, o2.p, o2.b))
        return fail(KVX_ERR_ALIAS, "%s overlaps %s", o.name, o2.name);
  }
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  const bool same = same_rope(*rs, *rt);
  const Tables tb = tables(m, w, same);
  kvx::InvFreq fs, ft;
  inv_freq(*rs, m.d, fs);
  inv_freq(*rt, m.d, ft);
  hipError_t e = hipSuccess;
  const bool planes_ready = (flags & KVX_FLAG_PLANES_READY) != 0;
  if (!planes_ready) {
    e = kvx::launch_rope_tables(pos, m.T, m.d, fs, ft, same, tb.cs_src, tb.cs_tgt, tb.cs16,
                                tb.cs16_tgt, hs);
    if (e != hipSuccess) return fail(KVX_ERR_HIP, "RoPE table launch: %s", hipGetErrorString(e));
  }
  kvx::FitArgs a;
  std::memset(&a, 0, sizeof(a));
  a.src = static_cast<const uint16_t*>(src);
  a.tgt = static_cast<const uint16_t*>(tgt);
  a.cs_src = tb.cs_src;
  a.cs_tgt = tb.cs_tgt;
  size_t off = f.tables;
  a.planes = reinterpret_cast<uint16_t*>(w + off);
  off += f.planes;
  a.sums = reinterpret_cast<double*>(w + off);
  off += f.sums;
  a.sumsq = reinterpret_cast<double*>(w + off);
  off += f.sumsq;
  a.G = reinterpret_cast<float*>(w + off);
  off += f.G;
  a.Ascr = mode == 0 ? reinterpret_cast<double*>(w + off) : nullptr;
  off += f.A;
  a.Bscr = mode == 0 ? reinterpret_cast<double*>(w + off) : nullptr;
  off += f.B;
  void* plan = mode == 0 ? static_cast<void*>(w + off) : nullptr;
  a.W_K = wk;
  a.W_V = wv;
  a.b_K = bk;
  a.b_V = bv;
  a.r2 = r2;
  a.lam = lam;
  a.L_s = m.L_s;
  a.L_t = m.L_t;
  a.H = m.H;
  a.N = m.T;
  a.Npad = (int32_t)f.Npad;
  a.P = (m.L_s + m.L_t) * 2 * m.H;
  a.k = mode == 0 ? m.k : 1;
  a.style = rs->style;
  a.mode = mode;
  if (mode == 0)
    for (int64_t n = 0; n < (int64_t)m.L_t * m.k; ++n) a.idx[n] = (uint8_t)idx[n];
  e = kvx::launch_fit(a, plan, !planes_ready, hs);
  if (e != hipSuccess) return fail(KVX_ERR_HIP, "%s launch: %s", mode == 0 ? "fit" : "probe",
                                   hipGetErrorString(e));
  return ok();
}

// ---- MLP mapper (Sec. 4.4): validation, workspace layout and launches

struct MlpLayout {
  size_t tables, xs, act, total;
};

kvx_status check_mlp_dims(const kvx_dims* dims, int32_t F) {
  kvx_status st = check_dims(dims);
  if (st != KVX_OK) return st;
  const kvx_dims& m = *dims;
  if (F < 1) return fail(KVX_ERR_SHAPE, "hidden width F=%d must be >= 1", F);
  if (m.d != 128) return fail(KVX_ERR_UNSUPPORTED, "the MLP mapper is built for d = 128 (got %d)", m.d);
  if (m.k > kvx::kMaxMlpK)
    return fail(KVX_ERR_UNSUPPORTED, "the MLP mapper is built for k <= %d (got %d)", kvx::kMaxMlpK, m.k);
  if (F % 256) return fail(KVX_ERR_UNSUPPORTED, "hidden width F=%d is not a multiple of 256", F);
  if (((uint64_t)m.T + 512) * (uint64_t)F * 2 >= ((uint64_t)1 << 32) ||
      (uint64_t)F * F * 2 >= ((uint64_t)1 << 32))
    return fail(KVX_ERR_UNSUPPORTED, "T=%d, F=%d: an activation plane or W2 reaches 2^32 bytes",
                m.T, F);
  if ((int64_t)m.L_t * m.k > kvx::kMaxIdx)
    return fail(KVX_ERR_UNSUPPORTED, "L_t*k=%lld index entries exceed %d", (long long)m.L_t * m.k,
                kvx::kMaxIdx);
  return KVX_OK;
}

MlpLayout mlp_layout(const kvx_dims& m, int32_t F) {
  MlpLayout f;
  f.tables = tables_bytes(m);
  f.xs = up256((size_t)m.L_s * m.H * (size_t)m.T * m.d * 2);
  f.act = up256((size_t)2 * m.H * (size_t)m.T * F * 2);
  f.total = m.T == 0 ? 0 : f.tables + f.xs + 2 * f.act;
  return f;
}

kvx_status run_mlp(const kvx_dims* dims, kvx_dtype dtype, int32_t F, const void* src,
                   const int32_t* idx, const kvx_mlp* nk, const kvx_mlp* nv, const kvx_rope* rs,
                   const kvx_rope* rt, const int32_t* pos, void* tgt, void* ws, size_t wsb,
                   uint32_t flags, void* stream_, int l0, int nl) {
  kvx_status st = check_mlp_dims(dims, F);
  if (st != KVX_OK) return st;
  const kvx_dims& m = *dims;
  if (l0 < 0 || l0 + nl > m.L_t)
    return fail(KVX_ERR_INDEX, "target layer %d is outside [0, %d)", l0, m.L_t);
  if (dtype != KVX_BF16 && dtype != KVX_F32)
    return fail(KVX_ERR_DTYPE, "unknown dtype %d (0 = bf16, 1 = f32)", (int)dtype);
  if (dtype != KVX_BF16) return fail(KVX_ERR_UNSUPPORTED, "the MLP mapper is built for bf16 only");
  if ((st = check_rope(rs, "source")) != KVX_OK) return st;
  if ((st = check_rope(rt, "target")) != KVX_OK) return st;
  if (rs->style != rt->style)
    return fail(KVX_ERR_UNSUPPORTED, "source and target RoPE styles differ (%d vs %d)", rs->style,
                rt->style);
  if (idx == nullptr) return fail(KVX_ERR_NULL, "src_idx is NULL");
  if (nk == nullptr || nv == nullptr) return fail(KVX_ERR_NULL, "mlp_K or mlp_V is NULL");
  if (nk->W1 == nullptr || nk->W2 == nullptr || nk->W3 == nullptr || nv->W1 == nullptr ||
      nv->W2 == nullptr || nv->W3 == nullptr)
    return fail(KVX_ERR_NULL, "a weight matrix (W1, W2 or W3) is NULL");
  if (m.T > 0) {
    if (src == nullptr) return fail(KVX_ERR_NULL, "src_kv is NULL");
    if (pos == nullptr) return fail(KVX_ERR_NULL, "positions is NULL");
    if (tgt == nullptr) return fail(KVX_ERR_NULL, "target is NULL");
  }
  for (int l = l0; l < l0 + nl; ++l)
    for (int i = 0; i < m.k; ++i) {
      const int32_t s = idx[(int64_t)l * m.k + i];
      if (s < 0 || s >= m.L_s)
        return fail(KVX_ERR_INDEX, "src_idx[%d][%d]=%d is outside [0, %d)", l, i, s, m.L_s);
    }
  const uint64_t nets = (uint64_t)m.L_t * m.H;
  const uint64_t kd = (uint64_t)m.k * m.d;
  const uint64_t w1_b = nets * F * kd * 2, w2_b = nets * F * F * 2, w3_b = nets * m.d * F * 2;
  const uint64_t bF_b = nets * F * 2, bd_b = nets * m.d * 2;
  const uint64_t src_b = (uint64_t)m.L_s * 2 * m.H * (uint64_t)m.T * m.d * 2;
  const uint64_t pos_b = (uint64_t)m.T * 4;
  const uint64_t tgt_b = (uint64_t)m.L_t * 2 * m.H * (uint64_t)m.T * m.d * 2;
  struct In {
    const void* p;
    uint64_t b;
    const char* name;
  } ins[] = {{src, src_b, "src_kv"},     {nk->W1, w1_b, "W1_K"}, {nk->b1, bF_b, "b1_K"},
             {nk->W2, w2_b, "W2_K"},     {nk->b2, bF_b, "b2_K"}, {nk->W3, w3_b, "W3_K"},
             {nk->b3, bd_b, "b3_K"},     {nv->W1, w1_b, "W1_V"}, {nv->b1, bF_b, "b1_V"},
             {nv->W2, w2_b, "W2_V"},     {nv->b2, bF_b, "b2_V"}, {nv->W3, w3_b, "W3_V"},
             {nv->b3, bd_b, "b3_V"},     {pos, pos_b, "positions"}};
  for (const In& in : ins)
    if (in.p != nullptr && !aligned(in.p, in.p == pos ? 4 : 16))
      return fail(KVX_ERR_UNSUPPORTED, "%s is not %d-byte aligned", in.name, in.p == pos ? 4 : 16);
  if (tgt != nullptr && !aligned(tgt, 16)) return fail(KVX_ERR_UNSUPPORTED, "target is not 16-byte aligned");
  if (m.T == 0) return ok();   // nothing to map: the workspace is not touched
  const MlpLayout L = mlp_layout(m, F);
  if (ws == nullptr)
    return fail(KVX_ERR_WORKSPACE, "workspace is NULL (%llu bytes needed)", (unsigned long long)L.total);
  if (wsb < L.total)
    return fail(KVX_ERR_WORKSPACE, "workspace has %llu bytes, %llu needed", (unsigned long long)wsb,
                (unsigned long long)L.total);
  if (!aligned(ws, 256)) return fail(KVX_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  for (const In& in : ins) {
    if (overlap(tgt, tgt_b, in.p, in.b)) return fail(KVX_ERR_ALIAS, "target overlaps %s", in.name);
    if (overlap(ws, L.total, in.p, in.b)) return fail(KVX_ERR_ALIAS, "workspace overlaps %s", in.name);
  }
  if (overlap(tgt, tgt_b, ws, L.total)) return fail(KVX_ERR_ALIAS, "target overlaps workspace");

  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  const bool same = same_rope(*rs, *rt);
  const Tables tb = tables(m, ws, same);
  if (!(flags & KVX_FLAG_TABLES_READY)) {
    kvx::InvFreq fs, ft;
    inv_freq(*rs, m.d, fs);
    inv_freq(*rt, m.d, ft);
    hipError_t e = kvx::launch_rope_tables(pos, m.T, m.d, fs, ft, same, tb.cs_src, tb.cs_tgt,
                                           tb.cs16, tb.cs16_tgt, stream);
    if (e != hipSuccess) return fail(KVX_ERR_HIP, "RoPE table launch: %s", hipGetErrorString(e));
  }
  char* wsc = static_cast<char*>(ws);
  uint16_t* xs = reinterpret_cast<uint16_t*>(wsc + L.tables);
  uint16_t* act1 = reinterpret_cast<uint16_t*>(wsc + L.tables + L.xs);
  uint16_t* act2 = reinterpret_cast<uint16_t*>(wsc + L.tables + L.xs + L.act);
  if (!(flags & KVX_FLAG_KEYS_STRIPPED)) {
    hipError_t e = kvx::launch_strip_keys(static_cast<const uint16_t*>(src), tb.cs_src, xs, m.L_s,
                                          m.H, m.T, m.d, rs->style, stream);
    if (e != hipSuccess) return fail(KVX_ERR_HIP, "key strip launch: %s", hipGetErrorString(e));
  }
  kvx::MlpArgs a;
  std::memset(&a, 0, sizeof(a));
  a.src = static_cast<const uint16_t*>(src);
  a.xs = xs;
  a.cs_tgt = tb.cs_tgt;
  a.tgt = static_cast<uint16_t*>(tgt);
  a.T = m.T;
  a.H = m.H;
  a.k = m.k;
  a.F = F;
  const kvx_mlp* nets2[2] = {nk, nv};
  for (int l = l0; l < l0 + nl; ++l) {
    a.l = l;
    for (int i = 0; i < m.k; ++i) a.src_l[i] = idx[(int64_t)l * m.k + i];
    for (int layer = 1; layer <= 3; ++layer) {
      for (int kv = 0; kv < 2; ++kv) {
        const kvx_mlp& n = *nets2[kv];
        const void* w = layer == 1 ? n.W1 : layer == 2 ? n.W2 : n.W3;
        const void* b = layer == 1 ? n.b1 : layer == 2 ? n.b2 : n.b3;
        a.w[kv] = static_cast<const uint16_t*>(w);
        a.b[kv] = static_cast<const uint16_t*>(b);
      }
      a.act_in = layer == 2 ? act1 : act2;
      a.act_out = layer == 1 ? act1 : act2;
      hipError_t e = kvx::launch_mlp_layer(a, layer, rs->style, stream);
      if (e != hipSuccess)
        return fail(KVX_ERR_HIP, "MLP layer %d launch (target layer %d): %s", layer, l,
                    hipGetErrorString(e));
    }
  }
  return ok();
}

}  // namespace

namespace kvx {
kvx_status set_error(kvx_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}
}  // namespace kvx

extern "C" {

size_t kvx_workspace_bytes(const kvx_dims* dims, kvx_dtype dtype) {
  if (dims == nullptr || dims->T < 0 || dims->d < 2 || dims->d % 2) return 0;
  if (dtype != KVX_BF16 && dtype != KVX_F32) return 0;
  return ws_bytes(*dims, dtype);
}

kvx_status kvx_rope_prepare(const kvx_dims* dims, const kvx_rope* rope_src,
                            const kvx_rope* rope_tgt, const int32_t* positions,
                            void* workspace, size_t workspace_bytes, void* stream) {
  kvx_status st = check_dims(dims);
  if (st != KVX_OK) return st;
  if ((st = check_rope(rope_src, "source")) != KVX_OK) return st;
  if ((st = check_rope(rope_tgt, "target")) != KVX_OK) return st;
  const kvx_dims& m = *dims;
  if (m.T == 0) return ok();
  if (positions == nullptr) return fail(KVX_ERR_NULL, "positions is NULL");
  if (!aligned(positions, 4)) return fail(KVX_ERR_UNSUPPORTED, "positions must be 4-byte aligned");
  const size_t need = tables_bytes(m);   // the tables lead the workspace for every dtype
  if (workspace == nullptr) return fail(KVX_ERR_WORKSPACE, "workspace is NULL");
  if (workspace_bytes < need)
    return fail(KVX_ERR_WORKSPACE, "workspace has %llu bytes, %llu needed",
                (unsigned long long)workspace_bytes, (unsigned long long)need);
  if (!aligned(workspace, 256)) return fail(KVX_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (overlap(workspace, need, positions, (uint64_t)m.T * 4))
    return fail(KVX_ERR_ALIAS, "workspace overlaps positions");
  const bool same = same_rope(*rope_src, *rope_tgt);
  const Tables tb = tables(m, workspace, same);
  kvx::InvFreq fs, ft;
  inv_freq(*rope_src, m.d, fs);
  inv_freq(*rope_tgt, m.d, ft);
  hipError_t e = kvx::launch_rope_tables(positions, m.T, m.d, fs, ft, same, tb.cs_src,
                                         tb.cs_tgt, tb.cs16, tb.cs16_tgt,
                                         reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KVX_ERR_HIP, "RoPE table launch: %s", hipGetErrorString(e));
  return ok();
}

kvx_status kvx_map_cache(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                         const int32_t* src_idx, const void* W_K, const void* W_V,
                         const void* b_K, const void* b_V, const kvx_rope* rope_src,
                         const kvx_rope* rope_tgt, const int32_t* positions, void* tgt_kv,
                         void* workspace, size_t workspace_bytes, uint32_t flags,
                         void* stream) {
  Call c = make_call(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                     positions, tgt_kv, workspace, workspace_bytes, flags, stream);
  kvx_status st = check_dims(dims);
  if (st != KVX_OK) return st;
  return run(c);
}

kvx_status kvx_map_layer(const kvx_dims* dims, kvx_dtype dtype, int32_t l_t,
                         const void* src_kv, const int32_t* src_idx, const void* W_K,
                         const void* W_V, const void* b_K, const void* b_V,
                         const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                         const int32_t* positions, void* tgt_kv, void* workspace,
                         size_t workspace_bytes, uint32_t flags, void* stream) {
  Call c = make_call(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                     positions, tgt_kv, workspace, workspace_bytes, flags, stream);
  kvx_status st = check_dims(dims);
  if (st != KVX_OK) return st;
  if (l_t < 0 || l_t >= dims->L_t)
    return fail(KVX_ERR_INDEX, "l_t=%d is outside [0, %d)", l_t, dims->L_t);
  c.l0 = l_t;
  c.nl = 1;
  return run(c);
}

kvx_status kvx_map_cache_slots(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                               const int32_t* src_idx, const void* W_K, const void* W_V,
                               const void* b_K, const void* b_V, const kvx_rope* rope_src,
                               const kvx_rope* rope_tgt, const int32_t* positions,
                               const int32_t* slot_mapping, int64_t num_slots,
                               void* tgt_pool, void* workspace, size_t workspace_bytes,
                               uint32_t flags, void* stream) {
  Call c = make_call(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                     positions, tgt_pool, workspace, workspace_bytes, flags, stream);
  kvx_status st = check_dims(dims);
  if (st != KVX_OK) return st;
  if (num_slots < 1 || num_slots > 0x7fffffffLL)
    return fail(KVX_ERR_SHAPE, "num_slots=%lld must be in [1, 2^31)", (long long)num_slots);
  if (dims->T > 0 && slot_mapping == nullptr) return fail(KVX_ERR_NULL, "slot_mapping is NULL");
  if (tgt_pool == nullptr) return fail(KVX_ERR_NULL, "target pool is NULL");
  c.slots = slot_mapping;
  c.tgt_rows = num_slots;
  return run(c);
}

size_t kvx_xhead_workspace_bytes(const kvx_xdims* dims) {
  if (check_xdims(dims) != KVX_OK) return 0;
  return xws_bytes(*dims);
}

kvx_status kvx_map_cache_xhead(const kvx_xdims* dims, kvx_dtype dtype, const void* src_kv,
                               const int32_t* src_idx, const void* W_K, const void* W_V,
                               const void* b_K, const void* b_V, const kvx_rope* rope_src,
                               const kvx_rope* rope_tgt, const int32_t* positions, void* tgt_kv,
                               void* workspace, size_t workspace_bytes, uint32_t flags,
                               void* stream) {
  return run_xhead(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                   positions, tgt_kv, workspace, workspace_bytes, flags, stream, 0,
                   dims ? dims->L_t : 0, nullptr, 0, false);
}

kvx_status kvx_map_layer_xhead(const kvx_xdims* dims, kvx_dtype dtype, int32_t l_t,
                               const void* src_kv, const int32_t* src_idx, const void* W_K,
                               const void* W_V, const void* b_K, const void* b_V,
                               const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                               const int32_t* positions, void* tgt_kv, void* workspace,
                               size_t workspace_bytes, uint32_t flags, void* stream) {
  return run_xhead(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                   positions, tgt_kv, workspace, workspace_bytes, flags, stream, l_t, 1, nullptr,
                   0, false);
}

kvx_status kvx_map_cache_slots_xhead(const kvx_xdims* dims, kvx_dtype dtype, const void* src_kv,
                                     const int32_t* src_idx, const void* W_K, const void* W_V,
                                     const void* b_K, const void* b_V, const kvx_rope* rope_src,
                                     const kvx_rope* rope_tgt, const int32_t* positions,
                                     const int32_t* slot_mapping, int64_t num_slots,
                                     void* tgt_pool, void* workspace, size_t workspace_bytes,
                                     uint32_t flags, void* stream) {
  return run_xhead(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                   positions, tgt_pool, workspace, workspace_bytes, flags, stream, 0,
                   dims ? dims->L_t : 0, slot_mapping, num_slots, true);
}

size_t kvx_fit_workspace_bytes(const kvx_dims* dims) {
  if (check_fit_dims(dims, 0) != KVX_OK) return 0;
  return fit_layout(*dims, 0).total;
}

kvx_status kvx_fit_cache(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                         const int32_t* src_idx, const void* tgt_kv, const kvx_rope* rope_src,
                         const kvx_rope* rope_tgt, const int32_t* positions, double lambda,
                         float* W_K, float* W_V, float* b_K, float* b_V, void* workspace,
                         size_t workspace_bytes, uint32_t flags, void* stream) {
  return run_fit(dims, dtype, src_kv, src_idx, tgt_kv, rope_src, rope_tgt, positions, lambda, W_K,
                 W_V, b_K, b_V, nullptr, workspace, workspace_bytes, flags, stream, 0);
}

size_t kvx_probe_workspace_bytes(const kvx_dims* dims) {
  if (check_fit_dims(dims, 1) != KVX_OK) return 0;
  return fit_layout(*dims, 1).total;
}

kvx_status kvx_probe_r2(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                        const void* tgt_kv, const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                        const int32_t* positions, float* r2, void* workspace,
                        size_t workspace_bytes, uint32_t flags, void* stream) {
  return run_fit(dims, dtype, src_kv, nullptr, tgt_kv, rope_src, rope_tgt, positions, 0.0, nullptr,
                 nullptr, nullptr, nullptr, r2, workspace, workspace_bytes, flags, stream, 1);
}

kvx_status kvx_select_topk(int32_t L_s, int32_t L_t, int32_t H, int32_t k, const float* r2,
                           int32_t* src_idx, void* stream) {
  if (L_s < 1 || L_t < 1 || H < 1 || k < 1)
    return fail(KVX_ERR_SHAPE, "sizes out of range: L_s=%d L_t=%d H=%d k=%d", L_s, L_t, H, k);
  if (k > L_s) return fail(KVX_ERR_SHAPE, "k=%d exceeds L_s=%d", k, L_s);
  if (k > 32) return fail(KVX_ERR_UNSUPPORTED, "k=%d exceeds 32", k);
  if (r2 == nullptr || src_idx == nullptr) return fail(KVX_ERR_NULL, "R2 or the index output is NULL");
  if (!aligned(r2, 4) || !aligned(src_idx, 4))
    return fail(KVX_ERR_UNSUPPORTED, "R2 and the index output must be 4-byte aligned");
  if (overlap(r2, (uint64_t)L_s * L_t * H * 2 * 4, src_idx, (uint64_t)L_t * k * 4))
    return fail(KVX_ERR_ALIAS, "the index output overlaps R2");
  hipError_t e = kvx::launch_topk(r2, L_s, L_t, H, k, src_idx, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(KVX_ERR_HIP, "top-k launch: %s", hipGetErrorString(e));
  return ok();
}

size_t kvx_mlp_workspace_bytes(const kvx_dims* dims, int32_t F) {
  if (check_mlp_dims(dims, F) != KVX_OK) return 0;
  return mlp_layout(*dims, F).total;
}

kvx_status kvx_mlp_map_cache(const kvx_dims* dims, kvx_dtype dtype, int32_t F, const void* src_kv,
                             const int32_t* src_idx, const kvx_mlp* mlp_K, const kvx_mlp* mlp_V,
                             const kvx_rope* rope_src, const kvx_rope* rope_tgt,
                             const int32_t* positions, void* tgt_kv, void* workspace,
                             size_t workspace_bytes, uint32_t flags, void* stream) {
  return run_mlp(dims, dtype, F, src_kv, src_idx, mlp_K, mlp_V, rope_src, rope_tgt, positions,
                 tgt_kv, workspace, workspace_bytes, flags, stream, 0, dims ? dims->L_t : 0);
}

kvx_status kvx_mlp_map_layer(const kvx_dims* dims, kvx_dtype dtype, int32_t F, int32_t l_t,
                             const void* src_kv, const int32_t* src_idx, const kvx_mlp* mlp_K,
                             const kvx_mlp* mlp_V, const kvx_rope* rope_src,
                             const kvx_rope* rope_tgt, const int32_t* positions, void* tgt_kv,
                             void* workspace, size_t workspace_bytes, uint32_t flags,
                             void* stream) {
  return run_mlp(dims, dtype, F, src_kv, src_idx, mlp_K, mlp_V, rope_src, rope_tgt, positions,
                 tgt_kv, workspace, workspace_bytes, flags, stream, l_t, 1);
}

const char* kvx_last_error(void) { return g_err; }

int32_t kvx_version(void) { return 100; }

const char* kvx_map_kernel_name(const kvx_dims* dims, kvx_dtype dtype, int32_t n_layers) {
  if (dims == nullptr || (dtype != KVX_BF16 && dtype != KVX_F32) || n_layers < 1) return nullptr;
  switch (choose_kernel(dtype == KVX_BF16 ? 0 : 1, *dims, n_layers, dims->T, false, false)) {
    case Kernel::Ks: return "map_ks_kernel";
    case Kernel::Ks2: return "map_ks2_kernel";
    case Kernel::Sweep: return "map_sweep_kernel";
    case Kernel::W: return "map_w_kernel";
    default: return "map_kernel";
  }
}

}  // extern "C"
