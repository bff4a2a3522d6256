// kvx_map_cache_noalloc: kvx_map_cache for callers that cannot allocate
// device memory.  The workspace (RoPE tables, packed maps) lives in a
// file-scope device array instead of a caller buffer.
//
// Host code never passes the array's name to a kernel or a copy: in host
// code that name is only a stand-in, not the device address.  The device
// address is looked up once per device with hipGetSymbolAddress (with that
// device current) and kept; every call then hands that pointer to the
// existing entry point as its workspace.
#include <mutex>

#include "kvx.h"
#include "kvx_internal.h"

namespace {

// Device memory of the no-allocation entry point: every workspace
// kvx_workspace_bytes reports up to this size fits (the Qwen3-14B -> 32B
// shape at T = 32768 needs 184 MB; the Llama-3.1-8B -> 70B shape at T = 65536
// exactly 256 MiB).  Each device the library runs on holds one copy until the
// process ends.
static __device__ __align__(256) char scratch[KVX_SCRATCH_MAX_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

extern "C" {

kvx_status kvx_map_cache_noalloc(const kvx_dims* dims, kvx_dtype dtype, const void* src_kv,
                                 const int32_t* src_idx, const void* W_K, const void* W_V,
                                 const void* b_K, const void* b_V, const kvx_rope* rope_src,
                                 const kvx_rope* rope_tgt, const int32_t* positions,
                                 void* tgt_kv, uint32_t flags, void* stream) {
  // Sizes first, on the host: a call whose workspace would not fit is
  // rejected before any HIP call.
  if (dims != nullptr && (dtype == KVX_BF16 || dtype == KVX_F32)) {
    const size_t need = kvx_workspace_bytes(dims, dtype);
    if (need > (size_t)KVX_SCRATCH_MAX_BYTES)
      return kvx::set_error(KVX_ERR_WORKSPACE,
                           "kvx_map_cache_noalloc: this call needs %zu bytes of workspace, "
                           "more than the %zu bytes of the library's static scratch; use "
                           "kvx_map_cache with a caller workspace",
                           need, (size_t)KVX_SCRATCH_MAX_BYTES);
    if (need == 0)   // empty or invalid: no workspace is touched, the checks report
      return kvx_map_cache(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src,
                           rope_tgt, positions, tgt_kv, nullptr, 0, flags, stream);
  } else {
    // an invalid call: the regular checks report it, nothing is launched
    return kvx_map_cache(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                         positions, tgt_kv, nullptr, 0, flags, stream);
  }
  // the device of the launch stream (the current device for the null stream)
  int dev = -1;
  hipError_t e = stream != nullptr
                     ? hipStreamGetDevice(reinterpret_cast<hipStream_t>(stream), &dev)
                     : hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return kvx::set_error(KVX_ERR_HIP, "kvx_map_cache_noalloc: no device for the stream (%s)",
                         hipGetErrorString(e));
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_ptr[dev] == nullptr) {
      // with that device current: each device holds its own copy of the array
      int cur = -1;
      if ((e = hipGetDevice(&cur)) != hipSuccess)
        return kvx::set_error(KVX_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
      if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess)
        return kvx::set_error(KVX_ERR_HIP, "hipSetDevice(%d): %s", dev, hipGetErrorString(e));
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (cur != dev) (void)hipSetDevice(cur);
      if (e != hipSuccess || p == nullptr)
        return kvx::set_error(KVX_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                             hipGetErrorString(e));
      g_ptr[dev] = p;
    }
    ptr = g_ptr[dev];
  }
  return kvx_map_cache(dims, dtype, src_kv, src_idx, W_K, W_V, b_K, b_V, rope_src, rope_tgt,
                       positions, tgt_kv, ptr, (size_t)KVX_SCRATCH_MAX_BYTES, flags, stream);
}

}  // extern "C"
