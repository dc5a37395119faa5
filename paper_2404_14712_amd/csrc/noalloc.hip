// Allocation-free attention backward: the same kernels as
// orbit_attention_bwd, with their scratch (the per-row softmax-gradient
// offsets, the per-head feature sums of q and k and the column-reduction
// partials) in a library-owned device array instead of a caller workspace.
//
// Each GPU the library runs on holds its own copy of `scratch` until the
// process ends. Host code never passes the array's name to a kernel (in host
// code it names a host-side stand-in, not device memory): the device address
// of the current device's copy is looked up once per device with
// hipGetSymbolAddress and kept.
#include <mutex>

#include "kernels.h"

namespace {

constexpr size_t kScratchBytes = ORBIT_ATTN_BWD_NOALLOC_MAX_SCRATCH;  // per device
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// device address of the current device's scratch array
orbit_status scratch_address(const char* fn, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    orbit::set_error("%s: no usable current device (%s, device %d)", fn, hipGetErrorString(e), dev);
    return ORBIT_E_DEVICE;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      orbit::set_error("%s: hipGetSymbolAddress of the scratch array failed on device %d: %s", fn, dev,
                       hipGetErrorString(e));
      return ORBIT_E_DEVICE;
    }
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return ORBIT_OK;
}

}  // namespace

extern "C" {

orbit_status orbit_attention_bwd_noalloc(int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim,
                                         const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v,
                                         int64_t ldv, const void* o, int64_t ldo, int32_t o_f32, const float* lse,
                                         const void* dO, int64_t lddo, void* dq, void* dk, void* dv, int64_t ldg,
                                         void* stream) {
  const char* fn = "orbit_attention_bwd_noalloc";
  orbit::clear_error();
  ORBIT_TRY(orbit::attention_bwd_check(fn, dtype, B, H, L, head_dim, q, ldq, k, ldk, v, ldv, o, ldo, lse, dO, lddo,
                                       dq, dk, dv, ldg));
  const size_t need = orbit::attn_bwd_workspace_bytes(B, H, L, head_dim);
  if (need > kScratchBytes) {
    orbit::set_error("%s: B=%d H=%d L=%d head_dim=%d needs %zu bytes of scratch, more than the %zu bytes the "
                     "library holds per device (use orbit_attention_bwd with a workspace)",
                     fn, B, H, L, head_dim, need, kScratchBytes);
    return ORBIT_E_UNSUPPORTED;
  }
  void* ptr = nullptr;
  ORBIT_TRY(scratch_address(fn, &ptr));
  orbit::AttnIO io{q, k, v, ldq, ldk, ldv, B, H, L, head_dim};
  return orbit::attn_bwd((orbit_dtype)dtype, io, o, ldo, o_f32 ? 1 : 0, lse, dO, lddo, dq, dk, dv, ldg,
                         static_cast<float*>(ptr), static_cast<hipStream_t>(stream));
}

}  // extern "C"
