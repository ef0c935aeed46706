// sol_attn_fwd_noalloc: the prepared attention path (sol_attn_fwd_ws) on a
// workspace the library holds itself, for callers that cannot allocate device
// memory.  The workspace is one file-scope device array per GPU; host code
// reaches it only through the address hipGetSymbolAddress returns for the
// current device (the array's name in host code is not a device address).
#include <mutex>

#include "sol.h"
#include "sol_internal.h"

namespace {

constexpr size_t kScratchBytes = SOL_NOALLOC_MAX_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mutex;
void* g_scratch_ptr[kMaxDevices];  // per device, resolved on its first call

}  // namespace

extern "C" int sol_attn_fwd_noalloc(const void* q, const void* k, const void* v, void* out, int B,
                                    int H, int N, int D, int T, int Hl, int Wl,
                                    const float* rope_tab_dev, sol_stream_t stream) {
  const size_t need = sol_attn_workspace_bytes(B, H, N, D);
  if (need == 0)  // invalid sizes: the full validation below reports them
    return sol_attn_fwd_ws(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab_dev, nullptr, 0, stream);
  if (need > kScratchBytes)
    return sol::set_error(SOL_ERR_UNSUPPORTED,
                         "sol_attn_fwd_noalloc: this call needs a workspace larger than the "
                         "library's static one (SOL_NOALLOC_MAX_BYTES = 256 MiB); use "
                         "sol_attn_fwd_ws with a workspace of sol_attn_workspace_bytes()");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return sol::set_error(SOL_ERR_HIP, "sol_attn_fwd_noalloc: no current HIP device");
  void* ptr;
  {
    std::lock_guard<std::mutex> lock(g_mutex);
    if (!g_scratch_ptr[dev]) {
      void* p = nullptr;
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return sol::set_error(SOL_ERR_HIP, "sol_attn_fwd_noalloc: hipGetSymbolAddress failed");
      g_scratch_ptr[dev] = p;
    }
    ptr = g_scratch_ptr[dev];
  }
  return sol_attn_fwd_ws(q, k, v, out, B, H, N, D, T, Hl, Wl, rope_tab_dev, ptr, kScratchBytes, stream);
}
