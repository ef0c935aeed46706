// Host-only stand-ins for the HIP side of libsol, so that the C ABI's
// validation layer (sol_api.cpp) can be built with AddressSanitizer and
// UndefinedBehaviorSanitizer by the host compiler and exercised on a machine
// without a GPU.  Every launcher records that it was reached and returns
// success without touching its pointers; the range status reads as clear.
// Test infrastructure: never part of the product library.
#include "sol_internal.h"

namespace {
int g_launches = 0;
}

extern "C" int sol_stub_launches(void) { return g_launches; }

extern "C" const char* hipGetErrorString(hipError_t) { return "host stub"; }

// sol_noalloc.hip defines this entry point beside a device array, which a
// host compiler cannot build; here it only has to resolve.
extern "C" int sol_attn_fwd_noalloc(const void*, const void*, const void*, void*, int, int, int,
                                    int, int, int, int, const float*, sol_stream_t) {
  return sol::set_error(SOL_ERR_UNSUPPORTED, "host-only validation build");
}

namespace sol {

hipError_t launch_rope3d(const uint16_t*, uint16_t*, int64_t, const SeqGrid&, const float2*,
                         const float*, float, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_attn_fwd(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*, int,
                           const SeqGrid&, const float2*, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_prepare_kv(const uint16_t*, const uint16_t*, uint16_t*, uint16_t*, int,
                             const SeqGrid&, const float2*, int, int, const float*, float,
                             hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_attn_fwd_prepared(const uint16_t*, const uint16_t*, const uint16_t*, void*, int,
                                    const SeqGrid&, int, const float2*, const float*, float, int,
                                    const uint16_t*, const int*, int, hipStream_t, const uint8_t*,
                                    int) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_qkv_encode(const uint16_t*, const uint16_t*, const uint16_t*, uint8_t*, int, int,
                             const SeqGrid&, const float2*, const float*, const float*, float,
                             int64_t, int64_t, int64_t, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_qkv_decode(const uint8_t*, uint16_t*, uint16_t*, uint16_t*, int, int, int,
                             hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_prepare_kv_records(const uint8_t*, uint16_t*, uint16_t*, int, int, int, int, int,
                                     hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_sparse_route(const uint16_t*, const uint16_t*, int, const SeqGrid&, const float2*,
                               const float*, float, float, void*, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t launch_mfma_probe(const uint16_t*, float*, int, int, hipStream_t) {
  ++g_launches;
  return hipSuccess;
}

hipError_t range_status(unsigned* flags, bool) {
  *flags = 0;
  return hipSuccess;
}

}  // namespace sol
