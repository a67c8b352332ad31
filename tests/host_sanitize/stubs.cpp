// Stand-ins for the GPU-side symbols the host-only sources reference, so that
// they link into a plain g++ build with sanitizers (no HIP runtime, no GPU).
// Every stand-in that would touch a device reports ASYM_EUNSUPPORTED.  Test
// infrastructure only.
#include <string>

#include "../../paper_2609_24270_amd/csrc/internal.h"

namespace asym {
static std::string g_err;
int fail(int status, const std::string& msg) {
  g_err = msg;
  return status;
}
int hip_fail(hipError_t, const char* what) {
  g_err = what;
  return ASYM_EHIP;
}
int latency_measure(int, LatencyMeasure&) { return fail(ASYM_EUNSUPPORTED, "host build: no GPU"); }
int attn_page_tokens() { return 32; }
}  // namespace asym

extern "C" const char* asym_last_error(void) { return asym::g_err.c_str(); }
extern "C" int asym_device_query(int, asym_device_info*) { return asym::fail(ASYM_EUNSUPPORTED, "host build"); }
hipError_t hipSetDevice(int) { return hipErrorNoDevice; }
hipError_t hipMemGetInfo(size_t*, size_t*) { return hipErrorNoDevice; }
