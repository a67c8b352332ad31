// Per-XCD memory latency and affinity probe (placeholder until measured).
#include <hip/hip_runtime.h>

#include "internal.h"

namespace asym {

int probe_latency_run(int device, Topology& t) {
  (void)device;
  (void)t;
  return fail(ASYM_EUNSUPPORTED, "latency probe not built yet");
}

}  // namespace asym
