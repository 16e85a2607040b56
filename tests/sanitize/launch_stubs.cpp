// Host-only stand-ins for the kernel launchers of libprecog, so that the
// C-ABI layer (csrc/precog_abi.cpp) links into a sanitizer build without
// device code.  The driver only takes argument paths that are refused (or
// are no-ops) before anything would be launched; a stub that is reached
// anyway fails the run.  Test infrastructure only.
#include <cstdio>
#include <cstdlib>

#include "precog_kernels.h"

namespace {
hipError_t reached(const char* fn) {
  std::fprintf(stderr, "launcher %s reached in a host-only build\n", fn);
  std::abort();
}
}  // namespace

namespace precog {
hipError_t launch_scan(const ScanParams&, int, int, int, int, hipStream_t) { return reached("scan"); }
hipError_t launch_scan_traj(const ScanParams&, int, int, int, int, hipStream_t) {
  return reached("scan_traj");
}
hipError_t launch_scan_complex(const ScanParams&, int, int, int, int, hipStream_t) {
  return reached("scan_complex");
}
hipError_t launch_retrieve(const RetrieveParams&, hipStream_t) { return reached("retrieve"); }
hipError_t launch_retrieve_screen(RetrieveParams&, hipStream_t) { return reached("retrieve_screen"); }
hipError_t launch_retrieve_decide(const RetrieveParams&, hipStream_t) {
  return reached("retrieve_decide");
}
hipError_t launch_query_scan(const ScanParams&, const RetrieveParams&, int, int, hipStream_t) {
  return reached("query_scan");
}
hipError_t launch_retrieve_prepare(const RetrieveParams&, hipStream_t) {
  return reached("retrieve_prepare");
}
hipError_t launch_gather(const GatherParams&, int, int, hipStream_t) { return reached("gather"); }
hipError_t launch_compose(const ComposeParams&, int, int, hipStream_t) { return reached("compose"); }
hipError_t launch_fuse(const FuseParams&, int, int, hipStream_t) { return reached("fuse"); }
hipError_t launch_route(const RouteParams&, hipStream_t) { return reached("route"); }
hipError_t launch_ema(const EmaParams&, int, int, hipStream_t) { return reached("ema"); }
}  // namespace precog
