// Gated selective-SSM prefill scan (Eq. 1, Sec. 3): the launcher of the
// plain encode.  The kernels and their design are in scan_kernels.h; the
// trajectory-capturing variants are instantiated in scan_traj.hip.
#include "scan_kernels.h"

namespace precog {

hipError_t launch_scan(const ScanParams& p, int N, int in_dtype, int out_dtype,
                       int state_dtype, hipStream_t s) {
  return launch_scan_n<false>(p, N, in_dtype, out_dtype, state_dtype, s);
}

}  // namespace precog
