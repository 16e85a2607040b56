// Selective-SSM scan that also captures the thinned state trajectory of the
// SMC encode (Sec. 5.1 Eq. smc-trajectory; the fidelity dial of Sec. 5.2).
// Same kernels as scan.hip, instantiated with trajectory capture on.
#include "scan_kernels.h"

namespace precog {

hipError_t launch_scan_traj(const ScanParams& p, int N, int in_dtype, int out_dtype,
                            int state_dtype, hipStream_t s) {
  return launch_scan_n<true>(p, N, in_dtype, out_dtype, state_dtype, s);
}

}  // namespace precog
