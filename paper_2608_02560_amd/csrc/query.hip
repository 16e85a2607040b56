// The query-time path of Sec. 4.2 after the retrieval's screen: the exact
// top-1 decision, the injection of that stored state and the query prefill
// (Eq. 1) in one launch (query_scan_kernel in scan_kernels.h).
#include "scan_kernels.h"

namespace precog {

hipError_t launch_query_scan(const ScanParams& p, const RetrieveParams& rp, int out_dtype,
                             int state_dtype, hipStream_t s) {
  if (p.nchunks != 1 || p.h0_score != nullptr) return hipErrorInvalidValue;
  const bf16_t* X = static_cast<const bf16_t*>(p.x);
  const bf16_t* DT = static_cast<const bf16_t*>(p.dt);
  const bf16_t* Z = static_cast<const bf16_t*>(p.z);
  const bf16_t* BB = static_cast<const bf16_t*>(p.Bm);
  const bf16_t* CC = static_cast<const bf16_t*>(p.Cm);
  const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(p.dblocks) * p.B));
  const dim3 block(kSBlock);
  if (p.y != nullptr && (p.flags & kHasZ)) {
    if (out_dtype == 0 && state_dtype == 0)
      hipLaunchKernelGGL((query_scan_kernel<16, bf16_t, float, float, kReadout, true>), grid, block, 0,
                         s, X, DT, Z, BB, CC, static_cast<float*>(p.y), p, rp);
    else if (out_dtype == 0)
      hipLaunchKernelGGL((query_scan_kernel<16, bf16_t, float, f16_t, kReadout, true>), grid, block, 0,
                         s, X, DT, Z, BB, CC, static_cast<float*>(p.y), p, rp);
    else if (state_dtype == 0)
      hipLaunchKernelGGL((query_scan_kernel<16, bf16_t, bf16_t, float, kReadout, true>), grid, block,
                         0, s, X, DT, Z, BB, CC, static_cast<bf16_t*>(p.y), p, rp);
    else
      hipLaunchKernelGGL((query_scan_kernel<16, bf16_t, bf16_t, f16_t, kReadout, true>), grid, block,
                         0, s, X, DT, Z, BB, CC, static_cast<bf16_t*>(p.y), p, rp);
  } else if (p.y == nullptr) {
    if (state_dtype == 0)
      hipLaunchKernelGGL((query_scan_kernel<16, bf16_t, float, float, kStateOnly, false>), grid, block,
                         0, s, X, DT, Z, BB, CC, static_cast<float*>(nullptr), p, rp);
    else
      hipLaunchKernelGGL((query_scan_kernel<16, bf16_t, float, f16_t, kStateOnly, false>), grid, block,
                         0, s, X, DT, Z, BB, CC, static_cast<float*>(nullptr), p, rp);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace precog
