// Drives the C ABI's host-side argument validation and size queries
// (csrc/precog_abi.cpp, csrc/noalloc.hip) in a host-only build with
// AddressSanitizer and UndefinedBehaviorSanitizer: every entry point with
// malformed arguments (each refusal status), the no-op cases that return
// before a launch, and the workspace / index size queries over ordinary and
// extreme sizes (where an overflowing product would be undefined behaviour).
// No device is touched.  Exits nonzero on a wrong status; the sanitizers
// abort on any invalid access or undefined arithmetic.  Test infrastructure
// only.
#include <cstdint>
#include <cstdio>

#include "precog.h"

// precog_status_string as a C caller declares and calls it: the status is an
// int of any value (the same symbol, under an int-taking prototype).
extern "C" const char* status_string_as_c(int code) __asm__("precog_status_string");

namespace {
int failures = 0;
void expect(precog_status got, precog_status want, int line) {
  if (got != want) {
    std::fprintf(stderr, "line %d: status %d, expected %d\n", line, got, want);
    ++failures;
  }
}
#define EXPECT(call, want) expect((call), (want), __LINE__)
void* const F = reinterpret_cast<void*>(0x10000);  // aligned, never dereferenced
const float* const FF = static_cast<const float*>(F);
const int32_t* const FI = static_cast<const int32_t*>(F);
const double* const FD = static_cast<const double*>(F);
void* const MIS = reinterpret_cast<void*>(0x10008);  // 8-byte aligned only

precog_scan_desc desc(int64_t b, int64_t l, int64_t d, int64_t n, int64_t chunk = 0,
                      precog_dtype in = PRECOG_BF16, precog_dtype out = PRECOG_F32,
                      precog_dtype st = PRECOG_F32, int64_t s0 = 0, int64_t s1 = 0) {
  precog_scan_desc x;
  x.batch = b; x.seqlen = l; x.dim = d; x.dstate = n;
  x.in_dtype = in; x.out_dtype = out; x.state_dtype = st;
  x.h0_batch_stride = s0; x.hT_batch_stride = s1; x.chunk = chunk;
  return x;
}
precog_status enc(const precog_scan_desc& d, const void* x = F, const void* y = F,
                  void* ws = nullptr, size_t wsb = 0, const void* C = F) {
  return precog_scan_encode(&d, x, F, FF, F, C, F, FF, nullptr, const_cast<void*>(y), F, ws, wsb,
                            nullptr);
}
}  // namespace

int main() {
  const int64_t big = INT64_MAX;
  // scan
  EXPECT(precog_scan_encode(nullptr, F, F, FF, F, F, F, FF, nullptr, F, F, nullptr, 0, nullptr),
         PRECOG_ERR_NULL);
  EXPECT(enc(desc(-1, 16, 64, 16)), PRECOG_ERR_SHAPE);
  EXPECT(enc(desc(2, -1, 64, 16)), PRECOG_ERR_SHAPE);
  EXPECT(enc(desc(2, 16, 64, 3)), PRECOG_ERR_SHAPE);
  EXPECT(enc(desc(big, big, big, 16)), PRECOG_ERR_SHAPE);
  EXPECT(enc(desc(2, big, 64, 16)), PRECOG_ERR_SHAPE);
  EXPECT(enc(desc(2, 16, 60, 16)), PRECOG_ERR_ALIGN);
  EXPECT(enc(desc(2, 16, 64, 16, 0, PRECOG_F16)), PRECOG_ERR_DTYPE);
  EXPECT(enc(desc(2, 16, 64, 16, 0, PRECOG_BF16, PRECOG_F32, PRECOG_F32, 64 * 16 - 8)),
         PRECOG_ERR_STRIDE);
  EXPECT(enc(desc(2, 16, 64, 16), nullptr), PRECOG_ERR_NULL);
  EXPECT(enc(desc(2, 16, 64, 16), MIS), PRECOG_ERR_ALIGN);
  EXPECT(enc(desc(2, 16, 64, 16), F, F, nullptr, 0, nullptr), PRECOG_ERR_NULL);  // C for y
  const precog_scan_desc chunked = desc(2, 1024, 64, 16, 128);
  const size_t need = precog_scan_workspace_bytes(&chunked);
  if (need == 0) ++failures;
  EXPECT(enc(chunked), PRECOG_ERR_WORKSPACE);
  EXPECT(enc(chunked, F, F, F, need - 1), PRECOG_ERR_WORKSPACE);
  EXPECT(enc(desc(0, 16, 64, 16)), PRECOG_OK);
  EXPECT(enc(desc(2, 16, 0, 16)), PRECOG_OK);
  EXPECT(precog_scan_encode_indexed(nullptr, F, F, FF, F, F, F, FF, F, 4, FI, nullptr, 1, 1.0, F,
                                    F, nullptr, 0, nullptr),
         PRECOG_ERR_NULL);
  {
    const precog_scan_desc g = desc(2, 16, 64, 16);
    EXPECT(precog_scan_encode_indexed(&g, F, F, FF, F, F, F, FF, F, 4, nullptr, nullptr, 1, 1.0,
                                      F, F, nullptr, 0, nullptr),
           PRECOG_ERR_NULL);
    EXPECT(precog_scan_encode_indexed(&g, F, F, FF, F, F, F, FF, F, 4, FI, FD, 65, 1.0, F, F,
                                      nullptr, 0, nullptr),
           PRECOG_ERR_SHAPE);
    EXPECT(precog_scan_encode_indexed(&g, F, F, FF, F, F, F, FF, F, 4, FI, FD, 3, 0.0, F, F,
                                      nullptr, 0, nullptr),
           PRECOG_ERR_SHAPE);
    EXPECT(precog_scan_trajectory(&g, F, F, FF, F, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr, 0, nullptr, 0, nullptr),
           PRECOG_ERR_SHAPE);
    EXPECT(precog_scan_trajectory(&g, F, F, FF, F, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr, 4, nullptr, 0, nullptr),
           PRECOG_ERR_NULL);
    EXPECT(precog_scan_trajectory(&g, F, F, FF, F, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr, 17, nullptr, 0, nullptr),
           PRECOG_OK);
  }
  // complex scan
  {
    const precog_scan_desc c32 = desc(2, 16, 64, 32);
    EXPECT(precog_scan_complex(&c32, F, F, FF, FF, F, F, F, FF, nullptr, F, F, nullptr, 0, nullptr),
           PRECOG_ERR_SHAPE);
    const precog_scan_desc cc = desc(2, 1024, 64, 16, 128);
    const size_t cneed = precog_scan_complex_workspace_bytes(&cc);
    if (cneed == 0) ++failures;
    EXPECT(precog_scan_complex(&cc, F, F, FF, FF, F, F, F, FF, nullptr, F, F, F, cneed - 1, nullptr),
           PRECOG_ERR_WORKSPACE);
    EXPECT(precog_scan_complex(&cc, F, F, FF, nullptr, F, F, F, FF, nullptr, F, F, F, cneed, nullptr),
           PRECOG_ERR_NULL);
  }
  // size queries over ordinary and extreme sizes
  const int64_t sizes[] = {0, 1, 7, 8, 64, 4096, 1LL << 20, 1LL << 31, 1LL << 40, big, -1, -big};
  for (int64_t a : sizes)
    for (int64_t b : sizes) {
      for (int64_t c : {int64_t(8), int64_t(16), int64_t(384), int64_t(4096), big}) {
        (void)precog_retrieve_workspace_bytes(a, b, c);
        (void)precog_retrieve_index_bytes(a, c);
        const precog_scan_desc d1 = desc(a, b, c, 16);
        const precog_scan_desc d2 = desc(a, b, c, 64, a);
        const precog_scan_desc d3 = desc(1, a, b, 8, c);
        (void)precog_scan_workspace_bytes(&d1);
        (void)precog_scan_workspace_bytes(&d2);
        (void)precog_scan_workspace_bytes(&d3);
        (void)precog_scan_complex_workspace_bytes(&d1);
        (void)precog_scan_complex_workspace_bytes(&d3);
      }
    }
  // retrieval
  const size_t rws = precog_retrieve_workspace_bytes(4, 10, 16);
  EXPECT(precog_retrieve_top1(FF, FF, -1, 10, 16, static_cast<int32_t*>(F), F, rws, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_retrieve_top1(FF, FF, 4, 10, 18, static_cast<int32_t*>(F), F, rws, nullptr),
         PRECOG_ERR_ALIGN);
  EXPECT(precog_retrieve_top1(FF, FF, 4, 10, 16, static_cast<int32_t*>(F), F, rws - 1, nullptr),
         PRECOG_ERR_WORKSPACE);
  EXPECT(precog_retrieve_top1(FF, FF, big, big, 16, static_cast<int32_t*>(F), F, rws, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_retrieve_top1(FF, FF, 0, 10, 16, nullptr, nullptr, 0, nullptr), PRECOG_OK);
  EXPECT(precog_retrieve_top1_noalloc(FF, FF, -1, 10, 16, static_cast<int32_t*>(F), nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_retrieve_top1_noalloc(FF, FF, 16384, 100000, 64, static_cast<int32_t*>(F), nullptr),
         PRECOG_ERR_WORKSPACE);
  EXPECT(precog_retrieve_top1_noalloc(FF, FF, big, big, 64, static_cast<int32_t*>(F), nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_retrieve_topk(FF, FF, 4, 10, 16, 0, static_cast<int32_t*>(F),
                              static_cast<double*>(F), F, rws, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_retrieve_topk(FF, FF, 4, 10, 16, 11, static_cast<int32_t*>(F),
                              static_cast<double*>(F), F, rws, nullptr),
         PRECOG_ERR_SHAPE);
  const size_t nb = precog_retrieve_index_bytes(10, 16);
  EXPECT(precog_retrieve_prepare(FF, 0, 16, F, nb, nullptr), PRECOG_ERR_SHAPE);
  EXPECT(precog_retrieve_prepare(FF, 10, 16, F, nb - 1, nullptr), PRECOG_ERR_WORKSPACE);
  EXPECT(precog_retrieve_topk_prepared(FF, FF, nullptr, nb, 4, 10, 16, 3, static_cast<int32_t*>(F),
                                       static_cast<double*>(F), F, rws, nullptr),
         PRECOG_ERR_NULL);
  // the query-time path in one call: both halves' arguments are checked
  {
    const precog_scan_desc qd = desc(4, 16, 64, 16);
    const size_t qws = precog_query_workspace_bytes(&qd, 10, 16);
    if (qws < rws) ++failures;
    EXPECT(precog_query_top1_prefill(&qd, FF, FF, nullptr, 0, 10, 16, F, static_cast<int32_t*>(F),
                                     F, F, FF, F, F, F, FF, F, F, F, qws - 1, nullptr),
           PRECOG_ERR_WORKSPACE);
    EXPECT(precog_query_top1_prefill(&qd, FF, FF, nullptr, 0, 10, 16, nullptr,
                                     static_cast<int32_t*>(F), F, F, FF, F, F, F, FF, F, F, F, qws,
                                     nullptr),
           PRECOG_ERR_NULL);
    EXPECT(precog_query_top1_prefill(&qd, FF, FF, F, nb - 1, 10, 16, F, static_cast<int32_t*>(F),
                                     F, F, FF, F, F, F, FF, F, F, F, qws, nullptr),
           PRECOG_ERR_WORKSPACE);
    EXPECT(precog_query_top1_prefill(&qd, FF, FF, nullptr, 0, big, 16, F, static_cast<int32_t*>(F),
                                     F, F, FF, F, F, F, FF, F, F, F, qws, nullptr),
           PRECOG_ERR_SHAPE);
    const precog_scan_desc q0 = desc(0, 16, 64, 16);
    EXPECT(precog_query_top1_prefill(&q0, nullptr, nullptr, nullptr, 0, 10, 16, nullptr, nullptr,
                                     nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                     nullptr, nullptr, nullptr, 0, nullptr),
           PRECOG_OK);
  }
  // injection
  EXPECT(precog_inject_gather(F, PRECOG_BF16, 10, 64, FI, 3, F, PRECOG_F32, nullptr),
         PRECOG_ERR_DTYPE);
  EXPECT(precog_inject_gather(F, PRECOG_F16, 10, 12, FI, 3, F, PRECOG_F32, nullptr),
         PRECOG_ERR_ALIGN);
  EXPECT(precog_inject_gather(F, PRECOG_F16, big, big - 7, FI, big, F, PRECOG_F32, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_inject_gather(F, PRECOG_F16, 10, 64, FI, 0, F, PRECOG_F32, nullptr), PRECOG_OK);
  EXPECT(precog_inject_compose(F, PRECOG_F16, 10, 64, FI, FD, 3, 0, 1.0, F, PRECOG_F32, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_inject_compose(F, PRECOG_F16, 10, 64, FI, FD, 3, 3, -1.0, F, PRECOG_F32, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_inject_fuse(F, 10, FI, FD, 3, F, 20, FI, FD, 3, PRECOG_F16, 64, 3, 7, 1.0, nullptr,
                            nullptr, 0, 1.0, F, PRECOG_F32, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_inject_fuse(F, 10, FI, FD, 3, F, 20, FI, FD, 3, PRECOG_F16, 64, 3, 3, 1.0, F,
                            nullptr, 4, 1.0, F, PRECOG_F32, nullptr),
         PRECOG_ERR_NULL);
  EXPECT(precog_inject_fuse(F, 10, FI, FD, 3, F, 20, FI, FD, 3, PRECOG_F16, 64, 0, 3, 1.0, nullptr,
                            nullptr, 0, 1.0, F, PRECOG_F32, nullptr),
         PRECOG_OK);
  // SMC
  EXPECT(precog_smc_route(FF, 3, 16, FF, 0, FF, 4, static_cast<int32_t*>(F),
                          static_cast<int32_t*>(F), nullptr, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_smc_route(FF, 0, 16, FF, 5, FF, 4, static_cast<int32_t*>(F),
                          static_cast<int32_t*>(F), nullptr, nullptr),
         PRECOG_OK);
  EXPECT(precog_smc_consolidate(F, PRECOG_F16, 20, 64, F, PRECOG_F16, FI, 5, 0.0, nullptr),
         PRECOG_ERR_SHAPE);
  EXPECT(precog_smc_consolidate(F, PRECOG_F16, 70000, 64, F, PRECOG_F16, FI, 5, 0.5, nullptr),
         PRECOG_ERR_SHAPE);
  // any int a C caller passes, including codes outside the enum
  for (int s : {-1, 0, 1, 8, 9, 99, 1 << 30})
    if (status_string_as_c(s) == nullptr) ++failures;
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("abi driver: all checks passed\n");
  return 0;
}
