// C-ABI layer of libprecog: host-side validation, chunk selection and
// launches.  Declared in include/precog.h.  Nothing here allocates, copies
// between host and device or synchronises.
#include "precog.h"

#include <cmath>

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>

#include "precog_kernels.h"

namespace {

constexpr int kMaxDevices = 64;
// 0 = unknown, 1 = gfx950, 2 = other architecture
std::atomic<int> g_arch_ok[kMaxDevices];
// compute units of each device (0 = not yet queried)
std::atomic<int> g_cus[kMaxDevices];

// Checks that the current device is a gfx950; `cus`, if given, receives its
// compute-unit count.  Both are queried once per device and cached.
precog_status check_device(int* cus = nullptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return PRECOG_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return PRECOG_ERR_ARCH;
  int st = g_arch_ok[dev].load(std::memory_order_relaxed);
  if (st == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return PRECOG_ERR_HIP;
    st = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    g_cus[dev].store(prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 1,
                     std::memory_order_relaxed);
    g_arch_ok[dev].store(st, std::memory_order_relaxed);
  }
  if (cus) *cus = g_cus[dev].load(std::memory_order_relaxed);
  return st == 1 ? PRECOG_OK : PRECOG_ERR_ARCH;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_n(int64_t n) {
  return n == 1 || n == 2 || n == 4 || n == 8 || n == 16 || n == 32 || n == 64;
}

constexpr int64_t kBlock = precog::kScanThreads;  // lanes per scan workgroup (real and complex A)
constexpr int64_t kTargetWaves = 2048;    // 2 waves per SIMD on 256 CUs
constexpr int64_t kMinAutoChunk = 8;

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int64_t auto_chunk(const precog_scan_desc* d);

// Longest chunk whose per-token streams stay addressable with the kernels'
// 32-bit buffer offsets: x, dt, z, y take D elements per token and B, C take
// N, at most 4 bytes each, so chunk * max(D, N) * 4 < 2^31.
int64_t max_chunk(const precog_scan_desc* d) {
  const int64_t w = d->dim > d->dstate ? d->dim : d->dstate;
  const int64_t row = (w > 0 ? w : 1) * 4;
  return ((1LL << 31) - 1) / row;
}

// Time-chunk length used for a descriptor (after validation).
int64_t effective_chunk(const precog_scan_desc* d) {
  const int64_t L = d->seqlen;
  if (L <= 0) return 1;
  const int64_t cap = max_chunk(d);
  if (d->chunk > 0) {
    const int64_t c = d->chunk >= L ? L : d->chunk;
    return c < cap ? c : cap;
  }
  if (L <= cap) return auto_chunk(d);
  const int64_t a = auto_chunk(d);
  return a < cap ? a : cap;
}

// Auto policy: one pass when batch x channel waves already fill the SIMDs;
// otherwise cut time so that about kTargetWaves waves run.
int64_t auto_chunk(const precog_scan_desc* d) {
  const int64_t L = d->seqlen;
  const int64_t lanes_per_channel = d->dstate > 16 ? d->dstate / 16 : 1;
  const int64_t waves = d->batch * ceil_div(d->dim * lanes_per_channel, 64);
  if (waves >= kTargetWaves || L <= 2 * kMinAutoChunk) return L;
  int64_t nch = ceil_div(kTargetWaves, waves > 0 ? waves : 1);
  const int64_t max_nch = L / kMinAutoChunk;
  if (nch > max_nch) nch = max_nch;
  if (nch <= 1) return L;
  return ceil_div(L, nch);
}

size_t align_up(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

struct ScanWs {
  size_t carry_bytes, dtsum_bytes, total;
};

ScanWs scan_ws(const precog_scan_desc* d, int64_t nchunks) {
  ScanWs w{0, 0, 0};
  if (nchunks <= 1) return w;
  w.carry_bytes = align_up(static_cast<size_t>(d->batch) * nchunks * d->dim * d->dstate * 4);
  w.dtsum_bytes = align_up(static_cast<size_t>(d->batch) * nchunks * d->dim * 4);
  w.total = w.carry_bytes + w.dtsum_bytes;
  return w;
}

precog_status validate_desc(const precog_scan_desc* d) {
  if (!d) return PRECOG_ERR_NULL;
  if (d->batch < 0 || d->seqlen < 0 || d->dim < 0 || d->chunk < 0) return PRECOG_ERR_SHAPE;
  if (!valid_n(d->dstate)) return PRECOG_ERR_SHAPE;
  if (d->batch > (1LL << 30) || d->dim > (1LL << 24) || d->seqlen > (1LL << 40))
    return PRECOG_ERR_SHAPE;
  if (d->in_dtype != PRECOG_F32 && d->in_dtype != PRECOG_BF16) return PRECOG_ERR_DTYPE;
  if (d->out_dtype != PRECOG_F32 && d->out_dtype != PRECOG_BF16) return PRECOG_ERR_DTYPE;
  if (d->state_dtype != PRECOG_F32 && d->state_dtype != PRECOG_F16) return PRECOG_ERR_DTYPE;
  const int64_t dn = d->dim * d->dstate;
  if (d->h0_batch_stride != 0 && d->h0_batch_stride < dn) return PRECOG_ERR_STRIDE;
  if (d->hT_batch_stride != 0 && d->hT_batch_stride < dn) return PRECOG_ERR_STRIDE;
  if (d->dim % 8 != 0) return PRECOG_ERR_ALIGN;
  if (d->h0_batch_stride % 8 != 0 || d->hT_batch_stride % 8 != 0) return PRECOG_ERR_ALIGN;
  return PRECOG_OK;
}

}  // namespace

extern "C" {

const char* precog_status_string(precog_status s) {
  // A C caller may pass any int: read the code as one, since loading an
  // enum object that holds a value outside the enum's range is undefined in
  // C++.
  int code = 0;
  std::memcpy(&code, &s, sizeof code);
  switch (code) {
    case static_cast<int>(PRECOG_OK): return "ok";
    case static_cast<int>(PRECOG_ERR_NULL): return "a required pointer is NULL";
    case static_cast<int>(PRECOG_ERR_SHAPE): return "unsupported or negative size";
    case static_cast<int>(PRECOG_ERR_DTYPE): return "unsupported dtype for this tensor";
    case static_cast<int>(PRECOG_ERR_STRIDE): return "state batch stride smaller than D*N";
    case static_cast<int>(PRECOG_ERR_ALIGN): return "pointer or size breaks the alignment rule";
    case static_cast<int>(PRECOG_ERR_WORKSPACE): return "workspace missing or too small";
    case static_cast<int>(PRECOG_ERR_ARCH): return "current device is not gfx950";
    case static_cast<int>(PRECOG_ERR_HIP): return "HIP runtime call or launch failed";
  }
  return "unknown status";
}

size_t precog_scan_workspace_bytes(const precog_scan_desc* desc) {
  if (validate_desc(desc) != PRECOG_OK) return 0;
  const int64_t ch = effective_chunk(desc);
  const int64_t nch = desc->seqlen > 0 ? ceil_div(desc->seqlen, ch) : 1;
  return scan_ws(desc, nch).total;
}

}  // extern "C"

namespace {
// precog_scan_encode, and with traj != NULL precog_scan_trajectory.
// Initial states taken from a state store (precog_scan_encode_indexed): batch
// row b starts from the h0_rows-row store h0 at row h0_idx[b] (h0_score
// NULL, k = 1) or from the softmax composition of rows h0_idx[b * k + j].
struct StoreStart {
  const int32_t* idx;
  int64_t rows;
  const double* score;
  int64_t k;
  double tau;
};

// Validates a scan call and fills `p` for its launch; `launch` is false when
// there is nothing to compute (the call returns PRECOG_OK without launching).
// Nothing is launched here.
precog_status scan_prepare(const precog_scan_desc* desc, const void* x, const void* dt,
                           const float* A, const void* B, const void* C, const void* z,
                           const float* Dskip, const void* h0, const StoreStart& from, void* y,
                           void* hT, void* traj, int64_t every, void* workspace,
                           size_t workspace_bytes, precog::ScanParams& p, bool& launch,
                           bool dev_check = true) {
  launch = false;
  const int32_t* h0_idx = from.idx;
  const int64_t h0_rows = from.rows;
  precog_status st = validate_desc(desc);
  if (st != PRECOG_OK) return st;
  const int64_t Bt = desc->batch, L = desc->seqlen, D = desc->dim, N = desc->dstate;
  if (Bt == 0 || D == 0) return PRECOG_OK;  // nothing to compute
  const bool work = L > 0;
  if (!A) return PRECOG_ERR_NULL;
  if (work && (!x || !dt || !B)) return PRECOG_ERR_NULL;
  if (work && y && !C) return PRECOG_ERR_NULL;
  const int64_t traj_count = traj ? L / every : 0;
  if (!y && !hT && traj_count == 0) return PRECOG_OK;  // nothing requested
  if (h0_idx && h0_rows < 0) return PRECOG_ERR_SHAPE;
  if (h0_idx && (from.k < 1 || from.k > precog::kMaxTopK || (!from.score && from.k != 1)))
    return PRECOG_ERR_SHAPE;
  if (from.score && (!(from.tau > 0.0) || !std::isfinite(from.tau))) return PRECOG_ERR_SHAPE;
  if (h0_idx && h0_rows > 0 && !h0) return PRECOG_ERR_NULL;
  const void* ptrs[] = {x, dt, A, B, C, z, Dskip, h0, h0_idx, from.score, y, hT, workspace, traj};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;

  const int64_t chunk = effective_chunk(desc);
  const int64_t nchunks = work ? ceil_div(L, chunk) : 1;
  if (nchunks > (1LL << 20)) return PRECOG_ERR_SHAPE;
  const ScanWs ws = scan_ws(desc, nchunks);
  if (ws.total > 0 && (!workspace || workspace_bytes < ws.total)) return PRECOG_ERR_WORKSPACE;
  // channels per workgroup: kBlock lanes, N / 16 lanes per channel when N > 16
  const int64_t lanes_per_channel = N > 16 ? N / 16 : 1;
  const int64_t dblocks = ceil_div(D, kBlock / lanes_per_channel);
  if (dblocks * Bt * nchunks > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if (Bt * D * N / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;

  int cus = 1;
  if (!dev_check) return PRECOG_OK;  // arguments checked, nothing prepared
  st = check_device(&cus);
  if (st != PRECOG_OK) return st;

  p = precog::ScanParams{};
  p.x = x;
  p.dt = dt;
  p.z = y ? z : nullptr;
  p.Bm = B;
  p.Cm = y ? C : nullptr;
  p.A = A;
  p.Dskip = y ? Dskip : nullptr;
  p.h0 = h0;
  p.h0_idx = h0_idx;
  p.h0_rows = h0_rows;
  p.h0_score = from.score;
  p.h0_k = static_cast<int>(from.k);
  p.h0_inv_tau = from.score ? 1.0 / from.tau : 1.0;
  p.y = work ? y : nullptr;
  p.hT = hT;
  p.carry = ws.total ? static_cast<float*>(workspace) : nullptr;
  p.dtsum = ws.total ? reinterpret_cast<float*>(static_cast<char*>(workspace) + ws.carry_bytes)
                     : nullptr;
  p.B = Bt;
  p.L = L;
  p.D = D;
  p.chunk = chunk;
  p.h0_stride = desc->h0_batch_stride ? desc->h0_batch_stride : D * N;
  p.hT_stride = desc->hT_batch_stride ? desc->hT_batch_stride : D * N;
  p.nchunks = static_cast<int>(nchunks);
  p.dblocks = static_cast<int>(dblocks);
  p.flags = (p.z ? precog::kHasZ : 0) | (p.Dskip ? precog::kHasD : 0) |
            ((h0 || h0_idx) ? precog::kHasH0 : 0) | (hT ? precog::kHasHT : 0);
  // Progress balancing between the two waves of a SIMD pays when every wave
  // of the launch is resident from the start (at most 4 per SIMD); in launches
  // of many rounds it was measured to cost time, so it is left off there.
  const int64_t final_waves = dblocks * Bt * nchunks * (kBlock / 64);
  if (final_waves <= 4LL * 4 * cus) p.flags |= precog::kBalance;
  p.traj = traj;
  p.traj_every = traj ? every : 1;
  p.traj_count = traj_count;
  if (!p.y && !p.hT && traj_count == 0) return PRECOG_OK;  // L == 0 and no state requested
  launch = true;
  return PRECOG_OK;
}

hipError_t scan_launch(const precog_scan_desc* desc, const precog::ScanParams& p, void* stream) {
  const int N = static_cast<int>(desc->dstate);
  return p.traj_count > 0
             ? precog::launch_scan_traj(p, N, desc->in_dtype, desc->out_dtype, desc->state_dtype,
                                        static_cast<hipStream_t>(stream))
             : precog::launch_scan(p, N, desc->in_dtype, desc->out_dtype, desc->state_dtype,
                                   static_cast<hipStream_t>(stream));
}

precog_status scan(const precog_scan_desc* desc, const void* x, const void* dt, const float* A,
                   const void* B, const void* C, const void* z, const float* Dskip,
                   const void* h0, const StoreStart& from, void* y, void* hT, void* traj,
                   int64_t every, void* workspace, size_t workspace_bytes, void* stream) {
  precog::ScanParams p;
  bool launch = false;
  const precog_status st = scan_prepare(desc, x, dt, A, B, C, z, Dskip, h0, from, y, hT, traj,
                                        every, workspace, workspace_bytes, p, launch);
  if (st != PRECOG_OK || !launch) return st;
  (void)hipGetLastError();
  return scan_launch(desc, p, stream) == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}
}  // namespace

extern "C" {

precog_status precog_scan_encode(const precog_scan_desc* desc, const void* x, const void* dt,
                                 const float* A, const void* B, const void* C, const void* z,
                                 const float* Dskip, const void* h0, void* y, void* hT,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  return scan(desc, x, dt, A, B, C, z, Dskip, h0, StoreStart{nullptr, 0, nullptr, 1, 1.0}, y, hT,
              nullptr, 1, workspace, workspace_bytes, stream);
}

precog_status precog_scan_encode_indexed(const precog_scan_desc* desc, const void* x,
                                         const void* dt, const float* A, const void* B,
                                         const void* C, const void* z, const float* Dskip,
                                         const void* store, int64_t store_rows,
                                         const int32_t* h0_idx, const double* h0_score,
                                         int64_t k, double tau, void* y, void* hT,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!h0_idx && desc && desc->batch > 0 && desc->dim > 0) return PRECOG_ERR_NULL;
  return scan(desc, x, dt, A, B, C, z, Dskip, store,
              StoreStart{h0_idx, store_rows, h0_score, k, tau}, y, hT, nullptr, 1, workspace,
              workspace_bytes, stream);
}

precog_status precog_scan_trajectory(const precog_scan_desc* desc, const void* x, const void* dt,
                                     const float* A, const void* B, const void* C, const void* z,
                                     const float* Dskip, const void* h0, void* y, void* hT,
                                     void* traj, int64_t every, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  if (every < 1) return PRECOG_ERR_SHAPE;
  // traj may be NULL only when nothing would be captured (L < every)
  if (!traj && desc && desc->seqlen >= every) return PRECOG_ERR_NULL;
  return scan(desc, x, dt, A, B, C, z, Dskip, h0, StoreStart{nullptr, 0, nullptr, 1, 1.0}, y, hT,
              traj, every, workspace, workspace_bytes, stream);
}

namespace {
// Retrieval workspace: query operands ([nqg, nks, 64] x 16 B), the screen's
// per-(query, 32-key block) summaries -- largest score [Q, nkb], second
// largest [Q, nkb], key of the largest [Q, nkb] (1 B) -- key norms [M] and
// block norms [nkb], each 256-byte aligned: about 9 Q M / 32 bytes.
struct RetrieveWs {
  size_t qop, blockmax, blocksec, blockarg, rownorm, blocknorm, total;
};
RetrieveWs retrieve_ws(int64_t Q, int64_t M, int64_t E) {
  RetrieveWs w;
  const size_t nkb = static_cast<size_t>((M + 31) / 32);
  const size_t qpw = 32 * precog::kRetWaves;  // queries per screen workgroup
  const size_t nqg = static_cast<size_t>((Q + qpw - 1) / qpw) * precog::kRetWaves;
  const size_t nks = static_cast<size_t>((E + 15) / 16);
  w.qop = align_up(nqg * nks * 64 * 16);
  w.blockmax = align_up(static_cast<size_t>(Q) * nkb * 4);
  w.blocksec = align_up(static_cast<size_t>(Q) * nkb * 4);
  w.blockarg = align_up(static_cast<size_t>(Q) * nkb);
  w.rownorm = align_up(static_cast<size_t>(M) * 4);
  w.blocknorm = align_up(nkb * 4);
  w.total = w.qop + w.blockmax + w.blocksec + w.blockarg + w.rownorm + w.blocknorm;
  return w;
}
}  // namespace

size_t precog_retrieve_workspace_bytes(int64_t Q, int64_t M, int64_t E) {
  if (Q < 0 || M < 0 || E < 4 || E > 4096 || E % 4 != 0) return 0;
  if (Q > 0x7fffffffLL || M > 0x7fffffffLL || ceil_div(M, 32) * ceil_div(Q, 128) > 0x7fffffffLL)
    return 0;
  return retrieve_ws(Q, M, E).total;
}

namespace {
// Prepared index: operands [nkb, nks, 2, 32] x 16 B, squared key norms [M],
// block norm maxima [nkb], each 256-byte aligned.
struct IndexLayout {
  size_t ops, rownorm, blocknorm, total;
};
IndexLayout index_layout(int64_t M, int64_t E) {
  IndexLayout l;
  const size_t nkb = static_cast<size_t>((M + 31) / 32);
  const size_t nks = static_cast<size_t>((E + 15) / 16);
  l.ops = align_up(nkb * nks * 64 * 16);
  l.rownorm = align_up(static_cast<size_t>(M) * 4);
  l.blocknorm = align_up(nkb * 4);
  l.total = l.ops + l.rownorm + l.blocknorm;
  return l;
}
}  // namespace

size_t precog_retrieve_index_bytes(int64_t M, int64_t E) {
  if (M < 1 || E < 4 || E > 4096 || E % 4 != 0 || M > 0x7fffffffLL) return 0;
  return index_layout(M, E).total;
}

precog_status precog_retrieve_prepare(const float* index_emb, int64_t M, int64_t E, void* prepared,
                                      size_t prepared_bytes, void* stream) {
  if (M < 1 || E < 4 || E > 4096 || M > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if (E % 4 != 0) return PRECOG_ERR_ALIGN;
  if (!index_emb || !prepared) return PRECOG_ERR_NULL;
  if (!aligned16(index_emb) || !aligned16(prepared)) return PRECOG_ERR_ALIGN;
  if (prepared_bytes < precog_retrieve_index_bytes(M, E)) return PRECOG_ERR_WORKSPACE;
  const int64_t nkb = ceil_div(M, 32);
  if (nkb * ((E + 15) / 16) * 64 / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;
  const IndexLayout l = index_layout(M, E);
  char* at = static_cast<char*>(prepared);
  precog::RetrieveParams p{};
  p.K = index_emb;
  p.kop = at;
  p.rownorm2 = reinterpret_cast<float*>(at + l.ops);
  p.blocknorm2 = reinterpret_cast<float*>(at + l.ops + l.rownorm);
  p.M = M;
  p.E = E;
  p.nkb = static_cast<int>(nkb);
  p.nks = static_cast<int>((E + 15) / 16);
  (void)hipGetLastError();
  const hipError_t e = precog::launch_retrieve_prepare(p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}

}  // extern "C"

namespace precog {
precog_status retrieve_setup(const float* query_emb, const float* index_emb, const void* prepared,
                             int64_t Q, int64_t M, int64_t E, int64_t k, int32_t* idx,
                             double* score, void* workspace, size_t workspace_bytes,
                             RetrieveParams& p, bool dev_check) {
  if (Q < 0 || M < 0 || E < 4 || E > 4096) return PRECOG_ERR_SHAPE;
  if (E % 4 != 0) return PRECOG_ERR_ALIGN;
  if (Q > 0x7fffffffLL || M > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  // screen workgroups (at most one per 32 keys and 128 queries) and the
  // workspace sizes must stay within their integer types
  if (ceil_div(M, 32) * ceil_div(Q, 128) > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  p = RetrieveParams{};
  if (Q == 0) return PRECOG_OK;
  if (!query_emb || !idx) return PRECOG_ERR_NULL;
  if (M > 0 && !index_emb) return PRECOG_ERR_NULL;
  const void* ptrs[] = {query_emb, index_emb, idx, workspace, score, prepared};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;
  const size_t need = precog_retrieve_workspace_bytes(Q, M, E);
  if (M > 0 && (!workspace || workspace_bytes < need)) return PRECOG_ERR_WORKSPACE;
  if (!dev_check) return PRECOG_OK;  // arguments checked, nothing prepared
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;

  const RetrieveWs w = retrieve_ws(Q, M, E);
  char* ws = static_cast<char*>(workspace);
  p.q = query_emb;
  p.K = index_emb;
  if (M > 0) {
    p.qop = ws;
    char* at = ws + w.qop;
    p.blockmax = reinterpret_cast<float*>(at);
    at += w.blockmax;
    p.blocksec = reinterpret_cast<float*>(at);
    at += w.blocksec;
    p.blockarg = reinterpret_cast<uint8_t*>(at);
    at += w.blockarg;
    p.rownorm2 = reinterpret_cast<float*>(at);
    at += w.rownorm;
    p.blocknorm2 = reinterpret_cast<float*>(at);
    if (prepared) {
      // operands and norms from the prepared index
      const IndexLayout l = index_layout(M, E);
      const char* pb = static_cast<const char*>(prepared);
      p.kop = pb;
      p.rownorm2 = reinterpret_cast<float*>(const_cast<char*>(pb + l.ops));
      p.blocknorm2 = reinterpret_cast<float*>(const_cast<char*>(pb + l.ops + l.rownorm));
    }
  }
  p.idx = idx;
  p.score = score;
  p.Q = Q;
  p.M = M;
  p.E = E;
  p.nkb = static_cast<int>((M + 31) / 32);
  p.nqg = static_cast<int>((Q + 32 * precog::kRetWaves - 1) / (32 * precog::kRetWaves) *
                           precog::kRetWaves);
  p.nks = static_cast<int>((E + 15) / 16);
  p.k = static_cast<int>(k);
  return PRECOG_OK;
}

precog_status retrieve_entry(const float* query_emb, const float* index_emb, const void* prepared,
                             int64_t Q, int64_t M, int64_t E, int64_t k, int32_t* idx,
                             double* score, void* workspace, size_t workspace_bytes,
                             void* stream) {
  RetrieveParams p;
  const precog_status st = retrieve_setup(query_emb, index_emb, prepared, Q, M, E, k, idx, score,
                                          workspace, workspace_bytes, p, true);
  if (st != PRECOG_OK || Q == 0) return st;
  (void)hipGetLastError();
  const hipError_t e = precog::launch_retrieve(p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}
}  // namespace precog

extern "C" {

precog_status precog_retrieve_top1(const float* query_emb, const float* index_emb, int64_t Q,
                                   int64_t M, int64_t E, int32_t* idx, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  return precog::retrieve_entry(query_emb, index_emb, nullptr, Q, M, E, 1, idx, nullptr, workspace,
                  workspace_bytes, stream);
}

precog_status precog_retrieve_topk(const float* query_emb, const float* index_emb, int64_t Q,
                                   int64_t M, int64_t E, int64_t k, int32_t* idx, double* score,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  if (k < 1 || k > precog::kMaxTopK || k > M) return PRECOG_ERR_SHAPE;
  return precog::retrieve_entry(query_emb, index_emb, nullptr, Q, M, E, k, idx, score, workspace,
                  workspace_bytes, stream);
}

precog_status precog_retrieve_topk_prepared(const float* query_emb, const float* index_emb,
                                            const void* prepared, size_t prepared_bytes, int64_t Q,
                                            int64_t M, int64_t E, int64_t k, int32_t* idx,
                                            double* score, void* workspace, size_t workspace_bytes,
                                            void* stream) {
  if (k < 1 || k > precog::kMaxTopK || k > M) return PRECOG_ERR_SHAPE;
  if (!prepared) return PRECOG_ERR_NULL;
  if (prepared_bytes < precog_retrieve_index_bytes(M, E)) return PRECOG_ERR_WORKSPACE;
  return precog::retrieve_entry(query_emb, index_emb, prepared, Q, M, E, k, idx, score, workspace,
                  workspace_bytes, stream);
}

size_t precog_query_workspace_bytes(const precog_scan_desc* desc, int64_t M, int64_t E) {
  if (validate_desc(desc) != PRECOG_OK) return 0;
  const size_t r = precog_retrieve_workspace_bytes(desc->batch, M, E);
  if (r == 0) return 0;
  return align_up(r) + precog_scan_workspace_bytes(desc);
}

// Retrieval workspace first, then the scan's (time chunks only), 256-byte
// aligned.
precog_status precog_query_top1_prefill(const precog_scan_desc* desc, const float* query_emb,
                                        const float* index_emb, const void* prepared,
                                        size_t prepared_bytes, int64_t M, int64_t E,
                                        const void* state_store, int32_t* idx, const void* x,
                                        const void* dt, const float* A, const void* B,
                                        const void* C, const void* z, const float* Dskip,
                                        void* y, void* hT, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  precog_status st = validate_desc(desc);
  if (st != PRECOG_OK) return st;
  const int64_t Q = desc->batch;
  if (prepared && prepared_bytes < precog_retrieve_index_bytes(M, E)) return PRECOG_ERR_WORKSPACE;
  const size_t rbytes = precog_retrieve_workspace_bytes(Q, M, E);
  const size_t roff = align_up(rbytes);
  void* sws = workspace && workspace_bytes > roff ? static_cast<char*>(workspace) + roff : nullptr;
  const size_t sbytes = workspace_bytes > roff ? workspace_bytes - roff : 0;
  const StoreStart from{idx, M, nullptr, 1, 1.0};
  precog::RetrieveParams rp;
  precog::ScanParams p;
  bool launch = false;
  // every argument of both halves first, then the device
  for (const bool dev : {false, true}) {
    st = precog::retrieve_setup(query_emb, index_emb, prepared, Q, M, E, 1, idx, nullptr,
                                workspace, workspace_bytes, rp, dev);
    if (st != PRECOG_OK || Q == 0) return st;
    st = scan_prepare(desc, x, dt, A, B, C, z, Dskip, state_store, from, y, hT, nullptr, 1, sws,
                      sbytes, p, launch, dev);
    if (st != PRECOG_OK) return st;
  }
  (void)hipGetLastError();
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = precog::launch_retrieve_screen(rp, s);
  if (e == hipSuccess) {
    const bool fused = launch && desc->dstate == 16 && desc->in_dtype == PRECOG_BF16 &&
                       p.nchunks == 1 && (p.y == nullptr || (p.flags & precog::kHasZ));
    if (fused) {
      e = precog::launch_query_scan(p, rp, desc->out_dtype, desc->state_dtype, s);
    } else {
      e = precog::launch_retrieve_decide(rp, s);
      if (e == hipSuccess && launch) e = scan_launch(desc, p, stream);
    }
  }
  return e == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}

precog_status precog_inject_gather(const void* state_store, precog_dtype store_dtype, int64_t M,
                                   int64_t S, const int32_t* idx, int64_t Q, void* h0,
                                   precog_dtype h0_dtype, void* stream) {
  if (M < 0 || S < 0 || Q < 0) return PRECOG_ERR_SHAPE;
  if ((store_dtype != PRECOG_F32 && store_dtype != PRECOG_F16) ||
      (h0_dtype != PRECOG_F32 && h0_dtype != PRECOG_F16))
    return PRECOG_ERR_DTYPE;
  if (S % 8 != 0) return PRECOG_ERR_ALIGN;
  if (Q == 0 || S == 0) return PRECOG_OK;
  if (!idx || !h0 || (M > 0 && !state_store)) return PRECOG_ERR_NULL;
  const void* ptrs[] = {state_store, idx, h0};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;
  if (S / 8 / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;

  (void)hipGetLastError();
  const int out_bytes = h0_dtype == PRECOG_F32 ? 4 : 2;
  // gridDim.y is limited to 65535: walk the queries in slices.
  for (int64_t q0 = 0; q0 < Q; q0 += 65535) {
    precog::GatherParams p{};
    p.store = state_store;
    p.idx = idx + q0;
    p.out = static_cast<char*>(h0) + q0 * S * out_bytes;
    p.M = M;
    p.S = S;
    p.Q = (Q - q0) < 65535 ? (Q - q0) : 65535;
    const hipError_t e = precog::launch_gather(p, store_dtype, h0_dtype,
                                               static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return PRECOG_ERR_HIP;
  }
  return PRECOG_OK;
}

precog_status precog_inject_compose(const void* state_store, precog_dtype store_dtype, int64_t M,
                                    int64_t S, const int32_t* idx, const double* score, int64_t Q,
                                    int64_t k, double tau, void* h0, precog_dtype h0_dtype,
                                    void* stream) {
  if (M < 0 || S < 0 || Q < 0 || k < 1 || k > precog::kMaxTopK) return PRECOG_ERR_SHAPE;
  if (!(tau > 0.0) || !std::isfinite(tau)) return PRECOG_ERR_SHAPE;
  if ((store_dtype != PRECOG_F32 && store_dtype != PRECOG_F16) ||
      (h0_dtype != PRECOG_F32 && h0_dtype != PRECOG_F16))
    return PRECOG_ERR_DTYPE;
  if (S % 8 != 0) return PRECOG_ERR_ALIGN;
  if (Q == 0 || S == 0) return PRECOG_OK;
  if (!idx || !score || !h0 || (M > 0 && !state_store)) return PRECOG_ERR_NULL;
  const void* ptrs[] = {state_store, idx, score, h0};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;
  if (S / 8 / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;

  (void)hipGetLastError();
  const int out_bytes = h0_dtype == PRECOG_F32 ? 4 : 2;
  for (int64_t q0 = 0; q0 < Q; q0 += 65535) {
    precog::ComposeParams p{};
    p.store = state_store;
    p.idx = idx + q0 * k;
    p.score = score + q0 * k;
    p.out = static_cast<char*>(h0) + q0 * S * out_bytes;
    p.M = M;
    p.S = S;
    p.Q = (Q - q0) < 65535 ? (Q - q0) : 65535;
    p.k = static_cast<int>(k);
    p.inv_tau = 1.0 / tau;
    const hipError_t e = precog::launch_compose(p, store_dtype, h0_dtype,
                                                static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return PRECOG_ERR_HIP;
  }
  return PRECOG_OK;
}

precog_status precog_inject_fuse(const void* episodic_store, int64_t episodic_rows,
                                 const int32_t* episodic_idx, const double* episodic_score,
                                 int64_t episodic_k, const void* corpus_store, int64_t corpus_rows,
                                 const int32_t* corpus_idx, const double* corpus_score,
                                 int64_t corpus_k, precog_dtype store_dtype, int64_t S, int64_t Q,
                                 int64_t k, double tau, const void* semantic,
                                 const int32_t* semantic_row, int64_t semantic_rows,
                                 double lambda, void* h0, precog_dtype h0_dtype, void* stream) {
  if (episodic_rows < 0 || corpus_rows < 0 || S < 0 || Q < 0 || semantic_rows < 0)
    return PRECOG_ERR_SHAPE;
  if (episodic_k < 0 || episodic_k > precog::kMaxTopK || corpus_k < 0 ||
      corpus_k > precog::kMaxTopK || k < 1 || k > precog::kMaxTopK ||
      k > episodic_k + corpus_k)
    return PRECOG_ERR_SHAPE;
  if (!(tau > 0.0) || !std::isfinite(tau) || !std::isfinite(lambda)) return PRECOG_ERR_SHAPE;
  if ((store_dtype != PRECOG_F32 && store_dtype != PRECOG_F16) ||
      (h0_dtype != PRECOG_F32 && h0_dtype != PRECOG_F16))
    return PRECOG_ERR_DTYPE;
  if (S % 8 != 0) return PRECOG_ERR_ALIGN;
  if (Q == 0 || S == 0) return PRECOG_OK;
  if (!h0) return PRECOG_ERR_NULL;
  if (episodic_k > 0 && (!episodic_idx || !episodic_score || (episodic_rows > 0 && !episodic_store)))
    return PRECOG_ERR_NULL;
  if (corpus_k > 0 && (!corpus_idx || !corpus_score || (corpus_rows > 0 && !corpus_store)))
    return PRECOG_ERR_NULL;
  if (semantic && !semantic_row) return PRECOG_ERR_NULL;
  const void* ptrs[] = {episodic_store, episodic_idx, episodic_score, corpus_store, corpus_idx,
                        corpus_score, semantic, semantic_row, h0};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;
  if (S / 8 / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;

  (void)hipGetLastError();
  const int out_bytes = h0_dtype == PRECOG_F32 ? 4 : 2;
  // gridDim.y is limited to 65535: walk the queries in slices
  for (int64_t q0 = 0; q0 < Q; q0 += 65535) {
    precog::FuseParams p{};
    p.store[0] = episodic_store;
    p.store[1] = corpus_store;
    p.rows[0] = episodic_rows;
    p.rows[1] = corpus_rows;
    p.idx[0] = episodic_k ? episodic_idx + q0 * episodic_k : nullptr;
    p.idx[1] = corpus_k ? corpus_idx + q0 * corpus_k : nullptr;
    p.score[0] = episodic_k ? episodic_score + q0 * episodic_k : nullptr;
    p.score[1] = corpus_k ? corpus_score + q0 * corpus_k : nullptr;
    p.kk[0] = static_cast<int>(episodic_k);
    p.kk[1] = static_cast<int>(corpus_k);
    p.sem = semantic;
    p.sem_row = semantic ? semantic_row + q0 : nullptr;
    p.sem_rows = semantic_rows;
    p.lambda = static_cast<float>(lambda);
    p.out = static_cast<char*>(h0) + q0 * S * out_bytes;
    p.S = S;
    p.Q = (Q - q0) < 65535 ? (Q - q0) : 65535;
    p.k = static_cast<int>(k);
    p.inv_tau = 1.0 / tau;
    const hipError_t e = precog::launch_fuse(p, store_dtype, h0_dtype,
                                             static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return PRECOG_ERR_HIP;
  }
  return PRECOG_OK;
}

precog_status precog_smc_route(const float* emb, int64_t C, int64_t E, const float* domain_protos,
                              int64_t n_domains, const float* sub_protos, int64_t n_sub,
                              int32_t* domain_out, int32_t* sub_out, int32_t* flat_out,
                              void* stream) {
  if (C < 0 || E < 4 || E > 4096 || n_domains < 1 || n_domains > 64 || n_sub < 1 || n_sub > 64)
    return PRECOG_ERR_SHAPE;
  if (E % 4 != 0) return PRECOG_ERR_ALIGN;
  if (C > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if (C == 0) return PRECOG_OK;
  if (!emb || !domain_protos || !sub_protos || !domain_out || !sub_out) return PRECOG_ERR_NULL;
  const void* ptrs[] = {emb, domain_protos, sub_protos, domain_out, sub_out, flat_out};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;
  precog::RouteParams p{};
  p.emb = emb;
  p.dom = domain_protos;
  p.sub = sub_protos;
  p.dom_out = domain_out;
  p.sub_out = sub_out;
  p.flat_out = flat_out;
  p.C = C;
  p.E = E;
  p.ndom = static_cast<int>(n_domains);
  p.nsub = static_cast<int>(n_sub);
  (void)hipGetLastError();
  const hipError_t e = precog::launch_route(p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}

precog_status precog_smc_consolidate(void* states, precog_dtype state_dtype, int64_t R, int64_t S,
                                     const void* contrib, precog_dtype contrib_dtype,
                                     const int32_t* target, int64_t C, double alpha,
                                     void* stream) {
  if (R < 0 || S < 0 || C < 0) return PRECOG_ERR_SHAPE;
  if (!(alpha > 0.0 && alpha <= 1.0)) return PRECOG_ERR_SHAPE;
  if ((state_dtype != PRECOG_F32 && state_dtype != PRECOG_F16) ||
      (contrib_dtype != PRECOG_F32 && contrib_dtype != PRECOG_F16))
    return PRECOG_ERR_DTYPE;
  if (S % 8 != 0) return PRECOG_ERR_ALIGN;
  if (R == 0 || S == 0 || C == 0) return PRECOG_OK;
  if (R > 65535 || S / 8 / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if (!states || !contrib || !target) return PRECOG_ERR_NULL;
  const void* ptrs[] = {states, contrib, target};
  for (const void* p : ptrs)
    if (!aligned16(p)) return PRECOG_ERR_ALIGN;
  const precog_status st = check_device();
  if (st != PRECOG_OK) return st;
  precog::EmaParams p{};
  p.states = states;
  p.contrib = contrib;
  p.target = target;
  p.R = R;
  p.S = S;
  p.C = C;
  p.alpha = static_cast<float>(alpha);
  p.one_minus_alpha = static_cast<float>(1.0 - alpha);
  (void)hipGetLastError();
  const hipError_t e = precog::launch_ema(p, state_dtype, contrib_dtype,
                                          static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}

namespace {
// Complex-A validation shared by the entry point and its workspace query:
// N <= 16, state strides counted in (re, im) pairs.
precog_status validate_complex_desc(const precog_scan_desc* desc) {
  const precog_status st = validate_desc(desc);
  if (st != PRECOG_OK) return st;
  if (desc->dstate > 16) return PRECOG_ERR_SHAPE;
  const int64_t dn2 = 2 * desc->dim * desc->dstate;
  if ((desc->h0_batch_stride != 0 && desc->h0_batch_stride < dn2) ||
      (desc->hT_batch_stride != 0 && desc->hT_batch_stride < dn2))
    return PRECOG_ERR_STRIDE;
  return PRECOG_OK;
}

// Complex-A workspace: carries [B, C, D, N, 2] fp32 and chunk dt sums
// [B, C, D] fp32, each 256-byte aligned.
ScanWs complex_ws(const precog_scan_desc* d, int64_t nchunks) {
  ScanWs w{0, 0, 0};
  if (nchunks <= 1) return w;
  w.carry_bytes = align_up(static_cast<size_t>(d->batch) * nchunks * d->dim * d->dstate * 2 * 4);
  w.dtsum_bytes = align_up(static_cast<size_t>(d->batch) * nchunks * d->dim * 4);
  w.total = w.carry_bytes + w.dtsum_bytes;
  return w;
}
}  // namespace

size_t precog_scan_complex_workspace_bytes(const precog_scan_desc* desc) {
  if (validate_complex_desc(desc) != PRECOG_OK) return 0;
  const int64_t ch = effective_chunk(desc);
  const int64_t nch = desc->seqlen > 0 ? ceil_div(desc->seqlen, ch) : 1;
  return complex_ws(desc, nch).total;
}

precog_status precog_scan_complex(const precog_scan_desc* desc, const void* x, const void* dt,
                                  const float* A_re, const float* A_im, const void* B,
                                  const void* C, const void* z, const float* Dskip,
                                  const void* h0, void* y, void* hT, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  precog_status st = validate_complex_desc(desc);
  if (st != PRECOG_OK) return st;
  const int64_t Bt = desc->batch, L = desc->seqlen, D = desc->dim, N = desc->dstate;
  if (Bt == 0 || D == 0) return PRECOG_OK;
  const bool work = L > 0;
  if (!A_re || !A_im) return PRECOG_ERR_NULL;
  if (work && (!x || !dt || !B)) return PRECOG_ERR_NULL;
  if (work && y && !C) return PRECOG_ERR_NULL;
  if ((!y || !work) && !hT) return PRECOG_OK;  // nothing requested
  const void* ptrs[] = {x, dt, A_re, A_im, B, C, z, Dskip, h0, y, hT, workspace};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return PRECOG_ERR_ALIGN;
  const int64_t chunk = effective_chunk(desc);
  const int64_t nchunks = work ? ceil_div(L, chunk) : 1;
  if (nchunks > (1LL << 20)) return PRECOG_ERR_SHAPE;
  const ScanWs ws = complex_ws(desc, nchunks);
  if (ws.total > 0 && (!workspace || workspace_bytes < ws.total)) return PRECOG_ERR_WORKSPACE;
  const int64_t dblocks = ceil_div(D, kBlock);
  if (dblocks * Bt * nchunks > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  if (Bt * D * N / 256 + 1 > 0x7fffffffLL) return PRECOG_ERR_SHAPE;
  int cus = 1;
  st = check_device(&cus);
  if (st != PRECOG_OK) return st;

  precog::ScanParams p{};
  p.x = x;
  p.dt = dt;
  p.z = y ? z : nullptr;
  p.Bm = B;
  p.Cm = y ? C : nullptr;
  p.A = A_re;
  p.A_im = A_im;
  p.Dskip = y ? Dskip : nullptr;
  p.h0 = h0;
  p.y = work ? y : nullptr;
  p.hT = hT;
  p.carry = ws.total ? static_cast<float*>(workspace) : nullptr;
  p.dtsum = ws.total ? reinterpret_cast<float*>(static_cast<char*>(workspace) + ws.carry_bytes)
                     : nullptr;
  p.B = Bt;
  p.L = L;
  p.D = D;
  p.chunk = chunk;
  p.h0_stride = desc->h0_batch_stride ? desc->h0_batch_stride : 2 * D * N;
  p.hT_stride = desc->hT_batch_stride ? desc->hT_batch_stride : 2 * D * N;
  p.nchunks = static_cast<int>(nchunks);
  p.dblocks = static_cast<int>(dblocks);
  p.flags = (p.z ? precog::kHasZ : 0) | (p.Dskip ? precog::kHasD : 0) |
            (h0 ? precog::kHasH0 : 0) | (hT ? precog::kHasHT : 0);
  // progress balancing when every wave of the final pass is resident from
  // the start (as for the real-A scan)
  if (dblocks * Bt * nchunks * (kBlock / 64) <= 4LL * 4 * cus) p.flags |= precog::kBalance;
  if (!p.y && !p.hT) return PRECOG_OK;  // L == 0 and no state requested
  (void)hipGetLastError();
  const hipError_t e = precog::launch_scan_complex(p, static_cast<int>(N), desc->in_dtype,
                                                   desc->out_dtype, desc->state_dtype,
                                                   static_cast<hipStream_t>(stream));
  return e == hipSuccess ? PRECOG_OK : PRECOG_ERR_HIP;
}

}  // extern "C"
