// Gated selective-SSM prefill scan for gfx950 (MI355X).
//
// Computes, per batch row b and channel d (Eq. 1, Sec. 3, with real A > 0):
//   h_t[n] = exp(-dt_t A[n]) h_{t-1}[n] + B_t[n] x_t dt_t
//   y_t    = (sum_n C_t[n] h_t[n] + Dskip x_t) * silu(z_t)
// from an injected h0, capturing hT = h_L (Sec. 4.2).
//
// Work decomposition (two levels over time):
//   * One lane owns one (b, d) channel and keeps its N state values in VGPRs,
//     walking a time chunk sequentially.  The 64 lanes of a wave are 64
//     adjacent channels, so every per-token load of x / dt / z and store of y
//     is one contiguous 128-byte (bf16) or 256-byte (fp32) segment.  For
//     N > 16, N / 16 lanes share a channel, 16 states each.
//   * B_t and C_t are shared by all channels of a row.  Lane l loads element
//     16 j + (l mod 16) into register j, so one register holds 16 state
//     coefficients replicated in each 16-lane DPP row; coefficient n reaches
//     every lane through the DPP row_newbcast:n operand modifier of the very
//     instruction that consumes it (v_mul_f32 for B_t[n] x_t dt_t,
//     v_fmac_f32 for C_t[n] h_t[n]).  The broadcast is free and B_t / C_t
//     cost 2 N / 16 loads and conversions per lane and token.
//   * When batch x channels alone cannot fill the 1024 SIMDs, the sequence is
//     cut into C time chunks (level 2):
//       pass 1 (summary): each chunk except the last is scanned from a zero
//              state; its end state and sum of dt are written to workspace;
//       pass 2 (carry):   per (b, d, n), H_c = exp(-A sum dt_{c-1}) H_{c-1}
//              + s_{c-1} (the composition of the affine maps h -> a h + s
//              that each chunk applies, App. A): sequential over chunks, or
//              for 9 to 64 chunks over few lanes a scan over the chunks'
//              maps within one wave;
//       pass 3 (replay):  each chunk is rescanned from its carried-in state,
//              producing y and, for the last chunk, hT.
//     The carried state is exact up to fp32 reassociation (Theorem 1 applied
//     at every chunk boundary).
//
// Per (token, channel, state): one v_mul (dt A'), one v_exp_f32, one
// v_mul_dpp (B x dt), one v_fmac (state) and one v_fmac_dpp (readout).  A is
// prescaled by -log2(e) once per lane, so exp(-dt A) = exp2(dt A').  The
// running state is always fp32.
#pragma once

#include <type_traits>
#include <utility>

#include "compose.h"
#include "decide.h"
#include "precog_kernels.h"

namespace precog {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kSBlock = kScanThreads;    // scan workgroups (real and complex A): 8 waves

constexpr int kSWaves = kSBlock / 64;

// Progress balancing (launches whose waves are all resident at once; the
// host sets kBalance).  Waves are placed on the four SIMDs of a CU in order,
// so waves w and w + 4 of an 8-wave workgroup share one.  Issue arbitration
// between waves of equal priority favours the older one, so with equal work
// one of the two would run well ahead and the other would finish its
// sequence alone on the SIMD, where a single wave issues at about half the
// rate of two.  Instead each wave publishes its tile count in LDS and, at
// the head of each iteration of its time loop, takes priority 0 while ahead
// of its partner and 1 otherwise, so the two advance together.  (Dead waves
// stay at 0; their live partners then run at priority 0, which changes
// nothing.)
__device__ __forceinline__ bool balance_enabled(const ScanParams& p) {
  return kSWaves == 8 && (p.flags & kBalance) != 0;
}
// Before any wave of the workgroup can leave: every wave starts at 0.
__device__ __forceinline__ void balance_init(int* progress, int wave) {
  __atomic_store_n(&progress[wave], 0, __ATOMIC_RELAXED);
  __syncthreads();
}
__device__ __forceinline__ void balance_step(int* progress, int wave, int tile) {
  __atomic_store_n(&progress[wave], tile, __ATOMIC_RELAXED);
  const int other = __builtin_amdgcn_readfirstlane(
      __atomic_load_n(&progress[wave ^ (kSWaves / 2)], __ATOMIC_RELAXED));
  if (tile > other)
    __builtin_amdgcn_s_setprio(0);
  else
    __builtin_amdgcn_s_setprio(1);
}
// Time steps of inputs per pipeline tile.  The plain scan kinds use 4: it
// keeps the readout kernel at 121 VGPRs (4 waves per SIMD), which lets short
// launches such as a 32-token query prefill over 4096 waves run in one round
// and helps the chunked passes, at no cost to the corpus encode (2 waves per
// SIMD either way).  Trajectory capture keeps 8: its state stores share the
// vector-memory counter with the tile loads, and longer tiles wait on them
// less often.
constexpr int kPFPlain = 4;
constexpr int kPFWide = 8;  // trajectory capture, complex-A kernel

enum Kind { kReadout = 0, kStateOnly = 1, kSummary = 2 };



__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v.bits) << 16);
}
__device__ __forceinline__ float to_f32(f16_t v) {
  return static_cast<float>(__builtin_bit_cast(_Float16, v.bits));
}

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  return bf16_t{__builtin_bit_cast(uint16_t, static_cast<__bf16>(v))};  // RNE
}
template <> __device__ __forceinline__ f16_t from_f32<f16_t>(float v) {
  return f16_t{__builtin_bit_cast(uint16_t, static_cast<_Float16>(v))};  // RNE
}

// Per-token streams go through buffer instructions: the address is the
// descriptor base (a wave-uniform row pointer) + a per-lane byte offset in a
// VGPR + a per-token byte offset in an SGPR, summed by the memory unit, so
// the time loop spends no VALU work on addresses.  Stores from lanes whose
// offset is at or past num_records are dropped by the hardware range check.

template <typename T> struct Stream;
template <> struct Stream<float> {
  using raw = uint32_t;
  static __device__ __forceinline__ raw load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
  }
  static __device__ __forceinline__ float f32(raw v) { return __uint_as_float(v); }
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, voff, soff, 0);
  }
};
template <> struct Stream<bf16_t> {
  using raw = uint16_t;
  static __device__ __forceinline__ raw load(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
  }
  static __device__ __forceinline__ float f32(raw v) { return __uint_as_float(static_cast<uint32_t>(v) << 16); }
  static __device__ __forceinline__ void store(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, float v) {
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, static_cast<__bf16>(v)), r, voff, soff, 0);
  }
};

template <int N, typename TSt>
__device__ __forceinline__ void load_state(float (&h)[N], const TSt* src) {
#pragma unroll
  for (int n = 0; n < N; ++n) h[n] = to_f32(src[n]);
}
template <int N>
__device__ __forceinline__ void load_state(float (&h)[N], const float* src) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int n = 0; n < N; n += 4) {
      const float4 v = *reinterpret_cast<const float4*>(src + n);
      h[n] = v.x; h[n + 1] = v.y; h[n + 2] = v.z; h[n + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int n = 0; n < N; ++n) h[n] = src[n];
  }
}

// Row of the initial state of batch row b: h0 + b * stride, or, with an
// index (the injection h_init <- store[idx] fused into the scan),
// h0 + h0_idx[b] * stride; null when that index is outside the store.
template <typename TSt>
__device__ __forceinline__ const TSt* h0_row(const ScanParams& p, int64_t b) {
  int64_t row = b;
  if (p.h0_idx != nullptr) {
    row = p.h0_idx[b];
    if (row < 0 || row >= p.h0_rows) return nullptr;
  }
  return static_cast<const TSt*>(p.h0) + row * p.h0_stride;
}
// The same for a store row already known to the workgroup.
template <typename TSt>
__device__ __forceinline__ const TSt* store_row(const ScanParams& p, int64_t row) {
  if (row < 0 || row >= p.h0_rows) return nullptr;
  return static_cast<const TSt*>(p.h0) + row * p.h0_stride;
}

// Initial state composed from the k store rows of batch row b (the top-k
// injection fused into the scan): sum_j w_j store[idx_j] with the weights of
// compose.h, one fp32 fma per row in rank order, rounded to the state dtype
// as the composition kernel would store it; NaN when any index is outside the
// store.  These are the composition kernel's operations, so the result is
// the same bits.  `off` is this thread's first element within a row.
template <int NL, typename TSt>
__device__ __forceinline__ void compose_state(float (&h)[NL], const ScanParams& p, int64_t b,
                                              int64_t off) {
  const int k = p.h0_k;
  const int32_t* irow = p.h0_idx + b * k;
  bool bad = false;
  for (int j = 0; j < k; ++j) bad |= irow[j] < 0 || irow[j] >= p.h0_rows;
  if (bad) {
#pragma unroll
    for (int n = 0; n < NL; ++n) h[n] = __builtin_nanf("");
    return;
  }
  const double* srow = p.h0_score + b * k;
  const SoftmaxDen den = softmax_den(srow, k, p.h0_inv_tau);
  float acc[NL];
#pragma unroll
  for (int n = 0; n < NL; ++n) acc[n] = 0.f;
  for (int j = 0; j < k; ++j) {
    const float wj = softmax_weight(srow[j], den, p.h0_inv_tau);
    float v[NL];
    load_state<NL>(v, static_cast<const TSt*>(p.h0) + irow[j] * p.h0_stride + off);
#pragma unroll
    for (int n = 0; n < NL; ++n) acc[n] = fmaf(wj, v[n], acc[n]);
  }
#pragma unroll
  for (int n = 0; n < NL; ++n) h[n] = to_f32(from_f32<TSt>(acc[n]));
}

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(__double2loint(v)), lane);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(__double2hiint(v)), lane);
  return __hiloint2double(hi, lo);
}

// compose_state for a whole wave whose lanes share batch row b (the scan
// kernel): lane i < k forms exp((s_i - m) / tau) once and the others read it
// back, the denominator is summed in rank order from those values, and every
// lane forms w_j = e_j / den: the operations of compose.h, so the same bits,
// without every lane evaluating 2k exponentials.  The k rows' loads are
// unrolled so several are in flight.  Every lane of the wave must call it.
template <int NL, typename TSt>
__device__ __forceinline__ void compose_state_wave(float (&h)[NL], const ScanParams& p, int64_t b,
                                                   int64_t off) {
  const int k = p.h0_k;
  const int lane = threadIdx.x & 63;
  const bool on = lane < k;
  const double si = on ? p.h0_score[b * k + lane] : -INFINITY;
  const int32_t ii = on ? p.h0_idx[b * k + lane] : 0;
  if (__ballot(on && (ii < 0 || ii >= p.h0_rows)) != 0) {
#pragma unroll
    for (int n = 0; n < NL; ++n) h[n] = __builtin_nanf("");
    return;
  }
  double mx = readlane_f64(si, 0);
  for (int i = 1; i < k; ++i) mx = fmax(mx, readlane_f64(si, i));
  const double ei = on ? exp((si - mx) * p.h0_inv_tau) : 0.0;
  double den = 0.0;
  for (int i = 0; i < k; ++i) den += readlane_f64(ei, i);
  float acc[NL];
#pragma unroll
  for (int n = 0; n < NL; ++n) acc[n] = 0.f;
#pragma unroll 4
  for (int j = 0; j < k; ++j) {
    const float wj = static_cast<float>(readlane_f64(ei, j) / den);
    const int64_t row = __builtin_amdgcn_readlane(ii, j);
    float v[NL];
    load_state<NL>(v, static_cast<const TSt*>(p.h0) + row * p.h0_stride + off);
#pragma unroll
    for (int n = 0; n < NL; ++n) acc[n] = fmaf(wj, v[n], acc[n]);
  }
#pragma unroll
  for (int n = 0; n < NL; ++n) h[n] = to_f32(from_f32<TSt>(acc[n]));
}

template <int N, typename TSt>
__device__ __forceinline__ void store_state(TSt* dst, const float (&h)[N]) {
#pragma unroll
  for (int n = 0; n < N; ++n) dst[n] = from_f32<TSt>(h[n]);
}
template <int N>
__device__ __forceinline__ void store_state(float* dst, const float (&h)[N]) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int n = 0; n < N; n += 4)
      *reinterpret_cast<float4*>(dst + n) = make_float4(h[n], h[n + 1], h[n + 2], h[n + 3]);
  } else {
#pragma unroll
    for (int n = 0; n < N; ++n) dst[n] = h[n];
  }
}

// Trajectory rows: 16-byte stores (8 fp16 or 4 fp32 states) where the
// states allow it; fp16 rounds to nearest even.
typedef _Float16 st_half8 __attribute__((ext_vector_type(8)));
typedef float st_float8 __attribute__((ext_vector_type(8)));
template <int N, typename TSt>
__device__ __forceinline__ void store_state_vec(TSt* dst, const float (&h)[N]) {
  if constexpr (std::is_same<TSt, f16_t>::value && N % 8 == 0) {
#pragma unroll
    for (int n = 0; n < N; n += 8) {
      const st_float8 v = {h[n], h[n + 1], h[n + 2], h[n + 3], h[n + 4], h[n + 5], h[n + 6], h[n + 7]};
      *reinterpret_cast<st_half8*>(dst + n) = __builtin_convertvector(v, st_half8);
    }
  } else {
    store_state<N>(dst, h);
  }
}

// Value of lane 16 r + m broadcast to all 16 lanes of DPP row r.  The
// compiler folds the move into the consuming v_mul_f32 as a DPP operand.
template <int m>
__device__ __forceinline__ float row_bcast(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x150 + m, 0xf, 0xf, false));
}

// Same broadcast for a lane chosen at run time (short groups, N < 16).
__device__ __forceinline__ float row_bcast_rt(float v, int m) {
  const int src = (static_cast<int>(threadIdx.x) & 48) + m;  // lane 16 r + m, r = row of this lane
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src * 4, __builtin_bit_cast(int, v)));
}

// acc += sum_m bcast_m(c) h[16 g + m] over the states of group g, each term
// one v_fmac_f32 with the broadcast as its DPP operand.  The compiler does
// not form v_fmac_f32_dpp itself, so the group is one asm block (one block
// rather than one statement per term: the hazard recognizer pads every asm
// statement conservatively).  Inside the block the DPP source `c` is never
// written; it was last written by a VALU conversion before the block, and a
// DPP source needs two wait states after a VALU write, hence s_nop 1.
template <int N, int g>
__device__ __forceinline__ void readout_group(float& acc, float c, const float (&h)[N]) {
  constexpr int kPer = N < 16 ? N : 16;
  constexpr int o = 16 * g;
  if constexpr (kPer == 16) {
    asm("s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %1, %2 row_newbcast:0 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %3 row_newbcast:1 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %4 row_newbcast:2 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %5 row_newbcast:3 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %6 row_newbcast:4 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %7 row_newbcast:5 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %8 row_newbcast:6 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %9 row_newbcast:7 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %10 row_newbcast:8 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %11 row_newbcast:9 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %12 row_newbcast:10 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %13 row_newbcast:11 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %14 row_newbcast:12 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %15 row_newbcast:13 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %16 row_newbcast:14 row_mask:0xf bank_mask:0xf\n\t"
        "v_fmac_f32_dpp %0, %1, %17 row_newbcast:15 row_mask:0xf bank_mask:0xf"
        : "+v"(acc)
        : "v"(c), "v"(h[o + 0]), "v"(h[o + 1]), "v"(h[o + 2]), "v"(h[o + 3]), "v"(h[o + 4]),
          "v"(h[o + 5]), "v"(h[o + 6]), "v"(h[o + 7]), "v"(h[o + 8]), "v"(h[o + 9]),
          "v"(h[o + 10]), "v"(h[o + 11]), "v"(h[o + 12]), "v"(h[o + 13]), "v"(h[o + 14]),
          "v"(h[o + 15]));
  } else {
    // N < 16: short groups, one statement per term (only small test shapes).
#pragma unroll
    for (int m = 0; m < kPer; ++m) acc = fmaf(row_bcast_rt(c, m), h[o + m], acc);
  }
}

// One token for the 16 states n = 16 g + m, m = 0..15 (or fewer when N < 16).
template <int N, bool READOUT, int g, int... m>
__device__ __forceinline__ void token_group(float (&h)[N], const float (&a2)[N], float dtv, float u,
                                            float bv, float cv, float& acc,
                                            std::integer_sequence<int, m...>) {
  ((h[16 * g + m] = fmaf(__builtin_amdgcn_exp2f(dtv * a2[16 * g + m]), h[16 * g + m],
                         u * row_bcast<m>(bv))),
   ...);
  if constexpr (READOUT) readout_group<N, g>(acc, cv, h);
}

// One token for 16 states with B_t / C_t already in VGPRs (the same value in
// every lane): the same arithmetic, in the same order, as token_group.
template <int N, bool READOUT, int... m>
__device__ __forceinline__ void token_vgpr(float (&h)[N], const float (&a2)[N], float dtv, float u,
                                           const float (&bl)[16], const float (&cl)[16], float& acc,
                                           std::integer_sequence<int, m...>) {
  ((h[m] = fmaf(__builtin_amdgcn_exp2f(dtv * a2[m]), h[m], u * bl[m])), ...);
  if constexpr (READOUT) ((acc = fmaf(cl[m], h[m], acc)), ...);
}

template <int N, bool READOUT, int... g>
__device__ __forceinline__ void token(float (&h)[N], const float (&a2)[N], float dtv, float u,
                                      const float (&bv)[(N + 15) / 16], const float (&cv)[(N + 15) / 16],
                                      float& acc, std::integer_sequence<int, g...>) {
  constexpr int kPer = N < 16 ? N : 16;
  (token_group<N, READOUT, g>(h, a2, dtv, u, bv[g], cv[g], acc, std::make_integer_sequence<int, kPer>{}),
   ...);
}

// Lanes per channel: N > 16 states are split into groups of 16 held by
// different lanes, which keeps every lane at 16 states (fewer VGPRs, more
// resident waves) at the price of a cross-lane sum in the readout.
template <int N>
constexpr int kLanesPerChannel = N > 16 ? N / 16 : 1;

// Value held by lane (l xor m) of the wave, through the LDS crossbar.
__device__ __forceinline__ float lane_xor(float v, int m) {
  const int src = (static_cast<int>(threadIdx.x & 63) ^ m) * 4;
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, v)));
}

// One lane = one (b, d) channel over one time chunk.  HASZ: gate present.
//   KIND == kReadout:   y and (last chunk) hT
//   KIND == kStateOnly: hT only (y == NULL: C, z, Dskip unread)
//   KIND == kSummary:   chunk end state from zero -> carry slot c+1, sum dt
// TRAJ (readout and state-only kinds): also store the state after every
// token t with (t + 1) mod every == 0 into traj[b, (t + 1) / every - 1],
// the fidelity dial of the SMC trajectory (Sec. 5.1-5.2).  The countdown to
// the next captured token is wave-uniform, so the test costs scalar
// instructions only.
// Every lane of a wave stays active through the time loop (DPP broadcasts
// read other lanes); lanes past D compute on clamped channels and store
// nothing.
// DEC (the query-time prefill, one pass, a store row per batch row): batch
// row b is query b of the retrieval `rp`; wave 0 of the workgroup first
// decides the query's exact top-1 (decide_query, which also writes it to
// rp.idx), and the workgroup starts from that store row: one launch instead
// of the decide and the prefill.  The results are those of the two
// launches, bit for bit.
template <int N, typename TIn, typename TOut, typename TSt, int KIND, bool HASZ, int TRAJ, bool DEC>
__device__ __forceinline__ void scan_body(
    const TIn* __restrict__ xg, const TIn* __restrict__ dtg, const TIn* __restrict__ zg,
    const TIn* __restrict__ Bg, const TIn* __restrict__ Cg, TOut* __restrict__ yg,
    const ScanParams& p, const RetrieveParams* rp) {
  // P lanes share a channel when N > 16, one 16-state group each; group g
  // occupies DPP rows with (row mod P) == g, so every lane of a row needs the
  // same coefficients B_t[16 g + m] / C_t[16 g + m] from its row's lane m.
  constexpr int P = kLanesPerChannel<N>;
  constexpr int NL = N / P;                // states held by one lane
  constexpr int G = (NL + 15) / 16;        // registers per token for B_t (and C_t)
  constexpr int kChan = kSBlock / P;       // channels per workgroup
  constexpr int kPF = TRAJ != 0 ? kPFWide : kPFPlain;
  constexpr bool kRead = KIND == kReadout;
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int dblk = lb % p.dblocks;
  const int rest = lb / p.dblocks;
  const int b = rest % static_cast<int>(p.B);
  const int c = rest / static_cast<int>(p.B);
  const int64_t D = p.D;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = (lane >> 4) % P;  // this lane's state group
  // channel of this lane: 16 per row, rows of one channel set are P apart
  const int64_t wave_d0 = static_cast<int64_t>(dblk) * kChan + wave * (64 / P);

  // progress balancing: see balance_step
  const bool fair = balance_enabled(p);
  __shared__ int progress[kSWaves];
  if (fair) balance_init(progress, wave);  // uniform over the workgroup
  // whole wave past the last channel (DEC: wave 0 never is; the others
  // leave before the decision's barrier, which then waits for the waves
  // still running)
  if (wave_d0 >= D) return;
  const int64_t dtrue = wave_d0 + (lane & 15) + 16 * (lane / (16 * P));
  const bool live = dtrue < D;
  const int64_t d = live ? dtrue : D - 1;

  const int64_t t0 = static_cast<int64_t>(c) * p.chunk;
  const int64_t t1 = min(p.L, t0 + p.chunk);
  const int nsteps = static_cast<int>(t1 > t0 ? t1 - t0 : 0);

  // Decay exponents A' = -A log2(e): exp(-dt A) = exp2(dt A').
  const int64_t sofs = d * N + 16 * grp;  // this lane's states within a [D, N] row
  float a2[NL];
  load_state<NL>(a2, p.A + sofs);
#pragma unroll
  for (int n = 0; n < NL; ++n) a2[n] *= -kLog2e;

  // The initial state is read after the first tile's loads are issued: a
  // row taken from a state store first needs its index, and that round trip
  // then overlaps the tile's.
  float h[NL];
  int64_t row_known = 0;  // DEC: the decided store row
  auto init_state = [&]() {
    if constexpr (KIND == kSummary) {
#pragma unroll
      for (int n = 0; n < NL; ++n) h[n] = 0.f;
    } else {
      if (p.nchunks > 1) {
        load_state<NL>(h, p.carry + (static_cast<int64_t>(b) * p.nchunks + c) * D * N + sofs);
      } else if (p.h0_score != nullptr) {
        compose_state_wave<NL, TSt>(h, p, b, sofs);
      } else if (p.flags & kHasH0) {
        const TSt* src = DEC ? store_row<TSt>(p, row_known) : h0_row<TSt>(p, b);
        if (src != nullptr) {
          load_state<NL>(h, src + sofs);
        } else {
#pragma unroll
          for (int n = 0; n < NL; ++n) h[n] = __builtin_nanf("");
        }
      } else {
#pragma unroll
        for (int n = 0; n < NL; ++n) h[n] = 0.f;
      }
    }
  };

  const float dsk = (kRead && (p.flags & kHasD)) ? p.Dskip[d] : 0.f;

  // first captured token at or after t0: the smallest t >= t0 with
  // (t + 1) mod every == 0; slot = its index in the thinned trajectory
  int64_t cd = 0, slot = 0;
  if constexpr (TRAJ != 0) {
    const int64_t ev = p.traj_every;
    const int64_t first = (t0 + ev) / ev * ev - 1;
    cd = first - t0;
    slot = (first + 1) / ev - 1;
  }

  // Descriptors over this chunk's rows of x, dt, z, y ([nsteps, D]) and
  // B, C ([nsteps, N]); lane offsets in bytes.
  using SI = Stream<TIn>;
  using SO = Stream<TOut>;
  const int64_t row0 = static_cast<int64_t>(b) * p.L + t0;  // token index of t0
  const uint32_t in_row = static_cast<uint32_t>(D * sizeof(TIn));   // bytes per token
  const uint32_t out_row = static_cast<uint32_t>(D * sizeof(TOut));
  const uint32_t bc_row = static_cast<uint32_t>(N * sizeof(TIn));
  const uint32_t ns = static_cast<uint32_t>(nsteps > 0 ? nsteps : 1);
  const auto rx = make_rsrc(xg + row0 * D, ns * in_row);
  const auto rd = make_rsrc(dtg + row0 * D, ns * in_row);
  const auto rz = make_rsrc(zg + row0 * D, ns * in_row);
  const auto rb = make_rsrc(Bg + row0 * N, ns * bc_row);
  const auto rc = make_rsrc(Cg + row0 * N, ns * bc_row);
  const auto ry = make_rsrc(yg + row0 * D, ns * out_row);
  const uint32_t dl = static_cast<uint32_t>(d) * sizeof(TIn);
  // y is written once per channel, by the lanes of group 0.
  const uint32_t dly = (live && grp == 0) ? static_cast<uint32_t>(d) * sizeof(TOut) : kDropOffset;
  const int lane16 = lane & 15;
  const uint32_t el =
      static_cast<uint32_t>(16 * grp + (lane16 < NL ? lane16 : NL - 1)) * sizeof(TIn);

  // With 16 states per lane, B_t / C_t of a tile are written (as fp32) to a
  // wave-private LDS slice when the tile is consumed, by the lanes that
  // loaded them, and each token reads its 16 (+16) coefficients back with
  // same-address (broadcast) 16-byte reads into VGPRs, so the state update
  // and the readout use plain VALU operands instead of DPP broadcasts.  The
  // slice is private to the wave: no barrier.
  // Used where it was measured to pay: with a readout (32 broadcasts per
  // token replaced), when a channel spans several lanes (N > 16), and for
  // readout-free N = 16 scans over 16-bit inputs in 4-token tiles, whose
  // staging is one dword per lane (the long-context summary pass: 2.67 ->
  // 2.64 ms); with per-token staging a readout-free N = 16 scan saves only
  // the 16 B broadcasts, less than the staging costs.
  constexpr bool kLds = NL == 16 && (kRead || P > 1 || (sizeof(typename SI::raw) == 2 && kPF == 4));
  // 16-bit coefficients with N = 16 in one lane: a 4-token tile's B (and C)
  // rows are 4 x 16 x 2 bytes = 32 dwords, so lanes 0..31 fetch one dword
  // each (token l / 8, coefficients 2 (l mod 8) and 2 (l mod 8) + 1): one
  // load per array and tile instead of one per token, and two 16-bit LDS
  // writes (low half, high half) per lane (2.5% on the corpus encode,
  // 3.5% on the query prefill).
  constexpr bool kBcWord = kLds && P == 1 && sizeof(typename SI::raw) == 2 && kPF == 4;

  // Software pipeline over tiles of kPF tokens with two register buffers:
  // while tile i is computed from one buffer, tile i + 1 streams into the
  // other.  Each buffer keeps fixed registers (no rotation), and a buffer is
  // refilled only after its tile has been consumed.  Tiles past the chunk
  // reread its last token (in bounds, never used), so loads need no guards;
  // the coefficient dwords of tokens past the chunk lie past the
  // descriptor's range and read as zero (never used either).
  struct Tile {
    typename SI::raw x[kPF], dt[kPF], z[kPF], b[kPF][G], c[kPF][G];
    uint32_t bw, cw;  // kBcWord: this lane's dword of the tile's B / C rows
  };
  Tile t0b, t1b;

  __shared__ __attribute__((aligned(16))) float bc_lds[kLds ? kSBlock / 64 : 1][kLds ? kPF : 1][2][kLds ? N : 1];
  // bf16 coefficients go in as raw bits into the high half of a word whose
  // low half is zero (cleared once, below): the word is then the exact fp32
  // value with no conversion instruction.  Written as bytes, so the
  // compiler keeps their order with the float reads of the tile.
  constexpr bool kRawHigh = sizeof(typename SI::raw) == 2;
  auto put = [&](float* dst, typename SI::raw v) {
    if constexpr (kRawHigh) {
      __builtin_memcpy(reinterpret_cast<char*>(dst) + 2, &v, 2);
    } else {
      *dst = SI::f32(v);
    }
  };
  if constexpr (kLds && kRawHigh) {
    float* slice = &bc_lds[wave][0][0][0];
#pragma unroll
    for (int i = lane; i < kPF * 2 * N; i += 64) slice[i] = 0.f;
  }
  auto stage = [&](const Tile& tb) {
    if constexpr (kBcWord) {
      if (lane < 32) {
        // the dword's low half is coefficient j, its high half j + 1
        const int k = lane >> 3;
        const int j = 2 * (lane & 7);
        const uint16_t b0 = static_cast<uint16_t>(tb.bw), b1 = static_cast<uint16_t>(tb.bw >> 16);
        put(&bc_lds[wave][k][0][j], b0);
        put(&bc_lds[wave][k][0][j + 1], b1);
        if constexpr (kRead) {
          const uint16_t c0 = static_cast<uint16_t>(tb.cw), c1 = static_cast<uint16_t>(tb.cw >> 16);
          put(&bc_lds[wave][k][1][j], c0);
          put(&bc_lds[wave][k][1][j + 1], c1);
        }
      }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the writes are done before any read
    } else if constexpr (kLds) {
      if ((lane >> 4) < P) {
#pragma unroll
        for (int k = 0; k < kPF; ++k) {
          put(&bc_lds[wave][k][0][16 * grp + lane16], tb.b[k][0]);
          if constexpr (kRead) put(&bc_lds[wave][k][1][16 * grp + lane16], tb.c[k][0]);
        }
      }
      // Wait until the writes have completed (lgkmcnt(0); vmcnt and expcnt
      // untouched) before any lane reads the tile: without this explicit
      // wait, tail tiles were computed with stale coefficients.
      __builtin_amdgcn_s_waitcnt(0xc07f);
    }
  };
  const int last = nsteps > 0 ? nsteps - 1 : 0;
  // lane offset of the coefficient dwords (lanes past 31 fetch nothing)
  const uint32_t bcw_off =
      lane < 32 ? static_cast<uint32_t>(lane >> 3) * bc_row + 4u * static_cast<uint32_t>(lane & 7)
                : kDropOffset;
  auto fetch = [&](Tile& tb, int tile) {
    if constexpr (kBcWord) {
      const uint32_t sb = static_cast<uint32_t>(tile * kPF) * bc_row;
      tb.bw = __builtin_amdgcn_raw_buffer_load_b32(rb, bcw_off, sb, 0);
      if constexpr (kRead) tb.cw = __builtin_amdgcn_raw_buffer_load_b32(rc, bcw_off, sb, 0);
    }
#pragma unroll
    for (int k = 0; k < kPF; ++k) {
      int st = tile * kPF + k;
      st = st < last ? st : last;
      const uint32_t so = static_cast<uint32_t>(st) * in_row;
      tb.x[k] = SI::load(rx, dl, so);
      tb.dt[k] = SI::load(rd, dl, so);
      if constexpr (HASZ) tb.z[k] = SI::load(rz, dl, so);
      if constexpr (!kBcWord) {
        const uint32_t sb = static_cast<uint32_t>(st) * bc_row;
#pragma unroll
        for (int j = 0; j < G; ++j) {
          tb.b[k][j] = SI::load(rb, el + 16 * j * sizeof(TIn), sb);
          if constexpr (kRead) tb.c[k][j] = SI::load(rc, el + 16 * j * sizeof(TIn), sb);
        }
      }
    }
  };

  // coefficients of the current token, read from the staged tile
  struct Coef {
    float b[16], c[16];
  };
  // Read as float, the type the values were stored with, so the compiler
  // sees the reads and the staging writes as possibly aliasing and keeps
  // their order (a vector-typed read could be reordered across the writes
  // of the next tile); consecutive aligned reads still merge into
  // ds_read_b128.
  auto read_coef = [&](Coef& cd, int k) {
    if constexpr (kLds) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        cd.b[j] = bc_lds[wave][k][0][16 * grp + j];
        cd.c[j] = kRead ? bc_lds[wave][k][1][16 * grp + j] : 0.f;
      }
    }
  };

  // fp16 trajectory with 16 states per lane: the wave's 64 state rows
  // (2 KB, contiguous in traj) go out as two stores that are each contiguous
  // across the wave, transposed through a wave-private LDS slice: lane l
  // writes its 32 bytes at 32 l, then reads the 16 bytes at 16 l and at
  // 1024 + 16 l, which hold half l mod 2 of channels l / 2 and 32 + l / 2
  // (each store instruction then fills whole lines).  Its own
  // instantiation (TRAJ == 2), launched where the stores bound the kernel:
  // every = 1 0.659 -> 0.500 ms, every = 2 0.350 -> 0.308 ms, but every = 4
  // 0.200 -> 0.249 ms (SMC workload).
  constexpr bool kTrajT = TRAJ == 2 && P == 1 && NL == 16 && std::is_same<TSt, f16_t>::value;
  __shared__ __attribute__((aligned(16))) st_half8 traj_lds[kTrajT ? kSBlock / 64 : 1][kTrajT ? 128 : 1];
  const int nlive = static_cast<int>(D - wave_d0 < 64 ? D - wave_d0 : 64);  // live channels of the wave
  float dtacc = 0.f;
  auto step = [&](const Tile& tb, int k, int st) {
    const float xv = SI::f32(tb.x[k]);
    const float dtv = SI::f32(tb.dt[k]);
    const float u = dtv * xv;
    float acc = 0.f;
    if constexpr (kLds) {
      Coef cf;
      read_coef(cf, k);
      token_vgpr<NL, kRead>(h, a2, dtv, u, cf.b, cf.c, acc, std::make_integer_sequence<int, 16>{});
    } else {
      float cv[G];
#pragma unroll
      for (int j = 0; j < G; ++j) cv[j] = kRead ? SI::f32(tb.c[k][j]) : 0.f;
      float bv[G];
#pragma unroll
      for (int j = 0; j < G; ++j) bv[j] = SI::f32(tb.b[k][j]);
      token<NL, kRead>(h, a2, dtv, u, bv, cv, acc, std::make_integer_sequence<int, G>{});
    }
    if constexpr (kRead) {
      // sum the P groups' partial readouts (lanes 16 and 32 apart)
      if constexpr (P >= 2) acc += lane_xor(acc, 16);
      if constexpr (P >= 4) acc += lane_xor(acc, 32);
      float out = fmaf(dsk, xv, acc);
      if constexpr (HASZ) {
        const float zv = SI::f32(tb.z[k]);
        const float e = __builtin_amdgcn_exp2f(-kLog2e * zv);
        out *= zv * __builtin_amdgcn_rcpf(1.f + e);
      }
      SO::store(ry, dly, static_cast<uint32_t>(st) * out_row, out);
    }
    if constexpr (KIND == kSummary) dtacc += dtv;
    if constexpr (TRAJ != 0) {
      if (cd == 0) {  // wave-uniform
        TSt* row = static_cast<TSt*>(p.traj) + (static_cast<int64_t>(b) * p.traj_count + slot) * D * N;
        if constexpr (kTrajT) {
          const st_float8 v0 = {h[0], h[1], h[2], h[3], h[4], h[5], h[6], h[7]};
          const st_float8 v1 = {h[8], h[9], h[10], h[11], h[12], h[13], h[14], h[15]};
          traj_lds[wave][2 * lane] = __builtin_convertvector(v0, st_half8);
          traj_lds[wave][2 * lane + 1] = __builtin_convertvector(v1, st_half8);
          const st_half8 o0 = traj_lds[wave][lane];
          const st_half8 o1 = traj_lds[wave][64 + lane];
          TSt* wrow = row + wave_d0 * N;
          if ((lane >> 1) < nlive) *reinterpret_cast<st_half8*>(wrow + 8 * lane) = o0;
          if (32 + (lane >> 1) < nlive) *reinterpret_cast<st_half8*>(wrow + 512 + 8 * lane) = o1;
        } else if (live) {
          store_state_vec<NL>(row + sofs, h);
        }
        ++slot;
        cd = p.traj_every - 1;
      } else {
        --cd;
      }
    }
  };
  // The balance step runs at the head of each iteration of the time loop
  // (every 2 tiles), which is a block boundary anyway, so the unrolled body
  // stays one straight-line block whether or not the launch balances.
  auto run_tile = [&](const Tile& tb, int tile) {
    stage(tb);
#pragma unroll
    for (int k = 0; k < kPF; ++k) step(tb, k, tile * kPF + k);
  };
  auto run_tile_guarded = [&](const Tile& tb, int tile) {
    stage(tb);
#pragma unroll
    for (int k = 0; k < kPF; ++k)
      if (tile * kPF + k < nsteps) step(tb, k, tile * kPF + k);
  };

  if constexpr (DEC) {
    // Wave 0 decides while the others wait; then every wave requests its
    // first tile and its start state.  (Requesting the other waves' first
    // tiles, and speculatively the store row of the key with the largest
    // screen score, during the decision was measured to gain nothing: those
    // loads slowed the decision's own round trips as much as they saved.)
    __shared__ DecideShared dsh;
    __shared__ int32_t dec_row;
    if (wave == 0) {
      const int32_t r = decide_query<6>(*rp, b, dsh);
      if (lane == 0) dec_row = r;
    }
    __syncthreads();
    row_known = dec_row;
    if (nsteps > 0) fetch(t0b, 0);
    init_state();
  } else {
    if (nsteps > 0) fetch(t0b, 0);
    init_state();
  }
  if (nsteps > 0) {
    // Tile 0 completes before tile 1 is requested (vmcnt(0); lgkmcnt and
    // expcnt untouched): at launch every wave requests at once, and tile 0
    // then does not queue behind tile 1 (corpus encode 1.2445 -> 1.2297 ms).
    __builtin_amdgcn_s_waitcnt(0x0F70);
    int tile = 0;
    // Pairs of whole tiles: straight-line code, no per-token guards.
    for (; (tile + 2) * kPF <= nsteps; tile += 2) {
      if (fair) balance_step(progress, wave, tile);
      fetch(t1b, tile + 1);
      run_tile(t0b, tile);
      fetch(t0b, tile + 2);
      run_tile(t1b, tile + 1);
    }
    // Fewer than 2 kPF tokens remain: tile `tile` is in t0b.
    fetch(t1b, tile + 1);
    run_tile_guarded(t0b, tile);
    run_tile_guarded(t1b, tile + 1);
  }

  if (!live) return;
  if constexpr (KIND == kSummary) {
    store_state<NL>(p.carry + (static_cast<int64_t>(b) * p.nchunks + c + 1) * D * N + sofs, h);
    if (grp == 0) p.dtsum[(static_cast<int64_t>(b) * p.nchunks + c) * D + d] = dtacc;
  } else {
    if ((p.flags & kHasHT) && c == p.nchunks - 1)
      store_state<NL>(static_cast<TSt*>(p.hT) + b * p.hT_stride + sofs, h);
  }
}

// The readout-free kinds over 16-bit inputs with N = 16 (the chunked scan's
// summary pass, state-only encodes) are built for at most 128 VGPRs: four
// waves per SIMD, two 512-thread workgroups per CU.  Left to itself the
// compiler gave them 135-138, one workgroup per CU (two waves per SIMD) in
// the many-round launches of the summary pass; at 128 it keeps a few values
// that live across the time loop in scratch, none inside it.  Every other
// instantiation keeps the compiler's own allocation.
template <int N, typename TIn, int KIND, int TRAJ>
constexpr int kScanMinWaves = (KIND != kReadout && TRAJ == 0 && N == 16 && sizeof(TIn) == 2) ? 4 : 1;

template <int N, typename TIn, typename TOut, typename TSt, int KIND, bool HASZ, int TRAJ>
__global__ __launch_bounds__(kSBlock)
__attribute__((amdgpu_waves_per_eu(kScanMinWaves<N, TIn, KIND, TRAJ>))) void scan_kernel(
    const TIn* __restrict__ xg, const TIn* __restrict__ dtg, const TIn* __restrict__ zg,
    const TIn* __restrict__ Bg, const TIn* __restrict__ Cg, TOut* __restrict__ yg,
    const ScanParams p) {
  scan_body<N, TIn, TOut, TSt, KIND, HASZ, TRAJ, false>(xg, dtg, zg, Bg, Cg, yg, p, nullptr);
}

// The query-time prefill with its decision (DEC above).  At most 128 VGPRs
// (four waves per SIMD, as the plain prefill), so that a 4096-wave prefill
// still runs in one round; the decision's registers fit in that budget.
template <int N, typename TIn, typename TOut, typename TSt, int KIND, bool HASZ>
__global__ __launch_bounds__(kSBlock) __attribute__((amdgpu_waves_per_eu(4))) void query_scan_kernel(
    const TIn* __restrict__ xg, const TIn* __restrict__ dtg, const TIn* __restrict__ zg,
    const TIn* __restrict__ Bg, const TIn* __restrict__ Cg, TOut* __restrict__ yg,
    const ScanParams p, const RetrieveParams rp) {
  scan_body<N, TIn, TOut, TSt, KIND, HASZ, 0, true>(xg, dtg, zg, Bg, Cg, yg, p, &rp);
}

// Pass 2: per (b, d, n) lane, fold the chunk summaries in time order.
// carry[b, 0] = h0; carry[b, c] = exp2(A' S_{c-1}) carry[b, c-1] + s_{c-1},
// where pass 1 left s_{c-1} in carry[b, c] and S_{c-1} in dtsum[b, c-1].
template <typename TSt>
__global__ __launch_bounds__(256) void carry_kernel(const ScanParams p, int N) {
  const int64_t DN = p.D * N;
  const int64_t gid = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (gid >= p.B * DN) return;
  const int64_t b = gid / DN;
  const int64_t dn = gid - b * DN;
  const int64_t d = dn / N;
  const float a2 = -kLog2e * p.A[dn];
  float H = 0.f;
  if (p.h0_score != nullptr) {
    float hv[1];
    compose_state<1, TSt>(hv, p, b, dn);
    H = hv[0];
  } else if (p.flags & kHasH0) {
    const TSt* src = h0_row<TSt>(p, b);
    H = src != nullptr ? to_f32(src[dn]) : __builtin_nanf("");
  }
  float* cp = p.carry + b * p.nchunks * DN + dn;
  const float* sp = p.dtsum + b * p.nchunks * p.D + d;
  cp[0] = H;
  constexpr int kU = 8;
  for (int c0 = 1; c0 < p.nchunks; c0 += kU) {
    float sv[kU], Sv[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      if (c0 + k < p.nchunks) {
        sv[k] = cp[(c0 + k) * DN];
        Sv[k] = sp[(c0 + k - 1) * p.D];
      }
    }
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      if (c0 + k < p.nchunks) {
        H = fmaf(__builtin_amdgcn_exp2f(a2 * Sv[k]), H, sv[k]);
        cp[(c0 + k) * DN] = H;
      }
    }
  }
}

// Pass 2 for short sequences over few channels, where the fold's length
// and not its bytes is the cost: one wave per (b, d, n), lane j holding the
// step of chunk j, H -> m_j H + s_j with m_j = exp2(A' S_j), and an
// inclusive scan of the steps over the lanes (composition (m, s) after
// (m', s') = (m m', m s' + s); row shifts by 1, 2, 4, 8, then lane 15 of
// rows 0 and 2 into rows 1 and 3, then lane 31 into rows 2 and 3), so every
// carry needs one round trip instead of one per batch of chunks.  The same
// carries as carry_kernel up to fp32 reassociation.
constexpr int kCarryScanMaxChunks = 64;
constexpr int64_t kCarryScanMaxLanes = 8192;  // (b, d, n) lanes: waves of strided loads

template <int CTRL, int ROWS>
__device__ __forceinline__ void affine_step(float& m, float& s) {
  // lanes without a source keep the identity step (1, 0)
  const float mo = __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, 1.f), __builtin_bit_cast(int, m), CTRL,
                                         ROWS, 0xf, false));
  const float so = __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, 0.f), __builtin_bit_cast(int, s), CTRL,
                                         ROWS, 0xf, false));
  s = fmaf(m, so, s);
  m = m * mo;
}

template <typename TSt>
__global__ __launch_bounds__(256) void carry_scan_kernel(const ScanParams p, int N) {
  const int64_t DN = p.D * N;
  const int64_t w = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) >> 6;
  if (w >= p.B * DN) return;  // whole waves
  const int lane = threadIdx.x & 63;
  const int64_t b = w / DN;
  const int64_t dn = w - b * DN;
  const int64_t d = dn / N;
  const float a2 = -kLog2e * p.A[dn];
  float H = 0.f;
  if (p.h0_score != nullptr) {
    float hv[1];
    compose_state<1, TSt>(hv, p, b, dn);
    H = hv[0];
  } else if (p.flags & kHasH0) {
    const TSt* src = h0_row<TSt>(p, b);
    H = src != nullptr ? to_f32(src[dn]) : __builtin_nanf("");
  }
  float* cp = p.carry + b * p.nchunks * DN + dn;
  const float* sp = p.dtsum + b * p.nchunks * p.D + d;
  const bool on = lane < p.nchunks - 1;
  float m = 1.f, s = 0.f;
  if (on) {
    s = cp[static_cast<int64_t>(lane + 1) * DN];
    m = __builtin_amdgcn_exp2f(a2 * sp[static_cast<int64_t>(lane) * p.D]);
  }
  affine_step<0x111, 0xf>(m, s);  // row_shr:1
  affine_step<0x112, 0xf>(m, s);  // row_shr:2
  affine_step<0x114, 0xf>(m, s);  // row_shr:4
  affine_step<0x118, 0xf>(m, s);  // row_shr:8
  affine_step<0x142, 0xa>(m, s);  // row_bcast:15
  affine_step<0x143, 0xc>(m, s);  // row_bcast:31
  if (on) cp[static_cast<int64_t>(lane + 1) * DN] = fmaf(m, H, s);
  if (lane == 0) cp[0] = H;
}

// The final pass: readout (with or without gate) or state-only, with the
// trajectory mode TRAJ (0 none, 1 direct stores, 2 stores transposed
// through LDS).
template <int N, typename TIn, typename TOut, typename TSt, int TRAJ>
hipError_t launch_final(const ScanParams& p, int64_t g3, hipStream_t s) {
  const TIn* X = static_cast<const TIn*>(p.x);
  const TIn* DT = static_cast<const TIn*>(p.dt);
  const TIn* Z = static_cast<const TIn*>(p.z);
  const TIn* BB = static_cast<const TIn*>(p.Bm);
  const TIn* CC = static_cast<const TIn*>(p.Cm);
  if (p.y != nullptr && (p.flags & kHasZ))
    hipLaunchKernelGGL((scan_kernel<N, TIn, TOut, TSt, kReadout, true, TRAJ>), dim3(static_cast<unsigned>(g3)),
                       dim3(kSBlock), 0, s, X, DT, Z, BB, CC, static_cast<TOut*>(p.y), p);
  else if (p.y != nullptr)
    hipLaunchKernelGGL((scan_kernel<N, TIn, TOut, TSt, kReadout, false, TRAJ>), dim3(static_cast<unsigned>(g3)),
                       dim3(kSBlock), 0, s, X, DT, Z, BB, CC, static_cast<TOut*>(p.y), p);
  else
    hipLaunchKernelGGL((scan_kernel<N, TIn, float, TSt, kStateOnly, false, TRAJ>), dim3(static_cast<unsigned>(g3)),
                       dim3(kSBlock), 0, s, X, DT, Z, BB, CC, static_cast<float*>(nullptr), p);
  return hipGetLastError();
}

template <int N, typename TIn, typename TOut, typename TSt, bool TRAJ>
hipError_t launch_typed(const ScanParams& p, hipStream_t s) {
  const int64_t rows_blocks = static_cast<int64_t>(p.dblocks) * p.B;
  if (p.nchunks > 1) {
    const int64_t g1 = rows_blocks * (p.nchunks - 1);
    hipLaunchKernelGGL((scan_kernel<N, TIn, float, float, kSummary, false, 0>), dim3(static_cast<unsigned>(g1)),
                       dim3(kSBlock), 0, s, static_cast<const TIn*>(p.x), static_cast<const TIn*>(p.dt),
                       static_cast<const TIn*>(p.z), static_cast<const TIn*>(p.Bm),
                       static_cast<const TIn*>(p.Cm), static_cast<float*>(nullptr), p);
    const int64_t lanes = p.B * p.D * N;
    if (p.nchunks > 8 && p.nchunks <= kCarryScanMaxChunks && lanes <= kCarryScanMaxLanes)
      hipLaunchKernelGGL((carry_scan_kernel<TSt>), dim3(static_cast<unsigned>((lanes * 64 + 255) / 256)),
                         dim3(256), 0, s, p, N);
    else
      hipLaunchKernelGGL((carry_kernel<TSt>), dim3(static_cast<unsigned>((lanes + 255) / 256)), dim3(256),
                         0, s, p, N);
  }
  const int64_t g3 = rows_blocks * p.nchunks;
  if constexpr (!TRAJ) {
    return launch_final<N, TIn, TOut, TSt, 0>(p, g3, s);
  } else {
    // fp16 trajectories of 16 states per lane captured every token or every
    // other token: the store-bound case, transposed stores
    if constexpr (N == 16 && std::is_same<TSt, f16_t>::value) {
      if (p.traj_every <= 2) return launch_final<N, TIn, TOut, TSt, 2>(p, g3, s);
    }
    return launch_final<N, TIn, TOut, TSt, 1>(p, g3, s);
  }
}

template <int N, typename TIn, typename TOut, bool TRAJ>
hipError_t pick_state(const ScanParams& p, int state_dtype, hipStream_t s) {
  return state_dtype == 0 ? launch_typed<N, TIn, TOut, float, TRAJ>(p, s)
                          : launch_typed<N, TIn, TOut, f16_t, TRAJ>(p, s);
}

template <int N, typename TIn, bool TRAJ>
hipError_t pick_out(const ScanParams& p, int out_dtype, int state_dtype, hipStream_t s) {
  return out_dtype == 0 ? pick_state<N, TIn, float, TRAJ>(p, state_dtype, s)
                        : pick_state<N, TIn, bf16_t, TRAJ>(p, state_dtype, s);
}

template <int N, bool TRAJ>
hipError_t pick_in(const ScanParams& p, int in_dtype, int out_dtype, int state_dtype,
                   hipStream_t s) {
  return in_dtype == 0 ? pick_out<N, float, TRAJ>(p, out_dtype, state_dtype, s)
                       : pick_out<N, bf16_t, TRAJ>(p, out_dtype, state_dtype, s);
}

template <bool TRAJ>
hipError_t launch_scan_n(const ScanParams& p, int N, int in_dtype, int out_dtype, int state_dtype,
                         hipStream_t s) {
  switch (N) {
    case 1: return pick_in<1, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    case 2: return pick_in<2, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    case 4: return pick_in<4, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    case 8: return pick_in<8, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    case 16: return pick_in<16, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    case 32: return pick_in<32, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    case 64: return pick_in<64, TRAJ>(p, in_dtype, out_dtype, state_dtype, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace
}  // namespace precog
