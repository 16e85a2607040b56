// Structured Memory Consolidation on gfx950 (Sec. 5): two-stage cluster
// routing (Sec. 5.1, Eqs. smc-domain and smc-sub) and the semantic EMA
// (Sec. 5.3, Eq. smc-ema).
//
// Routing is exact: every score is the fp64 sum of the exact products of two
// fp32 values, summed in feature order (one fused multiply-add per term,
// which rounds exactly as multiply-then-add here), and the argmax keeps the
// lowest index among equal scores.  One wave per chunk embedding.  Each
// stage first orders its prototypes by lane-parallel fp64 sums with a proven
// error bound, which decides the argmax unless two scores lie within the
// bound of each other; then lane m scores prototype m sequentially, the sum
// of the definition itself.  The work is a few thousand fused multiply-adds
// per chunk, so the kernel is latency-bound by design.
//
// Consolidation applies s <- (1 - alpha) s + alpha h to the routed semantic
// state for every chunk in chunk order; rows and element slices run in
// parallel, the chunks of one row in order within one lane.
#include <type_traits>

#include "precog_kernels.h"
#include "wave_ops.h"

namespace precog {
namespace {

constexpr int kMaxE = 4096;
constexpr int kRowFloats = 8192;  // LDS floats for staged prototype rows

__device__ __forceinline__ double shfl_d(double v, int src_lane) {
  const int lo = __builtin_amdgcn_ds_bpermute(src_lane * 4, static_cast<int>(__double2loint(v)));
  const int hi = __builtin_amdgcn_ds_bpermute(src_lane * 4, static_cast<int>(__double2hiint(v)));
  return __hiloint2double(hi, lo);
}

// fp64 dot product of the embedding in LDS with one prototype row, in
// feature order.
__device__ __forceinline__ double exact_dot(const float4* e4, const float* row, int E) {
  const float4* r4 = reinterpret_cast<const float4*>(row);
  double s = 0.0;
  for (int i = 0; i < E / 4; ++i) {
    const float4 a = e4[i];
    const float4 b = r4[i];
    s = fma(static_cast<double>(a.x), static_cast<double>(b.x), s);
    s = fma(static_cast<double>(a.y), static_cast<double>(b.y), s);
    s = fma(static_cast<double>(a.z), static_cast<double>(b.z), s);
    s = fma(static_cast<double>(a.w), static_cast<double>(b.w), s);
  }
  return s;
}

// Lane holding the best (score, lowest index) among lanes < n.
__device__ __forceinline__ int wave_argmax(double s, int lane, int n) {
  double bs = lane < n ? s : -INFINITY;
  int bi = lane < n ? lane : 0x7fffffff;
  bool any = lane < n;
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const double os = shfl_d(bs, lane ^ m);
    const int oi = __builtin_amdgcn_ds_bpermute((lane ^ m) * 4, bi);
    const bool oany = __builtin_amdgcn_ds_bpermute((lane ^ m) * 4, static_cast<int>(any)) != 0;
    if (oany && (!any || os > bs || (os == bs && oi < bi))) {
      bs = os;
      bi = oi;
      any = true;
    }
  }
  return bi;
}

// One routing stage over the n prototype rows at `rows` (row stride E),
// decided without the sequential sums when that is provably safe: the index
// of the best (score, lowest index), or -1.  Each row's score is summed
// lane-parallel in fp64 (every product exact; lane l sums features l, l + 64,
// ... in order, then the 6-level wave tree), which differs from the exact
// real sum by at most gamma_{E/64+7} T, T = sum_e |x_e w_e| (summed the same
// way; the factor 1.01 covers its rounding); the sequential sum of the
// definition differs from the exact sum by at most gamma_E T.  If the best
// row's lower end beats every other row's upper end, that row is also the
// sequential argmax.  Otherwise (near or exact ties, NaN or infinite
// values) the caller scores the stage sequentially.  Rows are staged through
// LDS a batch at a time (fixed-width groups of predicated 16-byte loads, so
// a batch's loads are in flight together).
__device__ int fast_stage(const float* ex, float* rs, const float* rows, int n, int E, int lane) {
  const double u53 = 1.1102230246251565e-16;  // 2^-53
  const double dp = static_cast<double>(E / 64 + 7);
  const double en = static_cast<double>(E);
  const double gs = 1.01 * (dp * u53 / (1.0 - dp * u53) + en * u53 / (1.0 - en * u53));
  const int per = kRowFloats / E < 8 ? kRowFloats / E : 8;
  double best = 0.0, best_mu = 0.0, others = -INFINITY;
  int bi = -1;
  bool bad = false;
  for (int m0 = 0; m0 < n; m0 += per) {
    const int nb = n - m0 < per ? n - m0 : per;
    const int tot = nb * (E / 4);
    const float4* src = reinterpret_cast<const float4*>(rows + static_cast<int64_t>(m0) * E);
    __syncthreads();  // the previous batch is consumed
    for (int f0 = 0; f0 < tot; f0 += 8 * 64) {
      float4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int f = f0 + 64 * u + lane;
        v[u] = f < tot ? src[f] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int f = f0 + 64 * u + lane;
        if (f < tot) reinterpret_cast<float4*>(rs)[f] = v[u];
      }
    }
    __syncthreads();
    for (int r = 0; r < nb; ++r) {
      double part = 0.0, apart = 0.0;
      for (int e = lane; e < E; e += 64) {
        const double pr = static_cast<double>(ex[e]) * static_cast<double>(rs[r * E + e]);
        part += pr;
        apart += fabs(pr);
      }
      const double a = wave_sum_d(part);
      const double mu = gs * wave_sum_d(apart) + 1e-300;
      if (!(a == a) || !(mu < INFINITY)) bad = true;
      if (bi < 0 || a > best) {
        if (bi >= 0) others = fmax(others, best + best_mu);
        best = a;
        best_mu = mu;
        bi = m0 + r;
      } else {
        others = fmax(others, a + mu);
      }
    }
  }
  return !bad && best - best_mu > others ? bi : -1;
}

__global__ __launch_bounds__(64) void route_kernel(const RouteParams p) {
  const int64_t c = blockIdx.x;
  const int lane = threadIdx.x;
  const int E = static_cast<int>(p.E);
  __shared__ float4 e4[kMaxE / 4];
  const float4* src = reinterpret_cast<const float4*>(p.emb + c * p.E);
  for (int i = lane; i < E / 4; i += 64) e4[i] = src[i];
  __syncthreads();
  __shared__ float rs[kRowFloats];
  const float* ex = reinterpret_cast<const float*>(e4);
  // stage 1: domain m* = argmax_m <phi(c), p_m>; lane m scores prototype m
  // sequentially when the fast ordering cannot decide
  int m = fast_stage(ex, rs, p.dom, p.ndom, E, lane);
  if (m < 0) {
    double s = 0.0;
    if (lane < p.ndom) s = exact_dot(e4, p.dom + static_cast<int64_t>(lane) * p.E, E);
    m = wave_argmax(s, lane, p.ndom);
  }
  // stage 2: sub-cluster j* = argmax_j <phi(c), q_{m*, j}>
  const float* subs = p.sub + static_cast<int64_t>(m) * p.nsub * p.E;
  int j = fast_stage(ex, rs, subs, p.nsub, E, lane);
  if (j < 0) {
    double s = 0.0;
    if (lane < p.nsub) s = exact_dot(e4, subs + static_cast<int64_t>(lane) * p.E, E);
    j = wave_argmax(s, lane, p.nsub);
  }
  if (lane == 0) {
    p.dom_out[c] = m;
    p.sub_out[c] = j;
    if (p.flat_out) p.flat_out[c] = m * p.nsub + j;
  }
}

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float8 __attribute__((ext_vector_type(8)));

template <typename T> struct V8;
template <> struct V8<float> {
  static __device__ __forceinline__ float8 load(const void* b, int64_t i) {
    return *reinterpret_cast<const float8*>(static_cast<const float*>(b) + i);
  }
  static __device__ __forceinline__ void store(void* b, int64_t i, float8 v) {
    *reinterpret_cast<float8*>(static_cast<float*>(b) + i) = v;
  }
};
template <> struct V8<f16_t> {
  static __device__ __forceinline__ float8 load(const void* b, int64_t i) {
    return __builtin_convertvector(*reinterpret_cast<const half8*>(static_cast<const _Float16*>(b) + i),
                                   float8);
  }
  static __device__ __forceinline__ void store(void* b, int64_t i, float8 v) {
    *reinterpret_cast<half8*>(static_cast<_Float16*>(b) + i) = __builtin_convertvector(v, half8);
  }
};

// Workgroup (slice, r): state row r, elements [2048 slice, 2048 slice + 2048).
// The row slice is loaded once, every chunk routed to r is applied in chunk
// order in registers, and the slice is stored once, so states are read and
// written once and each contribution is read once.  The targets are read 64
// at a time, one per lane (in flight with the state row), and a ballot gives
// the chunks routed to r in order; their contributions are loaded
// kEmaBatch at a time before the batch is applied in chunk order.  Each
// update is s' = fma(alpha, h, (1 - alpha) s) in fp32 with both factors
// rounded once from fp64 (alpha = 1 gives s' = h exactly); fp16 states are
// rounded to nearest even after every update, as an fp16 store would be.
constexpr int kEmaBatch = 4;

template <typename TS, typename TH>
__global__ __launch_bounds__(256) void ema_kernel(const EmaParams p) {
  const int64_t r = blockIdx.y;
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  // whole waves past the row end leave; lanes past it stay for the ballots
  if (e - static_cast<int64_t>(threadIdx.x & 63) * 8 >= p.S) return;
  const bool live = e < p.S;
  const int lane = static_cast<int>(threadIdx.x & 63);
  const float a = p.alpha;
  const float b = p.one_minus_alpha;
  const int64_t so = r * p.S + e;
  float8 s = {};
  if (live) s = V8<TS>::load(p.states, so);
  bool touched = false;
  for (int64_t c0 = 0; c0 < p.C; c0 += 64) {
    const int64_t ci = c0 + lane;
    uint64_t m = __ballot(ci < p.C && p.target[ci] == r);
    while (m) {
      int64_t cb[kEmaBatch];
#pragma unroll
      for (int j = 0; j < kEmaBatch; ++j) {
        cb[j] = m ? c0 + __builtin_ctzll(m) : -1;
        m &= m - 1;
      }
      float8 h[kEmaBatch];
#pragma unroll
      for (int j = 0; j < kEmaBatch; ++j)
        if (cb[j] >= 0 && live) h[j] = V8<TH>::load(p.contrib, cb[j] * p.S + e);
#pragma unroll
      for (int j = 0; j < kEmaBatch; ++j) {
        if (cb[j] < 0) break;
#pragma unroll
        for (int k = 0; k < 8; ++k) s[k] = fmaf(a, h[j][k], b * s[k]);
        if constexpr (std::is_same<TS, f16_t>::value)
          s = __builtin_convertvector(__builtin_convertvector(s, half8), float8);
      }
      touched = true;
    }
  }
  if (touched && live) V8<TS>::store(p.states, so, s);
}

}  // namespace

hipError_t launch_route(const RouteParams& p, hipStream_t s) {
  hipLaunchKernelGGL(route_kernel, dim3(static_cast<unsigned>(p.C)), dim3(64), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_ema(const EmaParams& p, int state_dtype, int contrib_dtype, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>((p.S / 8 + 255) / 256), static_cast<unsigned>(p.R));
  if (state_dtype == 0 && contrib_dtype == 0)
    hipLaunchKernelGGL((ema_kernel<float, float>), grid, dim3(256), 0, s, p);
  else if (state_dtype == 0)
    hipLaunchKernelGGL((ema_kernel<float, f16_t>), grid, dim3(256), 0, s, p);
  else if (contrib_dtype == 0)
    hipLaunchKernelGGL((ema_kernel<f16_t, float>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((ema_kernel<f16_t, f16_t>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace precog
