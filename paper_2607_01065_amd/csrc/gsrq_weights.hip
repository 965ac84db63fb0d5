// Per-token weights of weighted GSKM on the GPU (arXiv 2607.01065, Sec. 5.3
// and Appendix B): w_i = ||g_i||_2, the norm of token i's gradient row, then
// the log smoothing w~_i = log(1 + lambda w_i) with lambda = tau /
// (median(w) + eps), eps = 1e-8.
//
// Three launches: a row-norm kernel (one wave per row, float64 sums, vector
// loads; HBM-bound), one workgroup that selects the median exactly by radix
// selection on the float bits (three 11-bit digit passes, histograms and,
// up to 32768 rows, the norms in LDS), and an element-wise transform over
// the whole grid.
#include "gsrq_common.h"

namespace {

constexpr int WN_THREADS = 256;     // row-norm kernel: one wave per row
constexpr int WS_THREADS = 1024;    // selection + transform: one workgroup
constexpr double LOGW_EPS = 1e-8;

template <typename T> struct NormVec;
template <> struct NormVec<_Float16> {
  static constexpr int E = 8;       // elements per 16-byte load
  static __device__ __forceinline__ double sq(const _Float16* p) {
    const h8 v = as_h8(*(const u4*)p);
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const double x = (double)(float)v[j];
      s = fma(x, x, s);
    }
    return s;
  }
};
template <> struct NormVec<float> {
  static constexpr int E = 4;
  static __device__ __forceinline__ double sq(const float* p) {
    const f4 v = *(const f4*)p;
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const double x = (double)v[j];
      s = fma(x, x, s);
    }
    return s;
  }
};

// ||g_i||_2 of every row: one wave per row, float64 sums of squares (exact
// products of the float16 / float32 elements), vector loads when the rows
// are 16-byte aligned.
template <typename T>
__global__ void __launch_bounds__(WN_THREADS) wnorm_kernel(const T* __restrict__ g, int64_t N,
                                                           int D, int64_t ldg, int vec,
                                                           float* __restrict__ norms) {
  constexpr int E = NormVec<T>::E;
  const int lane = threadIdx.x & 63;
  const int64_t step = (int64_t)gridDim.x * (WN_THREADS / 64);
  for (int64_t row = blockIdx.x * (int64_t)(WN_THREADS / 64) + (threadIdx.x >> 6); row < N;
       row += step) {
    const T* r = g + row * ldg;
    double s = 0.0;
    if (vec) {
#pragma unroll 4
      for (int j = lane * E; j < D; j += 64 * E) s += NormVec<T>::sq(r + j);
    } else {
      for (int j = lane; j < D; j += 64) {
        const double x = (double)(float)r[j];
        s = fma(x, x, s);
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if (lane == 0) norms[row] = (float)sqrt(s);
  }
}

constexpr int SEL_BITS = 11;                     // radix digit: 3 passes over 32 bits
constexpr int SEL_BINS = 1 << SEL_BITS;
constexpr int SEL_LDS_MAX = 32768;               // norms staged in LDS up to this N

// Exact median of the N norms (non-negative floats order like their bit
// patterns).  The (N-1)/2-th smallest value is found digit by digit, most
// significant first: a histogram of the digit over the values sharing the
// prefix found so far locates the bin holding the rank (bins searched in
// parallel from a block-wide prefix sum).  For even N the next value up is
// the same value if enough values tie with it, else the smallest larger
// value (one counting pass).  Writes {median, lambda} to stats.
__global__ void __launch_bounds__(WS_THREADS) wselect_kernel(const float* __restrict__ norms,
                                                             int64_t N, double tau,
                                                             double* __restrict__ stats) {
  extern __shared__ unsigned vals[];               // staged norm bits (N <= SEL_LDS_MAX)
  __shared__ unsigned hist[SEL_BINS];
  __shared__ unsigned wtot[WS_THREADS / 64];
  __shared__ unsigned sh_digit, sh_rank, sh_cnt, sh_min;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = (int)N;
  const bool staged = N <= SEL_LDS_MAX;
  if (staged)
    for (int i = tid; i < n; i += WS_THREADS) vals[i] = __float_as_uint(norms[i]);
  auto val = [&](int i) -> unsigned { return staged ? vals[i] : __float_as_uint(norms[i]); };
  const unsigned k = (unsigned)((N - 1) / 2);      // lower middle rank
  unsigned prefix = 0u, mask = 0u;
  // r: the rank still to find among the values sharing the prefix; every
  // thread holds it, and the one thread whose bin holds it publishes the
  // next digit and rank (read only after the pass's last barrier, and
  // written only after the next pass's third barrier)
  unsigned r = k;
  for (int shift = 32 - SEL_BITS; shift > -SEL_BITS; shift -= SEL_BITS) {
    const int sh = shift > 0 ? shift : 0;         // last digit: the low 32 - 2 * 11 bits
    const unsigned dmask = (shift > 0 ? (unsigned)SEL_BINS : (1u << (SEL_BITS + shift))) - 1u;
    for (int b = tid; b < SEL_BINS; b += WS_THREADS) hist[b] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += WS_THREADS) {
      const unsigned u = val(i);
      if ((u & mask) == prefix) atomicAdd(&hist[(u >> sh) & dmask], 1u);
    }
    __syncthreads();
    // block-wide exclusive prefix over the bins: thread t owns bins 2t, 2t+1
    const unsigned c0 = hist[2 * tid], c1 = hist[2 * tid + 1];
    unsigned inc = c0 + c1;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const unsigned v = __shfl_up(inc, off);
      if (lane >= off) inc += v;
    }
    if (lane == 63) wtot[wave] = inc;
    __syncthreads();
    unsigned base = inc - (c0 + c1);
    for (int w2 = 0; w2 < wave; ++w2) base += wtot[w2];
    if (r >= base && r < base + c0) { sh_digit = 2 * tid; sh_rank = r - base; }
    if (r >= base + c0 && r < base + c0 + c1) { sh_digit = 2 * tid + 1; sh_rank = r - base - c0; }
    __syncthreads();
    prefix |= sh_digit << sh;
    mask |= dmask << sh;
    r = sh_rank;
    __syncthreads();
  }
  const float lo = __uint_as_float(prefix);
  double med = (double)lo;
  if (!(N & 1)) {
    // upper middle rank k + 1: lo again if more than k + 1 values are <= lo
    if (tid == 0) { sh_cnt = 0u; sh_min = 0x7f800000u; }
    __syncthreads();
    unsigned cnt = 0u, mn = 0x7f800000u;
    for (int i = tid; i < n; i += WS_THREADS) {
      const unsigned u = val(i);
      if (u <= prefix) ++cnt;
      else mn = min(mn, u);
    }
    atomicAdd(&sh_cnt, cnt);
    atomicMin(&sh_min, mn);
    __syncthreads();
    const float hi = sh_cnt > k + 1 ? lo : __uint_as_float(sh_min);
    med = 0.5 * ((double)lo + (double)hi);
  }
  if (tid == 0) {
    stats[0] = med;
    stats[1] = tau / (med + LOGW_EPS);
  }
}

// w~_i = log(1 + lambda w_i), lambda from the selection kernel (float64).
__global__ void __launch_bounds__(256) wlog_kernel(const float* __restrict__ norms, int64_t N,
                                                   const double* __restrict__ stats,
                                                   float* __restrict__ w) {
  const double lambda = stats[1];
  for (int64_t i = blockIdx.x * (int64_t)256 + threadIdx.x; i < N; i += (int64_t)gridDim.x * 256)
    w[i] = (float)log1p(lambda * (double)norms[i]);
}

}  // namespace

extern "C" {

gsrq_status gsrq_row_weights(const void* grad, gsrq_dtype dtype, int64_t N, int32_t D,
                             int64_t ldg, float tau, float* norms, float* w, double* stats,
                             void* stream) {
  if (N < 1 || N > INT32_MAX || !norms || !w || !stats) return GSRQ_E_ARG;
  if (!(tau > 0.f) || !(tau < INFINITY)) return GSRQ_E_ARG;
  if (grad) {
    if (dtype != GSRQ_F32 && dtype != GSRQ_F16) return GSRQ_E_ARG;
    if (D < 1 || ldg < D) return GSRQ_E_ARG;
  }
  hipStream_t st = (hipStream_t)stream;
  if (grad) {
    const size_t esz = dtype == GSRQ_F16 ? 2 : 4;
    const int E = dtype == GSRQ_F16 ? 8 : 4;
    const int vec = ((uintptr_t)grad % 16 == 0) && ((ldg * esz) % 16 == 0) && (D % E == 0);
    const int grid = grid_for((N + WN_THREADS / 64 - 1) / (WN_THREADS / 64), 1);
    if (dtype == GSRQ_F16)
      wnorm_kernel<_Float16><<<grid, WN_THREADS, 0, st>>>((const _Float16*)grad, N, D, ldg, vec,
                                                          norms);
    else
      wnorm_kernel<float><<<grid, WN_THREADS, 0, st>>>((const float*)grad, N, D, ldg, vec, norms);
    gsrq_status e = launch_ok();
    if (e) return e;
  }
  const size_t lds = N <= SEL_LDS_MAX ? (size_t)N * sizeof(unsigned) : 0;
  if (lds > 65536 && hipFuncSetAttribute((const void*)wselect_kernel,
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds) != hipSuccess)
    return GSRQ_E_HIP;
  wselect_kernel<<<1, WS_THREADS, lds, st>>>(norms, N, (double)tau, stats);
  gsrq_status e = launch_ok();
  if (e) return e;
  wlog_kernel<<<grid_for(N, 256), 256, 0, st>>>(norms, N, stats, w);
  return launch_ok();
}

}  // extern "C"
