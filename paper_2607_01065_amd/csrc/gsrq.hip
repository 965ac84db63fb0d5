// GSRQ hot path for AMD MI355X (gfx950 / CDNA4): kernels and the C ABI.
//
// What is computed follows arXiv 2607.01065: gain-shape K-means (Sec. 5.2,
// eqs. 3-8, Algorithm 1) with per-row weights (Sec. 5.1, 5.3), product
// subspaces x residual stages (Sec. 3, Sec. 5.1), greedy residual encoding
// and gather-sum decoding.  How it is computed is specific to gfx950:
//
// Scoring (eq. 5) as an MFMA contraction.  For a subspace of dimension
// d <= 8 and one 16-codeword tile, one v_mfma_f32_16x16x32_f16 produces the
// squared distances ||r - g s||^2 = ||r||^2 + g^2 - 2 g s.r of 16 rows x 16
// codewords at once: the 32-long contraction carries the dot product in a
// hi/lo float16 split (a_hi b_hi + a_lo b_hi + a_hi b_lo, 22 significant
// bits per operand) plus the two bias terms g^2 and ||r||^2, each split hi/lo
// too.  Both operands are scaled by powers of two (sigma per codebook, rho
// per row) so every float16 is in range; the scaling multiplies all
// distances of a row by the same power of two and leaves the argmin exact.
// The argmin runs on packed integer keys: the low 6 bits of each float32
// distance are replaced by its (tile, slot) index and v_min3_i32 reduces two
// keys per instruction.  Rows whose key precision cannot separate a 1e-4
// relative top-2 margin are re-scored exactly in float64 (a rare fallback).
//
// Accumulation (eqs. 6-8): per-workgroup float64 LDS accumulators of
// sum w y, sum w x, sum w and the member count per codeword, flushed as
// per-chunk partials and reduced in a fixed order by the finalize kernel,
// which also rebuilds the MFMA operand tiles for the next iteration.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "gsrq.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int DP = 8;            // subvector slots per MFMA k-chunk
constexpr int TILES = 16;        // 16 tiles x 16 codewords = K <= 256
constexpr int KMAX = TILES * 16;
constexpr int ACC = 18;          // sum w y[8], sum w x[8], W, count
constexpr int PSTRIDE = KMAX * ACC + 2;  // + objective, changed flag
constexpr int TRAIN_WAVES = 8;
constexpr int TRAIN_CHUNK_ROWS = 8192;
constexpr int ENC_WAVES = 8;      // one subspace per wave
constexpr int ENC_CHUNK_ROWS = 1024;
constexpr float Y_EPS = 1e-8f;            // y = x / (||x|| + eps)
constexpr double SHAPE_KEEP_REL = 1e-6;   // keep s when ||sum w y|| <= 1e-6 W
constexpr float PAD_BIAS = 32768.f;       // g^2 slot of a padding codeword

enum { MODE_INIT = 0, MODE_ITER = 1 };

// ---------------------------------------------------------------- helpers

__device__ __forceinline__ uint32_t pack2(_Float16 lo, _Float16 hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

__device__ __forceinline__ h8 as_h8(u4 v) { return __builtin_bit_cast(h8, v); }

template <typename T> __device__ __forceinline__ float to_f(T v) { return (float)v; }

__device__ __forceinline__ int wave_lane() { return threadIdx.x & 63; }

// Build the 8 float16 A-operand values of tile entry (lane l) for codeword k
// of one codebook.  ex = exponent of sigma (sigma = 2^ex >= max gain).
//   lane group q = l / 16 selects the k-chunk:
//   q0: hi(a)   q1: lo(a)   q2: hi(a)   q3: [hi(gg) lo(gg) 1 1 0 0 0 0]
// with a_j = -2 g s_j / sigma and gg = (g / sigma)^2.
__device__ u4 make_a_entry(int q, bool real, float g, const float* s, int d, int ex) {
  _Float16 v[8];
  if (!real) {
    for (int j = 0; j < 8; ++j) v[j] = (_Float16)0.f;
    if (q == 3) { v[0] = (_Float16)PAD_BIAS; v[2] = (_Float16)1.f; v[3] = (_Float16)1.f; }
  } else if (q == 3) {
    float gs = ldexpf(g, -ex);
    float gg = gs * gs;
    _Float16 hi = (_Float16)gg;
    _Float16 lo = (_Float16)(gg - (float)hi);
    for (int j = 0; j < 8; ++j) v[j] = (_Float16)0.f;
    v[0] = hi; v[1] = lo; v[2] = (_Float16)1.f; v[3] = (_Float16)1.f;
  } else {
    for (int j = 0; j < 8; ++j) {
      float a = (j < d) ? ldexpf(-2.f * g * s[j], -ex) : 0.f;
      _Float16 hi = (_Float16)a;
      v[j] = (q == 1) ? (_Float16)(a - (float)hi) : hi;
    }
  }
  u4 r;
  r[0] = pack2(v[0], v[1]); r[1] = pack2(v[2], v[3]);
  r[2] = pack2(v[4], v[5]); r[3] = pack2(v[6], v[7]);
  return r;
}

__device__ __forceinline__ int sigma_exp(float maxg) {
  if (!(maxg > 0.f)) return 0;
  int e;
  frexpf(maxg, &e);   // maxg = m 2^e, m in [0.5, 1): 2^e >= maxg
  return e;
}

// One 256-thread block builds the TILES x 64 operand entries of a codebook.
// gl/sh: gains [K] and shapes [K][d] (may live in LDS); unit_gain treats
// every gain as 1.  red: >= 256 floats of LDS scratch.
__device__ void build_codebook_tiles(const float* gl, const float* sh, int d, int K,
                                     bool unit_gain, u4* frag, int* sig, float* red) {
  const int tid = threadIdx.x;
  float m = 0.f;
  for (int k = tid; k < K; k += blockDim.x) m = fmaxf(m, unit_gain ? 1.f : gl[k]);
  red[tid] = m;
  __syncthreads();
  for (int s = blockDim.x / 2; s > 0; s >>= 1) {
    if (tid < s) red[tid] = fmaxf(red[tid], red[tid + s]);
    __syncthreads();
  }
  const int ex = sigma_exp(red[0]);
  for (int e = tid; e < TILES * 64; e += blockDim.x) {
    const int t = e >> 6, l = e & 63;
    const int k = t * 16 + (l & 15);
    const bool real = k < K;
    const float g = real ? (unit_gain ? 1.f : gl[k]) : 0.f;
    frag[e] = make_a_entry(l >> 4, real, g, real ? sh + (size_t)k * d : sh, d, ex);
  }
  if (tid == 0) *sig = ex;
  __syncthreads();
}

// Per-row B operand.  x: the row's subvector (zero padded to 8).  ex: sigma
// exponent.  Returns the lane's operand; sets rr (= ||x||^2 / (sigma rho))
// and need_exact (row must go to the float64 fallback).
__device__ __forceinline__ h8 make_b(const float (&x)[8], int ex, int q, float& rr, float& ss,
                                     bool& need_exact) {
  float mx = 0.f;
  ss = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) { mx = fmaxf(mx, fabsf(x[j])); ss = fmaf(x[j], x[j], ss); }
  int er = 0;
  if (mx > 0.f) frexpf(mx, &er);
  int sr = ex - er;                        // sigma / rho = 2^sr
  need_exact = !(mx > 0.f) || sr > 5 || sr < -12 || !(ss < 3.0e38f);
  sr = sr < -12 ? -12 : (sr > 14 ? 14 : sr);
  rr = ldexpf(ss, -(ex + er));
  rr = fminf(rr, 60000.f);
  h8 b;
  if (q == 3) {
    const _Float16 sc = (_Float16)ldexpf(1.f, sr);
    const _Float16 hi = (_Float16)rr;
    const _Float16 lo = (_Float16)(rr - (float)hi);
    b[0] = sc; b[1] = sc; b[2] = hi; b[3] = lo;
    b[4] = b[5] = b[6] = b[7] = (_Float16)0.f;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float v = ldexpf(x[j], -er);
      const _Float16 hi = (_Float16)v;
      b[j] = (q == 2) ? (_Float16)(v - (float)hi) : hi;
    }
  }
  return b;
}

// 16 MFMA tiles -> the lane's minimum packed key over its 64 codewords.
// key = (bits(dist) & ~63) | (tile << 2 | slot); the lane's lane group q
// fixes the remaining index bits (k = 16 tile + 4 q + slot).
__device__ __forceinline__ int min_key(const u4 (&af)[TILES], h8 b) {
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  f4 c[TILES];
  // all products first so the scheduler can overlap MFMA latency with the
  // integer epilogue of earlier tiles
#pragma unroll
  for (int t = 0; t < TILES; ++t)
    c[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(af[t]), b, zero, 0, 0, 0);
  int best = 0x7fffffff;
#pragma unroll
  for (int t = 0; t < TILES; ++t) {
    const int k0 = (__float_as_int(c[t][0]) & ~63) | (t * 4 + 0);
    const int k1 = (__float_as_int(c[t][1]) & ~63) | (t * 4 + 1);
    const int k2 = (__float_as_int(c[t][2]) & ~63) | (t * 4 + 2);
    const int k3 = (__float_as_int(c[t][3]) & ~63) | (t * 4 + 3);
    best = min(min(best, k0), min(k1, min(k2, k3)));
  }
  return best;
}

// Combine the four lane groups of each row: smallest distance key, ties to
// the lowest codeword index.  Returns the codeword; dhat = approximate
// scaled distance of the winner.
__device__ __forceinline__ int reduce_rows(int key, int q, float& dhat) {
  const int kidx = ((key & 63) >> 2) * 16 + q * 4 + (key & 3);
  long long v = (long long)(key >> 6) * 4294967296ll + (long long)kidx;
  long long o = __shfl_xor(v, 16);
  v = o < v ? o : v;
  o = __shfl_xor(v, 32);
  v = o < v ? o : v;
  dhat = __int_as_float((int)(v >> 32) << 6);
  return (int)(v & 0xffffffffll);
}

// Exact float64 argmin over all K codewords for the rows flagged in `mask`
// (one bit per lane of lane group 0; bit i = row i of the block).  gain /
// shape: this codebook, [K] / [K][ld] with d used elements per row (any
// memory).  Every lane of the wave takes part; the lanes of a flagged row
// receive its codeword in kstar.
__device__ __forceinline__ void exact_rows(unsigned long long mask, const float (&x)[8], int d,
                                           int ld, int K, const float* gain, const float* shape,
                                           bool unit_gain, int& kstar) {
  const int lane = wave_lane();
  while (mask) {
    const int L = __ffsll((long long)mask) - 1;
    mask &= mask - 1;
    double xr[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) xr[j] = (double)__shfl(x[j], L);
    double bd = INFINITY;
    int bk = 0x7fffffff;
    for (int k = lane; k < K; k += 64) {
      const double g = unit_gain ? 1.0 : (double)gain[k];
      double dist = 0.0;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const double c = (j < d) ? g * (double)shape[(size_t)k * ld + j] : 0.0;
        const double r = xr[j] - c;
        dist = fma(r, r, dist);
      }
      if (dist < bd) { bd = dist; bk = k; }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const double od = __shfl_xor(bd, off);
      const int ok = __shfl_xor(bk, off);
      if (od < bd || (od == bd && ok < bk)) { bd = od; bk = ok; }
    }
    if ((lane & 15) == L) kstar = bk;
  }
}

// ---------------------------------------------------------------- kernels

__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// X [N][ldx] -> Xt [G][N][8] (zero padded past d), same element type.
template <typename T>
__global__ void transpose_kernel(const T* __restrict__ X, int64_t ldx, int64_t N, int d, int G,
                                 T* __restrict__ Xt) {
  // 64 consecutive threads cover 8 rows x 8 subspaces: coalesced reads of a
  // row's 8 subspaces and 8 full-line writes per subspace
  const int64_t rows8 = (N + 7) / 8;
  const int64_t total = rows8 * (int64_t)((G + 7) / 8) * 64;
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < total;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int64_t blk = c / 64;
    const int within = (int)(c % 64);
    const int64_t gb = blk / rows8, rb = blk % rows8;
    const int64_t row = rb * 8 + within / 8;
    const int g = (int)gb * 8 + within % 8;
    if (row >= N || g >= G) continue;
    const T* src = X + row * ldx + (int64_t)g * d;
    T v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = (j < d) ? src[j] : (T)0.f;
    T* dst = Xt + ((int64_t)g * N + row) * 8;
#pragma unroll
    for (int j = 0; j < 8; ++j) dst[j] = v[j];
  }
}

// Seed shapes: s_k = x_r / (||x_r|| + eps) for r = seed row of codeword k.
template <typename T>
__global__ void seed_kernel(const T* __restrict__ Xt, int64_t N, int d, int K,
                            const int32_t* __restrict__ seeds, float* __restrict__ shape,
                            float* __restrict__ seednorm) {
  const int g = blockIdx.x;
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    const int64_t row = seeds[(size_t)g * K + k];
    const T* x = Xt + ((int64_t)g * N + row) * 8;
    double ss = 0.0;
    for (int j = 0; j < d; ++j) { const double v = to_f(x[j]); ss = fma(v, v, ss); }
    const double nrm = sqrt(ss);
    for (int j = 0; j < d; ++j)
      shape[((size_t)g * K + k) * d + j] = (float)((double)to_f(x[j]) / (nrm + (double)Y_EPS));
    seednorm[(size_t)g * K + k] = (float)nrm;
  }
}

// Operand tiles for ncb codebooks (gain [ncb][K], shape [ncb][K][d]).
__global__ void tiles_kernel(const float* __restrict__ gain, const float* __restrict__ shape,
                             int d, int K, int unit_gain, u4* __restrict__ frag,
                             int* __restrict__ sig) {
  __shared__ float red[256];
  const int cb = blockIdx.x;
  build_codebook_tiles(gain + (size_t)cb * K, shape + (size_t)cb * K * d, d, K, unit_gain != 0,
                       frag + (size_t)cb * TILES * 64, sig + cb, red);
}

struct AssignArgs {
  const void* xt;        // [G][N][8]
  int64_t N;
  int d, K, G;
  const float* w;        // [N] or null
  const float* gain;     // [G][K]
  const float* shape;    // [G][K][d]
  const u4* frag;        // [G][TILES*64]
  const int* sig;        // [G]
  uint16_t* assign;      // [G][N]
  const int* done;       // [G]
  double* part;          // [G][chunks][PSTRIDE]
  int chunks;
  int force_changed;
};

// Fused assignment (eq. 5) + weighted accumulation (eqs. 6-8) for one
// (chunk of rows, subspace).  MODE_INIT scores with unit gains (largest
// projection) for the gain initialisation.
template <typename T, int MODE>
__global__ void __launch_bounds__(TRAIN_WAVES * 64)
assign_accumulate_kernel(AssignArgs a) {
  __shared__ double acc[KMAX * ACC];
  __shared__ float cbg[KMAX];
  __shared__ float cbs[KMAX * DP];
  __shared__ double objw[TRAIN_WAVES];
  __shared__ int changed;

  const int g = blockIdx.y;
  const int chunk = blockIdx.x;
  if (a.done[g]) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = lane & 15, q = lane >> 4;
  const int d = a.d, K = a.K;

  for (int e = tid; e < KMAX * ACC; e += blockDim.x) acc[e] = 0.0;
  for (int k = tid; k < KMAX; k += blockDim.x) {
    cbg[k] = (k < K) ? (MODE == MODE_INIT ? 1.f : a.gain[(size_t)g * K + k]) : 0.f;
    for (int j = 0; j < DP; ++j)
      cbs[k * DP + j] = (k < K && j < d) ? a.shape[((size_t)g * K + k) * d + j] : 0.f;
  }
  if (tid == 0) changed = a.force_changed;

  u4 af[TILES];
  const u4* fr = a.frag + (size_t)g * TILES * 64;
#pragma unroll
  for (int t = 0; t < TILES; ++t) af[t] = fr[t * 64 + lane];
  const int ex = a.sig[g];
  __syncthreads();

  const T* xt = (const T*)a.xt + (size_t)g * a.N * 8;
  const int64_t row_begin = (int64_t)chunk * TRAIN_CHUNK_ROWS;
  int64_t row_end = row_begin + TRAIN_CHUNK_ROWS;
  if (row_end > a.N) row_end = a.N;
  const int nblk = (int)((row_end - row_begin + 15) / 16);
  double obj = 0.0;
  bool any_changed = false;

  for (int rb = wave; rb < nblk; rb += TRAIN_WAVES) {
    const int64_t row = row_begin + (int64_t)rb * 16 + i;
    const bool valid = row < row_end;
    float x[8];
    if (valid) {
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = to_f(xt[row * 8 + j]);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = 0.f;
    }
    float rr, ss;
    bool need_exact;
    const h8 b = make_b(x, ex, q, rr, ss, need_exact);
    const int key = min_key(af, b);
    float dhat;
    int kstar = reduce_rows(key, q, dhat);
    need_exact = need_exact || !(dhat <= 2.f * rr) || kstar >= K;
    const unsigned long long fb = __ballot(valid && need_exact && q == 0);
    if (fb) exact_rows(fb, x, d, DP, K, cbg, cbs, MODE == MODE_INIT, kstar);
    if (kstar >= K) kstar = K - 1;   // only tail rows past N can get here
    // chosen-codeword distance, exact in float32 (objective)
    const float gk = cbg[kstar];
    float dist = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float r = fmaf(-gk, cbs[kstar * DP + j], x[j]);
      dist = fmaf(r, r, dist);
    }
    if (valid) {
      const double wv = a.w ? (double)a.w[row] : 1.0;
      const float inv = 1.f / (sqrtf(ss) + Y_EPS);
      // lane group q adds slots 4q..4q+3: q0/q1 the y half-vectors,
      // q2/q3 the x half-vectors; q0 also adds W, q1 the member count
      double* ak = acc + kstar * ACC;
      const float sc = (q < 2) ? inv : 1.f;
      // bitwise select keeps x in registers (a conditional would become a
      // dynamically indexed private array)
      const int hm = -(q & 1);
      float xv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        xv[j] = __int_as_float((__float_as_int(x[4 + j]) & hm) | (__float_as_int(x[j]) & ~hm));
#pragma unroll
      for (int j = 0; j < 4; ++j) unsafeAtomicAdd(ak + 4 * q + j, wv * (double)(xv[j] * sc));
      if (q < 2) unsafeAtomicAdd(ak + 16 + q, q == 0 ? wv : 1.0);
      if (q == 0) {
        obj += wv * (double)dist;
        uint16_t* ap = a.assign + (size_t)g * a.N + row;
        if (MODE == MODE_ITER && *ap != (uint16_t)kstar) any_changed = true;
        *ap = (uint16_t)kstar;
      }
    }
  }
  // wave sums of the objective and changed flag
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) obj += __shfl_xor(obj, off);
  if (lane == 0) objw[wave] = obj;
  if (__ballot(any_changed) && lane == 0) atomicOr(&changed, 1);
  __syncthreads();
  double* out = a.part + ((size_t)g * a.chunks + chunk) * PSTRIDE;
  for (int e = tid; e < KMAX * ACC; e += blockDim.x) out[e] = acc[e];
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < TRAIN_WAVES; ++w) s += objw[w];
    out[KMAX * ACC] = s;
    out[KMAX * ACC + 1] = (double)changed;
  }
}

struct FinalizeArgs {
  int d, K, G, chunks, T;
  int t;                  // iteration number (1-based); 0 for init
  int no_early_stop;
  const double* part;
  const float* seednorm;  // [G][K]
  float* gain;            // [G][K]
  float* shape;           // [G][K][d]
  u4* frag;
  int* sig;
  int* done;              // [G]
  int* iters;             // [G]
  double* trace;          // [G][T] or null
};

// Codebook update from the partial sums of every chunk (fixed order):
// init: eq. (8) gains for the seed shapes; iteration: eqs. (7) and (8).
// Then the stop test and the operand tiles of the new codebook.
template <int MODE>
__global__ void __launch_bounds__(256) finalize_kernel(FinalizeArgs a) {
  __shared__ float gl[KMAX];
  __shared__ float sh[KMAX * DP];
  __shared__ float red[256];
  __shared__ double objc[2];
  const int g = blockIdx.x;
  if (MODE == MODE_ITER && a.done[g]) return;
  const int k = threadIdx.x;
  const int d = a.d, K = a.K;
  if (k < K) {
    double s[ACC];
    for (int e = 0; e < ACC; ++e) s[e] = 0.0;
    for (int c = 0; c < a.chunks; ++c) {
      const double* p = a.part + ((size_t)g * a.chunks + c) * PSTRIDE + (size_t)k * ACC;
      for (int e = 0; e < ACC; ++e) s[e] += p[e];
    }
    float* sk = a.shape + ((size_t)g * K + k) * d;
    float* gk = a.gain + (size_t)g * K + k;
    double sn[DP];
    for (int j = 0; j < DP; ++j) sn[j] = (j < d) ? (double)sk[j] : 0.0;
    double gnew = (MODE == MODE_INIT) ? (double)a.seednorm[(size_t)g * K + k] : (double)*gk;
    const double W = s[16];
    if (W > 0.0) {
      if (MODE == MODE_ITER) {
        double mn = 0.0;
        for (int j = 0; j < d; ++j) mn = fma(s[j], s[j], mn);
        mn = sqrt(mn);
        if (mn > SHAPE_KEEP_REL * W)
          for (int j = 0; j < d; ++j) sn[j] = s[j] / mn;
      }
      double pr = 0.0;
      for (int j = 0; j < d; ++j) pr = fma(s[8 + j], sn[j], pr);
      gnew = fmax(0.0, pr / W);
    }
    for (int j = 0; j < d; ++j) sk[j] = (float)sn[j];
    *gk = (float)gnew;
    gl[k] = (float)gnew;
    for (int j = 0; j < DP; ++j) sh[k * DP + j] = (j < d) ? (float)sn[j] : 0.f;
  }
  if (k == 0) {
    double obj = 0.0, ch = 0.0;
    for (int c = 0; c < a.chunks; ++c) {
      const double* p = a.part + ((size_t)g * a.chunks + c) * PSTRIDE + KMAX * ACC;
      obj += p[0];
      ch = fmax(ch, p[1]);
    }
    objc[0] = obj;
    objc[1] = ch;
    if (MODE == MODE_ITER) {
      if (a.trace) a.trace[(size_t)g * a.T + (a.t - 1)] = obj;
      a.iters[g] = a.t;
      if (ch == 0.0 && !a.no_early_stop) a.done[g] = 1;
    }
  }
  __syncthreads();
  // operand tiles read the float32 codebook just stored (LDS copy, stride DP)
  {
    const int tid = threadIdx.x;
    float m = 0.f;
    for (int kk = tid; kk < K; kk += blockDim.x) m = fmaxf(m, gl[kk]);
    red[tid] = m;
    __syncthreads();
    for (int s2 = blockDim.x / 2; s2 > 0; s2 >>= 1) {
      if (tid < s2) red[tid] = fmaxf(red[tid], red[tid + s2]);
      __syncthreads();
    }
    const int ex = sigma_exp(red[0]);
    u4* fr = a.frag + (size_t)g * TILES * 64;
    for (int e = tid; e < TILES * 64; e += blockDim.x) {
      const int t = e >> 6, l = e & 63;
      const int kk = t * 16 + (l & 15);
      const bool real = kk < K;
      fr[e] = make_a_entry(l >> 4, real, real ? gl[kk] : 0.f, real ? sh + kk * DP : sh, d, ex);
    }
    if (tid == 0) a.sig[g] = ex;
  }
}

struct EncodeArgs {
  const void* x;         // [N][ldx]
  int64_t ldx, N;
  int d, K, G, M, b, words;
  const float* gain;     // [M][G][K]
  const float* shape;    // [M][G][K][d]
  const u4* frag;        // [M*G][TILES*64]
  const int* sig;        // [M*G]
  uint32_t* codes;       // [N][words] or null
  float* residual;       // [N][D] or null
  int byte_codes;        // b == 8: plain byte stores, else atomic OR
};

// Stage-fused encoder: one subspace per wave, the residual of a 16-row block
// stays in registers through all M stages.
template <typename T, bool MULTI>
__global__ void __launch_bounds__(ENC_WAVES * 64) encode_kernel(EncodeArgs a) {
  const int lane = wave_lane(), wave = threadIdx.x >> 6;
  const int g = blockIdx.y * ENC_WAVES + wave;
  if (g >= a.G) return;
  const int i = lane & 15, q = lane >> 4;
  const int d = a.d, K = a.K, G = a.G;
  u4 af[TILES];
  if (!MULTI) {
    const u4* fr = a.frag + (size_t)g * TILES * 64;
#pragma unroll
    for (int t = 0; t < TILES; ++t) af[t] = fr[t * 64 + lane];
  }
  const int64_t row_begin = (int64_t)blockIdx.x * ENC_CHUNK_ROWS;
  int64_t row_end = row_begin + ENC_CHUNK_ROWS;
  if (row_end > a.N) row_end = a.N;
  const T* X = (const T*)a.x;
  for (int64_t r0 = row_begin; r0 < row_end; r0 += 16) {
    const int64_t row = r0 + i;
    const bool valid = row < row_end;
    float x[8];
    const T* src = X + row * a.ldx + (int64_t)g * d;
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (valid && j < d) ? to_f(src[j]) : 0.f;
    for (int m = 0; m < a.M; ++m) {
      const int cb = m * G + g;
      if (MULTI) {
        const u4* fr = a.frag + (size_t)cb * TILES * 64;
#pragma unroll
        for (int t = 0; t < TILES; ++t) af[t] = fr[t * 64 + lane];
      }
      const int ex = a.sig[cb];
      float rr, ss;
      bool need_exact;
      const h8 b = make_b(x, ex, q, rr, ss, need_exact);
      const int key = min_key(af, b);
      float dhat;
      int kstar = reduce_rows(key, q, dhat);
      need_exact = need_exact || !(dhat <= 2.f * rr) || kstar >= K;
      const float* gcb = a.gain + (size_t)cb * K;
      const float* scb = a.shape + (size_t)cb * K * d;
      const unsigned long long fb = __ballot(valid && need_exact && q == 0);
      if (fb) exact_rows(fb, x, d, d, K, gcb, scb, false, kstar);
      if (kstar >= K) kstar = K - 1;   // only tail rows past N can get here
      const float gk = gcb[kstar];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < d) x[j] = fmaf(-gk, scb[(size_t)kstar * d + j], x[j]);
      if (valid && q == 0 && a.codes) {
        const int64_t t = (int64_t)m * G + g;
        if (a.byte_codes) {
          ((uint8_t*)(a.codes + row * a.words))[t] = (uint8_t)kstar;
        } else {
          const int64_t bit = t * a.b;
          uint32_t* wp = a.codes + row * a.words + bit / 32;
          const int off = (int)(bit % 32);
          atomicOr(wp, (uint32_t)kstar << off);
          if (off + a.b > 32) atomicOr(wp + 1, (uint32_t)kstar >> (32 - off));
        }
      }
    }
    if (valid && a.residual && q == 0) {
      float* dst = a.residual + row * (int64_t)(G * d) + (int64_t)g * d;
      for (int j = 0; j < d; ++j) dst[j] = x[j];
    }
  }
}

struct DecodeArgs {
  const uint32_t* codes;
  int64_t N, ldo;
  int d, K, G, M_use, b, words;
  const float* gain;
  const float* shape;
  void* out;
};

// Gather-sum decoder: one thread per (row, subspace), float32 accumulation
// in stage order with one fused multiply-add per stage.
template <typename TO>
__global__ void decode_kernel(DecodeArgs a) {
  const int64_t total = a.N * a.G;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = e / a.G;
    const int g = (int)(e % a.G);
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    const uint32_t* cr = a.codes + row * a.words;
    for (int m = 0; m < a.M_use; ++m) {
      const int64_t bit = ((int64_t)m * a.G + g) * a.b;
      const int64_t wi = bit / 32;
      const int off = (int)(bit % 32);
      uint64_t v = cr[wi];
      if (off + a.b > 32) v |= (uint64_t)cr[wi + 1] << 32;
      const int k = (int)((v >> off) & ((1ull << a.b) - 1));
      const size_t cb = (size_t)m * a.G + g;
      const float gk = a.gain[cb * a.K + k];
      const float* s = a.shape + (cb * a.K + k) * a.d;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < a.d) acc[j] = fmaf(gk, s[j], acc[j]);
    }
    TO* dst = (TO*)a.out + row * a.ldo + (int64_t)g * a.d;
    for (int j = 0; j < a.d; ++j) dst[j] = (TO)acc[j];
  }
}

// ------------------------------------------------------------- host side

inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

int log2i(int64_t v) {
  int b = 0;
  while ((1ll << b) < v) ++b;
  return b;
}

gsrq_status check_shape(const gsrq_shape* s, bool need_m) {
  if (!s) return GSRQ_E_ARG;
  if (s->N < 1 || s->D < 1 || s->d < 1 || s->D % s->d != 0) return GSRQ_E_ARG;
  if (s->K < 2 || s->K > 65536 || !is_pow2(s->K)) return GSRQ_E_ARG;
  if (need_m && s->M < 1) return GSRQ_E_ARG;
  return GSRQ_OK;
}

gsrq_status check_supported(const gsrq_shape* s) {
  if (s->d > DP || s->K > KMAX) return GSRQ_E_UNSUPPORTED;
  return GSRQ_OK;
}

struct TrainLayout {
  size_t xt, frag, sig, part, assign, done, iters, seednorm, seeds, total;
  int chunks;
};

TrainLayout train_layout(const gsrq_shape* s, size_t elt) {
  TrainLayout L;
  const int64_t G = s->D / s->d;
  L.chunks = (int)((s->N + TRAIN_CHUNK_ROWS - 1) / TRAIN_CHUNK_ROWS);
  size_t off = 0;
  L.xt = off; off = align256(off + (size_t)G * s->N * 8 * elt);
  L.frag = off; off = align256(off + (size_t)G * TILES * 64 * sizeof(u4));
  L.sig = off; off = align256(off + (size_t)G * sizeof(int));
  L.part = off; off = align256(off + (size_t)G * L.chunks * PSTRIDE * sizeof(double));
  L.assign = off; off = align256(off + (size_t)G * s->N * sizeof(uint16_t));
  L.done = off; off = align256(off + (size_t)G * sizeof(int));
  L.iters = off; off = align256(off + (size_t)G * sizeof(int));
  L.seednorm = off; off = align256(off + (size_t)G * s->K * sizeof(float));
  L.seeds = off; off = align256(off + (size_t)G * s->K * sizeof(int32_t));
  L.total = off;
  return L;
}

size_t encode_ws(const gsrq_shape* s) {
  const int64_t G = s->D / s->d;
  return align256((size_t)s->M * G * TILES * 64 * sizeof(u4)) +
         align256((size_t)s->M * G * sizeof(int));
}

int grid_for(int64_t work, int block) {
  int64_t b = (work + block - 1) / block;
  if (b > 65536) b = 65536;
  if (b < 1) b = 1;
  return (int)b;
}

gsrq_status launch_ok() {
  return hipGetLastError() == hipSuccess ? GSRQ_OK : GSRQ_E_HIP;
}

gsrq_status fill_u32(void* p, size_t n, uint32_t v, hipStream_t st) {
  if (n == 0) return GSRQ_OK;
  fill_u32_kernel<<<grid_for((int64_t)n, 256), 256, 0, st>>>((uint32_t*)p, n, v);
  return launch_ok();
}

template <typename T>
gsrq_status encode_launch(const gsrq_shape* s, const void* X, int64_t ldx, const float* gain,
                          const float* shape, const u4* frag, const int* sig, int M,
                          uint32_t* codes, float* residual, hipStream_t st) {
  EncodeArgs a;
  a.x = X; a.ldx = ldx; a.N = s->N; a.d = s->d; a.K = s->K; a.G = s->D / s->d; a.M = M;
  a.b = log2i(s->K);
  a.words = (int)((M * (int64_t)a.G * a.b + 31) / 32);
  a.gain = gain; a.shape = shape; a.frag = frag; a.sig = sig;
  a.codes = codes; a.residual = residual;
  a.byte_codes = (a.b == 8) && ((M * (int64_t)a.G) % 4 == 0);
  if (codes && !a.byte_codes) {
    gsrq_status e = fill_u32(codes, (size_t)s->N * a.words, 0u, st);
    if (e) return e;
  }
  dim3 grid((unsigned)((s->N + ENC_CHUNK_ROWS - 1) / ENC_CHUNK_ROWS),
            (unsigned)((a.G + ENC_WAVES - 1) / ENC_WAVES));
  if (M > 1)
    encode_kernel<T, true><<<grid, ENC_WAVES * 64, 0, st>>>(a);
  else
    encode_kernel<T, false><<<grid, ENC_WAVES * 64, 0, st>>>(a);
  return launch_ok();
}

template <typename T>
gsrq_status train_impl(const gsrq_shape* s, const void* X, int64_t ldx, const float* w, int T_,
                       const int32_t* seeds, uint32_t flags, float* gain, float* shape,
                       float* R_next, uint16_t* assign_io, int32_t* iters_run, double* trace,
                       void* ws, hipStream_t st) {
  const TrainLayout L = train_layout(s, sizeof(T));
  char* base = (char*)ws;
  T* xt = (T*)(base + L.xt);
  u4* frag = (u4*)(base + L.frag);
  int* sig = (int*)(base + L.sig);
  double* part = (double*)(base + L.part);
  uint16_t* assign = assign_io ? assign_io : (uint16_t*)(base + L.assign);
  int* done = (int*)(base + L.done);
  int* iters = iters_run ? iters_run : (int*)(base + L.iters);
  float* seednorm = (float*)(base + L.seednorm);
  int32_t* dseeds = (int32_t*)(base + L.seeds);
  const int G = s->D / s->d;
  const int K = s->K, d = s->d;
  const bool resume = flags & GSRQ_RESUME;
  gsrq_status e;

  {
    const int64_t work = ((s->N + 7) / 8) * (int64_t)((G + 7) / 8) * 64;
    transpose_kernel<T><<<grid_for(work, 256), 256, 0, st>>>((const T*)X, ldx, s->N, d, G, xt);
    if ((e = launch_ok())) return e;
  }
  if ((e = fill_u32(done, G, 0u, st))) return e;
  if ((e = fill_u32(iters, G, 0u, st))) return e;
  if (trace && T_ > 0 && (e = fill_u32(trace, (size_t)G * T_ * 2, 0u, st))) return e;

  AssignArgs aa;
  aa.xt = xt; aa.N = s->N; aa.d = d; aa.K = K; aa.G = G; aa.w = w;
  aa.gain = gain; aa.shape = shape; aa.frag = frag; aa.sig = sig; aa.assign = assign;
  aa.done = done; aa.part = part; aa.chunks = L.chunks; aa.force_changed = 0;
  FinalizeArgs fa;
  fa.d = d; fa.K = K; fa.G = G; fa.chunks = L.chunks; fa.T = T_; fa.t = 0;
  fa.no_early_stop = (flags & GSRQ_NO_EARLY_STOP) ? 1 : 0;
  fa.part = part; fa.seednorm = seednorm; fa.gain = gain; fa.shape = shape;
  fa.frag = frag; fa.sig = sig; fa.done = done; fa.iters = iters; fa.trace = trace;
  const dim3 agrid((unsigned)L.chunks, (unsigned)G);

  if (!resume) {
    if (hipMemcpyAsync(dseeds, seeds, (size_t)G * K * sizeof(int32_t), hipMemcpyHostToDevice,
                       st) != hipSuccess)
      return GSRQ_E_HIP;
    seed_kernel<T><<<G, 256, 0, st>>>(xt, s->N, d, K, dseeds, shape, seednorm);
    if ((e = launch_ok())) return e;
    tiles_kernel<<<G, 256, 0, st>>>(gain, shape, d, K, 1, frag, sig);
    if ((e = launch_ok())) return e;
    assign_accumulate_kernel<T, MODE_INIT><<<agrid, TRAIN_WAVES * 64, 0, st>>>(aa);
    if ((e = launch_ok())) return e;
    finalize_kernel<MODE_INIT><<<G, 256, 0, st>>>(fa);
    if ((e = launch_ok())) return e;
  } else {
    tiles_kernel<<<G, 256, 0, st>>>(gain, shape, d, K, 0, frag, sig);
    if ((e = launch_ok())) return e;
    aa.force_changed = (flags & GSRQ_ASSIGN_IN) ? 0 : 1;
  }
  for (int t = 1; t <= T_; ++t) {
    assign_accumulate_kernel<T, MODE_ITER><<<agrid, TRAIN_WAVES * 64, 0, st>>>(aa);
    if ((e = launch_ok())) return e;
    aa.force_changed = 0;
    fa.t = t;
    finalize_kernel<MODE_ITER><<<G, 256, 0, st>>>(fa);
    if ((e = launch_ok())) return e;
  }
  if (R_next) {
    gsrq_shape s1 = *s;
    s1.M = 1;
    return encode_launch<T>(&s1, X, ldx, gain, shape, frag, sig, 1, nullptr, R_next, st);
  }
  return GSRQ_OK;
}

}  // namespace

// ------------------------------------------------------------------ C ABI

extern "C" {

const char* gsrq_status_string(gsrq_status st) {
  switch (st) {
    case GSRQ_OK: return "ok";
    case GSRQ_E_ARG: return "invalid argument";
    case GSRQ_E_UNSUPPORTED: return "unsupported shape";
    case GSRQ_E_WORKSPACE: return "workspace too small";
    case GSRQ_E_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

size_t gsrq_code_words(const gsrq_shape* s) {
  if (check_shape(s, true) != GSRQ_OK) return 0;
  const int64_t G = s->D / s->d;
  return (size_t)((s->M * G * log2i(s->K) + 31) / 32);
}

double gsrq_bits_per_element(const gsrq_shape* s) {
  if (check_shape(s, true) != GSRQ_OK) return 0.0;
  return (double)s->M * log2i(s->K) / (double)s->d;
}

gsrq_status gsrq_train_workspace_bytes(const gsrq_shape* s, size_t* bytes) {
  gsrq_status e = check_shape(s, false);
  if (e) return e;
  if (!bytes) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  // sized for the wider input type so one workspace serves both
  *bytes = train_layout(s, sizeof(float)).total;
  return GSRQ_OK;
}

gsrq_status gsrq_encode_workspace_bytes(const gsrq_shape* s, size_t* bytes) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!bytes) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  *bytes = encode_ws(s);
  return GSRQ_OK;
}

gsrq_status gsrq_train_stage(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype,
                             int64_t ldx, const float* w, int32_t T, const int32_t* seed_rows,
                             uint32_t flags, float* gain, float* shape, float* R_next,
                             uint16_t* assign_io, int32_t* iters_run, double* obj_trace,
                             void* workspace, size_t ws_bytes, void* stream) {
  gsrq_status e = check_shape(s, false);
  if (e) return e;
  if (!X || !gain || !shape || !workspace) return GSRQ_E_ARG;
  if (x_dtype != GSRQ_F32 && x_dtype != GSRQ_F16) return GSRQ_E_ARG;
  if (ldx < s->D || T < 0 || s->N < s->K) return GSRQ_E_ARG;
  if (T == 0 && (flags & GSRQ_RESUME)) return GSRQ_E_ARG;
  if (flags & ~(uint32_t)(GSRQ_RESUME | GSRQ_ASSIGN_IN | GSRQ_NO_EARLY_STOP)) return GSRQ_E_ARG;
  if ((flags & GSRQ_ASSIGN_IN) && (!(flags & GSRQ_RESUME) || !assign_io)) return GSRQ_E_ARG;
  if (((uintptr_t)workspace & 255) != 0) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  const int64_t G = s->D / s->d;
  if (!(flags & GSRQ_RESUME)) {
    if (!seed_rows) return GSRQ_E_ARG;
    for (int64_t g = 0; g < G; ++g) {
      const int32_t* r = seed_rows + g * s->K;
      for (int k = 0; k < s->K; ++k)
        if (r[k] < 0 || r[k] >= s->N) return GSRQ_E_ARG;
      // distinct within the subspace: sort a copy
      int32_t* tmp = new int32_t[s->K];
      memcpy(tmp, r, sizeof(int32_t) * s->K);
      // insertion-free check via counting on a bitmap would need N bits;
      // K is at most 256 here, so a simple sort suffices
      for (int a = 1; a < s->K; ++a) {
        int32_t v = tmp[a];
        int b = a - 1;
        while (b >= 0 && tmp[b] > v) { tmp[b + 1] = tmp[b]; --b; }
        tmp[b + 1] = v;
      }
      bool dup = false;
      for (int a = 1; a < s->K; ++a) dup |= tmp[a] == tmp[a - 1];
      delete[] tmp;
      if (dup) return GSRQ_E_ARG;
    }
  }
  const size_t need = train_layout(s, x_dtype == GSRQ_F16 ? sizeof(_Float16) : sizeof(float)).total;
  if (ws_bytes < need) return GSRQ_E_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  if (x_dtype == GSRQ_F16)
    return train_impl<_Float16>(s, X, ldx, w, T, seed_rows, flags, gain, shape, R_next,
                                assign_io, iters_run, obj_trace, workspace, st);
  return train_impl<float>(s, X, ldx, w, T, seed_rows, flags, gain, shape, R_next, assign_io,
                           iters_run, obj_trace, workspace, st);
}

gsrq_status gsrq_encode(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype, int64_t ldx,
                        const float* gain, const float* shape, uint32_t* codes, float* residual,
                        void* workspace, size_t ws_bytes, void* stream) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!X || !gain || !shape || !workspace || (!codes && !residual)) return GSRQ_E_ARG;
  if (x_dtype != GSRQ_F32 && x_dtype != GSRQ_F16) return GSRQ_E_ARG;
  if (ldx < s->D) return GSRQ_E_ARG;
  if (((uintptr_t)workspace & 255) != 0) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  if (ws_bytes < encode_ws(s)) return GSRQ_E_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  const int64_t G = s->D / s->d;
  u4* frag = (u4*)workspace;
  int* sig = (int*)((char*)workspace + align256((size_t)s->M * G * TILES * 64 * sizeof(u4)));
  tiles_kernel<<<(unsigned)(s->M * G), 256, 0, st>>>(gain, shape, s->d, s->K, 0, frag, sig);
  if ((e = launch_ok())) return e;
  if (x_dtype == GSRQ_F16)
    return encode_launch<_Float16>(s, X, ldx, gain, shape, frag, sig, s->M, codes, residual, st);
  return encode_launch<float>(s, X, ldx, gain, shape, frag, sig, s->M, codes, residual, st);
}

gsrq_status gsrq_decode(const gsrq_shape* s, const uint32_t* codes, int32_t M_use,
                        const float* gain, const float* shape, void* Xhat, gsrq_dtype out_dtype,
                        int64_t ldo, void* stream) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!codes || !gain || !shape || !Xhat) return GSRQ_E_ARG;
  if (M_use < 1 || M_use > s->M || ldo < s->D) return GSRQ_E_ARG;
  if (out_dtype != GSRQ_F32 && out_dtype != GSRQ_F16) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  DecodeArgs a;
  a.codes = codes; a.N = s->N; a.ldo = ldo; a.d = s->d; a.K = s->K; a.G = s->D / s->d;
  a.M_use = M_use; a.b = log2i(s->K);
  a.words = (int)((s->M * (int64_t)a.G * a.b + 31) / 32);
  a.gain = gain; a.shape = shape; a.out = Xhat;
  hipStream_t st = (hipStream_t)stream;
  const int grid = grid_for(s->N * a.G, 256);
  if (out_dtype == GSRQ_F16)
    decode_kernel<_Float16><<<grid, 256, 0, st>>>(a);
  else
    decode_kernel<float><<<grid, 256, 0, st>>>(a);
  return launch_ok();
}

}  // extern "C"
