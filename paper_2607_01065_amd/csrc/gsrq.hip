// GSRQ hot path for AMD MI355X (gfx950 / CDNA4): kernels and the C ABI.
//
// What is computed follows arXiv 2607.01065: gain-shape K-means (Sec. 5.2,
// eqs. 3-8, Algorithm 1) with per-row weights (Sec. 5.1, 5.3), product
// subspaces x residual stages (Sec. 3, Sec. 5.1), greedy residual encoding
// and gather-sum decoding.  How it is computed is specific to gfx950:
//
// Scoring (eq. 5) as an MFMA contraction.  For a subspace of dimension
// d <= 8 and one tile of 32 codewords, two chained v_mfma_f32_32x32x16_f16
// produce the squared distances ||r - g s||^2 = ||r||^2 + g^2 - 2 g s.r of
// 32 rows x 32 codewords.  The 32-long contraction carries the dot product
// in a hi/lo float16 split of the codebook side (and of the row side when
// rows are float32), plus the bias terms g^2 and ||r||^2, each split hi/lo.
// Powers of two (sigma per codebook, rho per float32 row) keep every float16
// in range; they scale all distances of a row by one power of two, so the
// argmin is unchanged.  The argmin runs on packed integer keys: the low 7
// bits of each float32 distance are replaced by its (tile, slot) index and
// v_min3_i32 reduces two keys per instruction.  Rows whose key precision
// cannot separate a 1e-4 relative top-2 margin are re-scored exactly in
// float64 (a rare fallback).
//
// Accumulation (eqs. 6-8): per-workgroup float64 LDS accumulators of
// sum w y, sum w x, sum w and the member count per codeword, flushed as
// per-chunk partials and reduced in a fixed order by the update kernel.
#include <algorithm>

#include "gsrq_common.h"
#include "gsrq_wide.h"

GsrqTimingState g_gsrq_timing;

namespace {

constexpr int DP = 8;            // subvector slots of a k-chunk (d <= 8)
constexpr int NT = 8;            // tiles: K <= 256
constexpr int KMAX = NT * CW;
constexpr int ACC = 18;          // sum w y[8], sum w x[8], W, count
constexpr int PSTRIDE = KMAX * ACC + 2;  // + objective, changed flag
// LDS stride of a codeword's sums: odd in 8-byte units, so the rows of a wave
// (random codewords) spread over all bank pairs instead of one in eight
constexpr int ACC_LDS = ACC + 1;
constexpr int TRAIN_WAVES = 12;        // one 768-thread workgroup per CU
constexpr int WAVES_PER_SIMD = 3;      // 168 VGPRs: operand tiles stay in registers
constexpr int TRAIN_CHUNK_MAX = 16384;  // rows of one (chunk, subspace) workgroup, at most
constexpr int TRAIN_CHUNK_MIN = 2048;   // and at least (unless N is smaller)
constexpr int TRAIN_SLOTS = 256;        // workgroups resident at once (one per CU)
constexpr int ENC_SUBS = 4;            // subspaces per encode workgroup
constexpr int ENC_WAVES = 12;          // three waves per subspace, one workgroup per CU
constexpr int ENC_CODES_WORDS = 16384; // LDS-staged code words: stages x chunk rows, at most
constexpr int ENC_MAX_STAGES = 8;      // stages staged in LDS by one encode launch
constexpr int ENC_SMALL_ROWS = 256;    // prepared encode of at most this many rows: latency kernel
constexpr int ENC_SMALL_WAVES = 4;     // (row block, subspace) waves per latency-kernel workgroup
constexpr int KEY_BITS = 7;               // (tile, slot) bits packed into a key

enum { MODE_INIT = 0, MODE_ITER = 1 };
enum { UPD_NONE = 0, UPD_INIT = 1, UPD_ITER = 2 };   // update fused into an assignment launch

// ---------------------------------------------------------------- helpers

// Codeword operand tiles of one codebook, in registers.  Tile t covers
// codewords 32 t + c, c = lane % 32; lane half h = lane / 32 selects the
// k-chunk.  With a_j = -2 g s_j 2^SA / sigma and gg = (g / sigma)^2 2^SA:
//   a1: h0 hi(a), h1 lo(a)                        (contraction k 0..15)
//   a2: h0 hi(a), h1 [hi(gg) lo(gg) 2^SA 2^SA 0 0 0 0]   (k 16..31)
// The 2^SA factor keeps the lo parts out of the float16 subnormal range.
struct Tiles {
  u4 a1[NT], a2[NT];
};

__device__ __forceinline__ void tile_entry(int h, bool real, float g, const float* s, int ex,
                                           u4& a1, u4& a2) {
  // padding codewords (k >= K) have g = 0 and s = 0 in the LDS copy, so only
  // their bias slot needs a separate value
  _Float16 hi[8], lo[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float a = ldexpf(-2.f * g * s[j], SA - ex);
    hi[j] = (_Float16)a;
    lo[j] = (_Float16)(a - (float)hi[j]);
  }
  const float gs = ldexpf(g, -ex);
  const float gg = ldexpf(gs * gs, SA);
  _Float16 bias[8];
  bias_codeword_h(real, gg, bias);
  a1 = pack_h8(h ? lo : hi);
  a2 = pack_h8(h ? bias : hi);
}

// Build this lane's tiles from an LDS codebook (gains [KMAX], shapes
// [KMAX][DP], zero padded); unit_gain treats every real gain as 1.
__device__ __forceinline__ void build_tiles(Tiles& tl, const float* cbg, const float* cbs, int K,
                                            int ex, bool unit_gain, int lane) {
  const int c = lane & 31, h = lane >> 5;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int k = t * CW + c;
    const bool real = k < K;
    tile_entry(h, real, unit_gain ? 1.f : cbg[k], cbs + k * DP, ex, tl.a1[t], tl.a2[t]);
  }
}

// Row-side operands of one row (this lane's row).
// F16ROWS: the row is exactly float16 (raw16), so it enters the contraction
// as is (rho = 1, no lo part):
//   b1 = x,  b2: h0 0, h1 [sigma sigma hi(rr) lo(rr) 0 0 0 0],
//   rr = ||x||^2 / sigma, giving D = 2^SA dist / sigma.
// Otherwise (float32 rows x, zero padded) rho = 2^er >= max|x| and
//   b = x 2^SB / rho, b1 = hi(b),
//   b2: h0 lo(b), h1 [2^SB sigma/rho (twice) hi(rr) lo(rr) 0 0 0 0],
//   rr = 2^SB ||x||^2 / (sigma rho), giving D = 2^(SA+SB) dist / (sigma rho).
// In both cases D <= 2^(SA+1) rr means dist <= 2 ||x||^2.  need_exact flags
// rows whose operands leave the float16 range.
template <bool F16ROWS>
__device__ __forceinline__ void make_b(const float (&x)[8], u4 raw16, int ex, int h, h8& b1,
                                       h8& b2, float& rr, bool& need_exact, float& ss) {
  int sr;
  if (F16ROWS) {
    // ||x||^2 from packed float16 dot products (exact products, float32 sums)
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    ss = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // copy the element first: a bit_cast of a vector element reads the
      // wrong element with this compiler
      const uint32_t wj = raw16[j];
      const h2 v = __builtin_bit_cast(h2, wj);
      ss = __builtin_amdgcn_fdot2(v, v, ss, false);
    }
    sr = ex;
    rr = ldexpf(ss, -ex);
    need_exact = ex > 15 || ex < -14 || !(rr < 32768.f);
  } else {
    float mx = 0.f;
    ss = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) { mx = fmaxf(mx, fabsf(x[j])); ss = fmaf(x[j], x[j], ss); }
    int er = 0;
    frexpf(mx, &er);
    // a row far below the codebook's scale is scaled relative to sigma
    // instead (keeps 2^sr in float16 range; b and rr shrink with it, D stays
    // a positive multiple of the distance); rows so small that b would
    // leave float16's normal range are re-scored exactly
    const int er_min = ex + SB - 15;
    const bool tiny = er < er_min - 12;
    er = er > er_min ? er : er_min;
    sr = ex - er + SB;
    rr = ldexpf(ss, SB - ex - er);
    need_exact = tiny || !(mx > 0.f) || sr < -14 || !(rr < 32768.f);
    _Float16 hi[8], lo[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float v = ldexpf(x[j], SB - er);
      hi[j] = (_Float16)v;
      lo[j] = (_Float16)(v - (float)hi[j]);
    }
    b1 = as_h8(pack_h8(hi));
    raw16 = pack_h8(lo);
  }
  rr = fminf(rr, 32768.f);
  sr = sr < -14 ? -14 : (sr > 15 ? 15 : sr);
  const u4 bias = bias_row(sr, rr);
  if (F16ROWS) {
    b1 = as_h8(raw16);
    b2 = as_h8(h ? bias : (u4){0u, 0u, 0u, 0u});
  } else {
    b2 = as_h8(h ? bias : raw16);   // raw16 holds lo(b) here
  }
}

// Minimum packed key of one tile: the low KEY_BITS bits of each distance
// are replaced by the slot j (an inline constant), the 16 keys reduced with
// v_min3, and the tile number OR'd in once (all keys of a tile share it, so
// the order is unchanged).
__device__ __forceinline__ int tile_min(const f16v& c, int t) {
  constexpr int MASK = ~((1 << KEY_BITS) - 1);
  int m = min3i((__float_as_int(c[0]) & MASK) | 0, (__float_as_int(c[1]) & MASK) | 1,
                (__float_as_int(c[2]) & MASK) | 2);
#pragma unroll
  for (int j = 3; j < 15; j += 2)
    m = min3i(m, (__float_as_int(c[j]) & MASK) | j, (__float_as_int(c[j + 1]) & MASK) | (j + 1));
  m = min(m, (__float_as_int(c[15]) & MASK) | 15);
  return m | (t << 4);
}

// All NT tiles -> the lane's minimum packed key over its 128 codewords.
// Lane l holds distances of codewords 32 t + 8 (j / 4) + 4 h + j % 4 of
// row l % 32.  The two k-chunks of a tile accumulate in place; the MFMA
// latency is hidden by the other waves on the SIMD.
__device__ __forceinline__ int min_key(const Tiles& tl, h8 b1, h8 b2) {
  const f16v zero = {};
  int best = 0x7fffffff;
#pragma unroll
  for (int t = 0; t < NT; t += 2) {
    f16v c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(tl.a1[t]), b1, zero, 0, 0, 0);
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(tl.a2[t]), b2, c0, 0, 0, 0);
    const int m0 = tile_min(c0, t);
    f16v c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(tl.a1[t + 1]), b1, zero, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(tl.a2[t + 1]), b2, c1, 0, 0, 0);
    best = min3i(best, m0, tile_min(c1, t + 1));
  }
  return best;
}

// Combine the two lane halves of each row: smallest distance key, ties to
// the lowest codeword index.  Returns the codeword; dhat = approximate
// scaled distance of the winner.
__device__ __forceinline__ int reduce_rows(int key, int h, float& dhat) {
  const int idx = key & ((1 << KEY_BITS) - 1);
  const int t = idx >> 4, j = idx & 15;
  const int kidx = t * CW + (j >> 2) * 8 + h * 4 + (j & 3);
  const int hi = key >> KEY_BITS;
  const auto sh = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  const auto sk = __builtin_amdgcn_permlane32_swap(kidx, kidx, false, false);
  // both halves see (own, partner) in some order and choose identically
  const long long v0 = (long long)(int)sh[0] * 4294967296ll + (long long)(unsigned)sk[0];
  const long long v1 = (long long)(int)sh[1] * 4294967296ll + (long long)(unsigned)sk[1];
  const long long v = v0 < v1 ? v0 : v1;
  dhat = __int_as_float((int)(v >> 32) << KEY_BITS);
  return (int)(v & 0xffffffffll);
}

// Exact float64 argmin of eq. (5) over all K codewords for the rows flagged
// in `mask` (bit i = row i of the block, lanes 0..31).  gain / shape: this codebook,
// [K] / [K][ld] with d used elements per row (any memory).  Every lane of
// the wave takes part; both lanes of a flagged row receive its codeword.
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
      // eq. (5) up to the row constant ||x||^2: g^2 - 2 g s.x
      const double g = unit_gain ? 1.0 : (double)gain[k];
      double dot = 0.0;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < d) dot = fma(xr[j], (double)shape[(size_t)k * ld + j], dot);
      const double dist = fma(-2.0 * g, dot, g * g);
      if (dist < bd) { bd = dist; bk = k; }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const double od = __shfl_xor(bd, off);
      const int ok = __shfl_xor(bk, off);
      if (od < bd || (od == bd && ok < bk)) { bd = od; bk = ok; }
    }
    if ((lane & 31) == L) kstar = bk;
  }
}

// exact_rows for a codebook in global memory ([K] gains, [K][d] shapes),
// in two parts: load() fetches this lane's codewords k = lane + 64 j, all in
// flight together (one memory round trip; the loop form pays one per
// codeword and per row), and rows() scores the flagged rows with
// exact_rows' arithmetic, order and tie rule.
struct ExactCodebook {
  static constexpr int KJ = KMAX / 64;
  float cg[KJ], cs[KJ][8];
  // D8: d == 8 with a 16-byte aligned shape array (two 16-byte loads per
  // codeword)
  template <bool D8>
  __device__ __forceinline__ void load(const float* gain, const float* shape, int d, int K) {
    const int lane = wave_lane();
#pragma unroll
    for (int j = 0; j < KJ; ++j) {
      const int k = lane + 64 * j;
      const int kc = k < K ? k : K - 1;
      cg[j] = gain[kc];
      if (D8) {
        const float4* p4 = (const float4*)(shape + (size_t)kc * 8);
        const float4 u = p4[0], v = p4[1];
        cs[j][0] = u.x; cs[j][1] = u.y; cs[j][2] = u.z; cs[j][3] = u.w;
        cs[j][4] = v.x; cs[j][5] = v.y; cs[j][6] = v.z; cs[j][7] = v.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) cs[j][e] = shape[(size_t)kc * d + (e < d ? e : 0)];
      }
    }
  }
  __device__ __forceinline__ void rows(unsigned long long mask, const float (&x)[8], int d, int K,
                                       int& kstar) const {
    const int lane = wave_lane();
    while (mask) {
      const int L = __ffsll((long long)mask) - 1;
      mask &= mask - 1;
      double xr[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) xr[e] = (double)__shfl(x[e], L);
      double bd = INFINITY;
      int bk = 0x7fffffff;
#pragma unroll
      for (int j = 0; j < KJ; ++j) {
        const int k = lane + 64 * j;
        if (k < K) {
          const double g = (double)cg[j];
          double dot = 0.0;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e < d) dot = fma(xr[e], (double)cs[j][e], dot);
          const double dist = fma(-2.0 * g, dot, g * g);
          if (dist < bd) { bd = dist; bk = k; }
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const double od = __shfl_xor(bd, off);
        const int ok = __shfl_xor(bk, off);
        if (od < bd || (od == bd && ok < bk)) { bd = od; bk = ok; }
      }
      if ((lane & 31) == L) kstar = bk;
    }
  }
};

// Eight subvector elements of one row in their storage type, kept packed in
// registers between a prefetch and their use.
template <typename T> struct RowVec;
template <> struct RowVec<_Float16> {
  u4 v;
  __device__ __forceinline__ void load(const _Float16* p) { v = *(const u4*)p; }
  __device__ __forceinline__ void zero() { v = (u4){0u, 0u, 0u, 0u}; }
  __device__ __forceinline__ void get(float (&x)[8]) const {
    const h8 hv = as_h8(v);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)hv[j];
  }
  __device__ __forceinline__ u4 raw16() const { return v; }
};
template <> struct RowVec<float> {
  u4 v0, v1;
  __device__ __forceinline__ void load(const float* p) {
    v0 = ((const u4*)p)[0];
    v1 = ((const u4*)p)[1];
  }
  __device__ __forceinline__ void zero() { v0 = v1 = (u4){0u, 0u, 0u, 0u}; }
  __device__ __forceinline__ void get(float (&x)[8]) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = __uint_as_float(v0[j]);
      x[4 + j] = __uint_as_float(v1[j]);
    }
  }
  __device__ __forceinline__ u4 raw16() const { return (u4){0u, 0u, 0u, 0u}; }
};

// One codeword (gain, shape padded to DP) read without branches: indices
// are clamped to valid entries and the padding is applied to the values.
__device__ __forceinline__ void read_codeword(const float* gain, const float* shape, int d, int K,
                                              int k, bool unit_gain, float& g, float (&sv)[DP]) {
  const int kk = k < K ? k : K - 1;
  const bool real = k < K;
  const float gr = unit_gain ? 1.f : gain[kk];
  g = real ? gr : 0.f;
  const float* sp = shape + (size_t)kk * d;
  if (d == DP && (((uintptr_t)sp) & 15) == 0) {
    const f4 lo4 = ((const f4*)sp)[0], hi4 = ((const f4*)sp)[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sv[j] = real ? lo4[j] : 0.f;
      sv[4 + j] = real ? hi4[j] : 0.f;
    }
  } else {
#pragma unroll
    for (int j = 0; j < DP; ++j) {
      const float v = sp[j < d ? j : 0];
      sv[j] = (real && j < d) ? v : 0.f;
    }
  }
}

// Load a codebook (gain [K], shape [K][d]) into zero-padded LDS arrays and
// return sigma's exponent (every thread of the block calls this).
// The maximum of v over the workgroup into *red (LDS, cleared beforehand):
// a wave reduction, then one atomic per wave.  Every thread calls it.
__device__ __forceinline__ void block_max_into(int v, int* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, __shfl_xor(v, off));
  if ((threadIdx.x & 63) == 0 && v > 0) atomicMax(red, v);
}

__device__ int load_codebook(const float* gain, const float* shape, int d, int K, bool unit_gain,
                             float* cbg, float* cbs, int* red) {
  const int tid = threadIdx.x;
  if (tid == 0) *red = 0;
  __syncthreads();
  int gm = 0;   // gains >= 0 order as ints
  for (int k = tid; k < KMAX; k += blockDim.x) {
    float g, sv[DP];
    read_codeword(gain, shape, d, K, k, unit_gain, g, sv);
    cbg[k] = g;
#pragma unroll
    for (int j = 0; j < DP; ++j) cbs[k * DP + j] = sv[j];
    if (g > 0.f) gm = max(gm, __float_as_int(g));
  }
  block_max_into(gm, red);
  __syncthreads();
  return sigma_exp(__int_as_float(*red));
}

// ---------------------------------------------------------------- kernels

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
// K-means seeding (kmeans != 0): the centroid is the seed row itself, held
// as gain ||x_r|| and shape x_r / ||x_r|| (0 for a zero row).
template <typename T>
__global__ void seed_kernel(const T* __restrict__ Xt, int64_t N, int d, int K,
                            const int32_t* __restrict__ seeds, float* __restrict__ shape,
                            float* __restrict__ seednorm, int kmeans, float* __restrict__ gain) {
  const int g = blockIdx.x;
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    const int64_t row = seeds[(size_t)g * K + k];
    const T* x = Xt + ((int64_t)g * N + row) * 8;
    double ss = 0.0;
    for (int j = 0; j < d; ++j) { const double v = to_f(x[j]); ss = fma(v, v, ss); }
    const double nrm = sqrt(ss);
    const double den = kmeans ? (nrm > 0.0 ? nrm : 1.0) : nrm + (double)Y_EPS;
    for (int j = 0; j < d; ++j)
      shape[((size_t)g * K + k) * d + j] = (float)((double)to_f(x[j]) / den);
    seednorm[(size_t)g * K + k] = (float)nrm;
    if (kmeans) gain[(size_t)g * K + k] = (float)nrm;
  }
}

// Operand tiles for ncb codebooks into a table (used by multi-stage encode).
// Header of a prepared codebook (gsrq_encode_prepare): magic, M, G, d, K,
// then zeros, and the complement of the magic in the last word.
constexpr uint32_t PREP_MAGIC = 0x50525147u;
constexpr int PREP_WORDS = 16;
struct PrepTag {
  uint32_t w[PREP_WORDS];
};

__host__ __device__ inline PrepTag prep_tag(int M, int G, int d, int K) {
  PrepTag t = {};
  t.w[0] = PREP_MAGIC;
  t.w[1] = (uint32_t)M;
  t.w[2] = (uint32_t)G;
  t.w[3] = (uint32_t)d;
  t.w[4] = (uint32_t)K;
  t.w[PREP_WORDS - 1] = ~PREP_MAGIC;
  return t;
}

__global__ void __launch_bounds__(64) tiles_kernel(const float* __restrict__ gain,
                                                   const float* __restrict__ shape, int d, int K,
                                                   u4* __restrict__ frag, int* __restrict__ sig,
                                                   uint32_t* __restrict__ tagp, PrepTag tag) {
  if (tagp && blockIdx.x == 0 && threadIdx.x < PREP_WORDS) tagp[threadIdx.x] = tag.w[threadIdx.x];
  __shared__ float cbg[KMAX];
  __shared__ float cbs[KMAX * DP];
  __shared__ int red;
  const int cb = blockIdx.x;
  const int ex = load_codebook(gain + (size_t)cb * K, shape + (size_t)cb * K * d, d, K, false,
                               cbg, cbs, &red);
  Tiles tl;
  build_tiles(tl, cbg, cbs, K, ex, false, threadIdx.x);
  u4* fr = frag + (size_t)cb * NT * 2 * 64;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    fr[(t * 2 + 0) * 64 + threadIdx.x] = tl.a1[t];
    fr[(t * 2 + 1) * 64 + threadIdx.x] = tl.a2[t];
  }
  if (threadIdx.x == 0) sig[cb] = ex;
}

struct AssignArgs {
  const void* xt;        // [G][N][8]
  int64_t N;
  int d, K, G;
  const float* w;        // [N] or null
  const float* gain;     // [G][K] codebook to score with (no fused update)
  const float* shape;    // [G][K][d]
  // codebook update at the start of an assignment launch (upd != UPD_NONE)
  // and in the update kernel: C_{t-1} is computed from the previous pass's
  // partial sums and the codebook before it (old_*), written to new_* by
  // the subspace's first chunk; the update kernel writes fin_* (the
  // caller's arrays) and, for subspaces that stopped inside a fused update,
  // copies their final codebook there from buf_*[iteration % 2]
  int upd;
  int upd_has_wxx;       // the previous pass accumulated sum w ||x||^2
  const float* old_gain;
  const float* old_shape;
  float* new_gain;
  float* new_shape;
  float* fin_gain;
  float* fin_shape;
  const float* buf_gain[2];
  const float* buf_shape[2];
  int copy_done;
  uint16_t* assign;      // [G][N]
  int* done;             // [G] iteration at which the subspace stopped, 0 = running
  int* iters;            // [G] iterations run
  double* part;          // [G][chunks][PSTRIDE]
  const float* seednorm; // [G][K] seed row norms (initial gains)
  double* trace;         // [G][T] objective per iteration, or null
  double* wxx;           // [G] sum_i w_i ||x_i||^2 (constant over the iterations)
  int want_wxx;          // this launch accumulates wxx (first pass that needs it)
  int chunks;
  int chunk_rows;        // rows per chunk (a multiple of RB)
  int force_changed;
  int t;                 // iteration number (1-based); 0 for the initialisation
  int T;
  int no_early_stop;
  int kmeans;            // K-means baseline update instead of eqs. (7)(8)
};

// Codebook update of subspace g from the partial sums of all its chunks,
// reduced in chunk order (every workgroup that computes it gets the same
// result).  Initialisation: eq. (8) gains of the seed shapes.  Iteration:
// eqs. (7) and (8), plus the weighted objective of the assignment just made,
// from the sufficient statistics of the codebook it was made with:
//   sum_i w_i ||x_i - g s||^2 = sum_i w_i ||x_i||^2
//                               - sum_k (2 g_k s_k . S_k - g_k^2 ||s_k||^2 W_k),
// S_k = sum of w x over the members of k, W_k = their weight (products and
// sums in float64, so the cancellation costs no accuracy); and the stop
// test (no assignment changed).  K-means baseline: the centroid becomes
// S_k / W_k (held as its norm and direction) and the objective is the
// distortion after the update, sum_i w_i ||x_i||^2 - sum_k ||S_k||^2 / W_k.

// Element-wise chunk sums of subspace g (coalesced, in chunk order) into
// sums[0, K ACC) and sums[KMAX ACC + {0, 1}] (sum w ||x||^2, changed flag);
// loads are unconditional (clamped indices, masked values) so a batch of
// chunks is in flight at once.
constexpr int UPD_CBATCH = 4;                                             // chunks per load batch
template <int NT>
__device__ __forceinline__ void sum_partials(const AssignArgs& a, int g, double* sums) {
  constexpr int EPT = (KMAX * ACC + 2 + NT - 1) / NT;
  const int tid = threadIdx.x, K = a.K;
  const double* pg = a.part + (size_t)g * a.chunks * PSTRIDE;
  const int nsum = K * ACC + 2;
  double v[EPT];
#pragma unroll
  for (int u = 0; u < EPT; ++u) v[u] = 0.0;
  for (int c0 = 0; c0 < a.chunks; c0 += UPD_CBATCH) {
    double pv[UPD_CBATCH][EPT];
#pragma unroll
    for (int cc = 0; cc < UPD_CBATCH; ++cc)
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = tid + u * NT;
        const int src = e < K * ACC ? e : KMAX * ACC + (e < nsum ? e - K * ACC : 0);
        const int c = c0 + cc < a.chunks ? c0 + cc : 0;
        pv[cc][u] = pg[(size_t)c * PSTRIDE + src];
      }
#pragma unroll
    for (int cc = 0; cc < UPD_CBATCH; ++cc)
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = tid + u * NT;
        const double x = c0 + cc < a.chunks ? pv[cc][u] : 0.0;
        v[u] = e == nsum - 1 ? fmax(v[u], x) : v[u] + x;
      }
  }
#pragma unroll
  for (int u = 0; u < EPT; ++u) {
    const int e = tid + u * NT;
    if (e < nsum) sums[e < K * ACC ? e : KMAX * ACC + (e - K * ACC)] = v[u];
  }
}

// Update of one codeword from its ACC sums s (w y[8], w x[8], W, count) and
// its previous gain / shape (float64, padded with zeros past d); returns its
// term of the objective (iteration) and leaves the new codeword in gnew, sn.
__device__ __forceinline__ double update_codeword(bool init, bool kmeans, const double* s,
                                                  double& gnew, double (&sn)[DP]) {
  double term = 0.0;
  const double W = s[16];
  if (!init && kmeans) {
    if (W > 0.0) {
      double c[DP], cn = 0.0, s2 = 0.0;
      // one float64 division per quotient vector, then products (within
      // an ulp of dividing every element)
      const double iw = 1.0 / W;
#pragma unroll
      for (int j = 0; j < DP; ++j) {
        c[j] = s[8 + j] * iw;
        cn = fma(c[j], c[j], cn);
        s2 = fma(s[8 + j], s[8 + j], s2);
      }
      term += s2 * iw;
      cn = sqrt(cn);
      const double icn = cn > 0.0 ? 1.0 / cn : 0.0;
#pragma unroll
      for (int j = 0; j < DP; ++j) sn[j] = c[j] * icn;
      gnew = cn;
    }
    return term;
  }
  if (!init) {
    // the stored shapes are unit only to float32 rounding: use ||s||^2
    double ps = 0.0, s2 = 0.0;
#pragma unroll
    for (int j = 0; j < DP; ++j) {
      ps = fma(s[8 + j], sn[j], ps);
      s2 = fma(sn[j], sn[j], s2);
    }
    term += gnew * (2.0 * ps - gnew * s2 * W);
  }
  if (W > 0.0) {
    if (!init) {
      double mn = 0.0;
#pragma unroll
      for (int j = 0; j < DP; ++j) mn = fma(s[j], s[j], mn);
      mn = sqrt(mn);
      if (mn > SHAPE_KEEP_REL * W) {
        const double imn = 1.0 / mn;
#pragma unroll
        for (int j = 0; j < DP; ++j) sn[j] = s[j] * imn;
      }
    }
    double pr = 0.0;
#pragma unroll
    for (int j = 0; j < DP; ++j) pr = fma(s[8 + j], sn[j], pr);
    gnew = fmax(0.0, pr / W);
  }
  return term;
}

// Sum of v over the workgroup (NT threads, per-wave partials in wred).
template <int NT>
__device__ __forceinline__ double block_sum(double v, double* wred) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if (lane == 0) wred[wave] = v;
  __syncthreads();
  double sum = 0.0;
  for (int w = 0; w < NT / 64; ++w) sum += wred[w];
  return sum;
}

// The objective entry, iteration count and stop flag of iteration t (one
// thread): returns whether the subspace stops.
__device__ __forceinline__ bool finish_iteration(const AssignArgs& a, int g, int t, double wxx,
                                                 double terms, double changed) {
  if (a.trace) a.trace[(size_t)g * a.T + (t - 1)] = wxx - terms;
  a.iters[g] = t;
  const bool stop = changed == 0.0 && !a.no_early_stop;
  if (stop) a.done[g] = t;
  return stop;
}

constexpr int UPD_THREADS = 1024;
static_assert(KMAX <= UPD_THREADS, "one thread per codeword");
// Standalone update: initialisation (T = 0) or the last iteration's update,
// old codebook from old_*, result to fin_* (the caller's arrays, possibly
// the same arrays: each thread reads its codeword before writing it).
template <int MODE>
__global__ void __launch_bounds__(UPD_THREADS) update_kernel(AssignArgs a) {
  __shared__ double sums[KMAX * ACC + 2];
  __shared__ double wred[UPD_THREADS / 64];
  const int g = blockIdx.x;
  const int tid = threadIdx.x;
  const int d = a.d, K = a.K;
  const int stopped = MODE == MODE_ITER ? a.done[g] : 0;
  const int kmine = tid < K ? tid : 0;
  if (stopped) {
    // stopped inside a fused update: its final codebook is in buf_*
    if (a.copy_done && tid < K) {
      const float* gs = a.buf_gain[stopped & 1] + (size_t)g * K + tid;
      const float* ss = a.buf_shape[stopped & 1] + ((size_t)g * K + tid) * d;
      a.fin_gain[(size_t)g * K + tid] = *gs;
      for (int j = 0; j < d; ++j) a.fin_shape[((size_t)g * K + tid) * d + j] = ss[j];
    }
    return;
  }
  const float* so = a.old_shape + ((size_t)g * K + kmine) * d;
  float sold[DP];
#pragma unroll
  for (int j = 0; j < DP; ++j) sold[j] = so[j < d ? j : 0];
  const float gold = MODE == MODE_INIT ? a.seednorm[(size_t)g * K + kmine]
                                       : a.old_gain[(size_t)g * K + kmine];
  sum_partials<UPD_THREADS>(a, g, sums);
  __syncthreads();
  double term = 0.0;
  if (tid < K) {
    double sn[DP];
#pragma unroll
    for (int j = 0; j < DP; ++j) sn[j] = (j < d) ? (double)sold[j] : 0.0;
    double gnew = (double)gold;
    term = update_codeword(MODE == MODE_INIT, a.kmeans != 0, sums + tid * ACC, gnew, sn);
    float* sk = a.fin_shape + ((size_t)g * K + tid) * d;
#pragma unroll
    for (int j = 0; j < DP; ++j)
      if (j < d) sk[j] = (float)sn[j];
    a.fin_gain[(size_t)g * K + tid] = (float)gnew;
  }
  if (MODE == MODE_INIT) {
    if (tid == 0 && a.want_wxx) a.wxx[g] = sums[KMAX * ACC];
  } else {
    const double terms = block_sum<UPD_THREADS>(term, wred);
    if (tid == 0) {
      if (a.upd_has_wxx) a.wxx[g] = sums[KMAX * ACC];
      finish_iteration(a, g, a.t, a.wxx[g], terms, sums[KMAX * ACC + 1]);
    }
  }
}

// Fused assignment (eq. 5) + weighted accumulation (eqs. 6-8) for one
// (chunk of rows, subspace).  MODE_INIT scores with unit gains (largest
// projection) for the gain initialisation.  Each wave walks 32-row blocks
// and prefetches the next block's rows, weights and previous codes while
// scoring the current one.
template <typename T, int MODE>
__global__ void __launch_bounds__(TRAIN_WAVES * 64, WAVES_PER_SIMD)
assign_accumulate_kernel(AssignArgs a) {
  constexpr bool F16ROWS = sizeof(T) == 2;
  __shared__ double acc[KMAX * ACC_LDS];
  __shared__ float cbg[KMAX];
  __shared__ float cbs[KMAX * DP];
  __shared__ u4 tiles_l[NT * 2 * 64];
  __shared__ double objw[TRAIN_WAVES];
  __shared__ uint16_t codes_l[TRAIN_CHUNK_MAX];   // this chunk's new assignment
  __shared__ int changed, red, next_blk;

  const int g = blockIdx.y;
  const int chunk = blockIdx.x;
  // a stopped subspace returns; the test waits until this launch's first
  // loads are in flight, so their latency overlaps that of the flag
  const int stopped = a.done[g];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = lane & 31, h = lane >> 5;
  const int d = a.d, K = a.K;

  // this chunk's rows, weights and codes, indexed from 0 in 32 bits
  const int64_t row_begin = (int64_t)chunk * a.chunk_rows;
  const int nrows = (int)(a.N - row_begin < a.chunk_rows ? a.N - row_begin : a.chunk_rows);
  const T* xc = (const T*)a.xt + ((size_t)g * a.N + row_begin) * 8;
  uint16_t* ac = a.assign + (size_t)g * a.N + row_begin;
  const int nblk = (nrows + RB - 1) / RB;
  const bool want_wxx = a.want_wxx != 0;

  // loads never branch: past the end they read the chunk's first row, whose
  // results are discarded, so prefetches stay in flight (without weights
  // the load reads a gain in place of a weight and the value is replaced by
  // 1: a global pointer keeps it a global load)
  const bool has_w = a.w != nullptr;
  const float* wc = has_w ? a.w + row_begin : a.gain;
  const int wstride = has_w ? 1 : 0;
  RowVec<T> nx;
  float nw = 0.f;
  uint16_t nold = 0;
  auto fetch = [&](int rb) {
    // unsigned 32-bit offsets from the chunk's uniform bases (no 64-bit
    // address arithmetic per lane)
    const uint32_t r0 = (uint32_t)(rb * RB + i);
    const uint32_t r = r0 < (uint32_t)nrows ? r0 : 0u;
    nx.load(xc + r * 8u);
    nw = wc[r * (uint32_t)wstride];
    if (MODE == MODE_ITER) nold = ac[r];
  };
  // the first block's loads are issued before the codebook is ready, so
  // they overlap its load or update
  if (wave < nblk) fetch(wave);

  int ex;
  if (MODE == MODE_ITER && a.upd != UPD_NONE) {
    // the previous pass's codebook update, computed here by every workgroup
    // of the subspace (same sums, same order, same result) straight into
    // LDS; the first chunk's workgroup stores it and records the iteration
    const bool init = a.upd == UPD_INIT;
    const int kmine = tid < K ? tid : 0;
    const float* so = a.old_shape + ((size_t)g * K + kmine) * d;
    float sold[DP];
#pragma unroll
    for (int j = 0; j < DP; ++j) sold[j] = so[j < d ? j : 0];
    const float gold = init ? a.seednorm[(size_t)g * K + kmine] : a.old_gain[(size_t)g * K + kmine];
    sum_partials<TRAIN_WAVES * 64>(a, g, acc);   // acc holds the dense sums for now
    if (stopped) return;   // uniform over the workgroup
    if (tid == 0) red = 0;
    __syncthreads();
    double term = 0.0;
    int gm = 0;
    if (tid < KMAX) {
      const bool real = tid < K;
      double sn[DP];
#pragma unroll
      for (int j = 0; j < DP; ++j) sn[j] = (real && j < d) ? (double)sold[j] : 0.0;
      double gnew = real ? (double)gold : 0.0;
      if (real) term = update_codeword(init, a.kmeans != 0, acc + tid * ACC, gnew, sn);
      cbg[tid] = (float)gnew;
#pragma unroll
      for (int j = 0; j < DP; ++j) cbs[tid * DP + j] = (float)sn[j];
      if ((float)gnew > 0.f) gm = __float_as_int((float)gnew);
      if (chunk == 0 && real) {
        a.new_gain[(size_t)g * K + tid] = (float)gnew;
        for (int j = 0; j < d; ++j) a.new_shape[((size_t)g * K + tid) * d + j] = (float)sn[j];
      }
    }
    block_max_into(gm, &red);
    const double wxx_p = acc[KMAX * ACC], chg = acc[KMAX * ACC + 1];
    const double terms = block_sum<TRAIN_WAVES * 64>(term, objw);
    if (chunk == 0 && tid == 0) {
      if (a.upd_has_wxx) a.wxx[g] = wxx_p;
      if (!init) finish_iteration(a, g, a.t - 1, a.upd_has_wxx ? wxx_p : a.wxx[g], terms, chg);
    }
    // a subspace whose previous assignment repeated stops here (uniform)
    if (!init && chg == 0.0 && !a.no_early_stop) return;
    __syncthreads();
    ex = sigma_exp(__int_as_float(red));
  } else {
    if (stopped) return;   // uniform over the workgroup
    ex = load_codebook(a.gain + (size_t)g * K, a.shape + (size_t)g * K * d, d, K,
                       MODE == MODE_INIT, cbg, cbs, &red);
  }
  for (int e = tid; e < KMAX * ACC_LDS; e += blockDim.x) acc[e] = 0.0;
  if (tid == 0) {
    changed = a.force_changed;
    next_blk = TRAIN_WAVES;   // wave w starts with block w
  }
  // operand tiles built once per workgroup (one (tile, lane) entry per
  // thread), then read by every wave into its registers
  for (int e = tid; e < NT * 64; e += blockDim.x) {
    const int t = e >> 6, l = e & 63;
    const int k = t * CW + (l & 31);
    u4 a1, a2;
    tile_entry(l >> 5, k < K, MODE == MODE_INIT ? 1.f : cbg[k], cbs + k * DP, ex, a1, a2);
    tiles_l[(2 * t) * 64 + l] = a1;
    tiles_l[(2 * t + 1) * 64 + l] = a2;
  }
  __syncthreads();
  Tiles tl;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    tl.a1[t] = tiles_l[(2 * t) * 64 + lane];
    tl.a2[t] = tiles_l[(2 * t + 1) * 64 + lane];
  }
  // the tile loads complete here, once: left pending into the loop, they
  // made the compiler wait for every LDS operation in flight (this wave's
  // float64 accumulations of the previous block) before each block's MFMAs
  lgkm_wait_all();

  double obj = 0.0;
  bool any_changed = false;
  // Blocks are handed out one at a time from an LDS counter, claimed one
  // block ahead so their rows can be prefetched.  A static round-robin split
  // left the youngest wave of each SIMD running alone for the last third of
  // the launch (the oldest wave issues first and finishes first); claimed
  // blocks keep all waves of a SIMD busy until the chunk is done.
  auto claim = [&]() {
    int v = 0;
    if (lane == 0) v = atomicAdd(&next_blk, 1);
    return __builtin_amdgcn_readfirstlane(v);
  };
  int rb_next = wave < nblk ? claim() : nblk;
  for (int rb = wave; rb < nblk;) {
    const int r = rb * RB + i;
    const bool valid = r < nrows;
    float x[8];
    nx.get(x);
    const u4 raw = nx.raw16();
    const float wcur = has_w ? nw : 1.f;
    const uint16_t old = nold;
    if (rb_next < nblk) fetch(rb_next);
    const int rb_after = rb_next < nblk ? claim() : nblk;

    h8 b1, b2;
    float rr, ss;
    bool need_exact;
    make_b<F16ROWS>(x, raw, ex, h, b1, b2, rr, need_exact, ss);
    const int key = min_key(tl, b1, b2);
    float dhat;
    int kstar = reduce_rows(key, h, dhat);
    need_exact = need_exact || !(dhat <= ldexpf(rr, SA + 1)) || kstar >= K;
    const unsigned long long fb = __ballot(valid && need_exact && h == 0);
    if (fb) {
      exact_rows(fb, x, d, DP, K, cbg, cbs, MODE == MODE_INIT, kstar);
      // the rare path's LDS reads end here, so the common path's
      // accumulations below are not held up waiting for them
      lgkm_wait_all();
    }
    if (kstar >= K) kstar = K - 1;   // only discarded rows can get here
    if (valid) {
      // lane half 0 adds w y (y = x / ||x||) and W, half 1 adds w x and the
      // member count
      double* ak = acc + kstar * ACC_LDS;
      const float inv = __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(ss) + Y_EPS);
      const float sc = h ? wcur : wcur * inv;
      // float64 products: exact for half 1, whose w x sums also give the
      // objective
#pragma unroll
      for (int j = 0; j < 8; ++j) unsafeAtomicAdd(ak + 8 * h + j, (double)x[j] * (double)sc);
      unsafeAtomicAdd(ak + 16 + h, h ? 1.0 : (double)wcur);
      if (h == 0) {
        if (want_wxx) {
          double s2 = 0.0;
#pragma unroll
          for (int j = 0; j < 8; ++j) s2 = fma((double)x[j], (double)x[j], s2);
          obj = fma((double)wcur, s2, obj);
        }
        if (MODE == MODE_ITER && old != (uint16_t)kstar) any_changed = true;
        // global stores would share vmcnt with the prefetch and stall the
        // next block, so codes go to LDS and leave in one pass at the end
        codes_l[r] = (uint16_t)kstar;
      }
    }
    rb = rb_next;
    rb_next = rb_after;
  }
  // wave sums of the objective and changed flag
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) obj += __shfl_xor(obj, off);
  if (lane == 0) objw[wave] = obj;
  if (__ballot(any_changed) && lane == 0) atomicOr(&changed, 1);
  __syncthreads();
  for (int r = tid; r < nrows; r += blockDim.x) ac[r] = codes_l[r];
  double* out = a.part + ((size_t)g * a.chunks + chunk) * PSTRIDE;
  for (int e = tid; e < K * ACC; e += blockDim.x) out[e] = acc[(e / ACC) * ACC_LDS + e % ACC];
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < TRAIN_WAVES; ++w) s += objw[w];
    out[KMAX * ACC] = s;
    out[KMAX * ACC + 1] = (double)changed;
  }
}

struct EncodeArgs {
  const void* x;         // [N][ldx]
  int64_t ldx, N;
  int d, K, G, M, b, words;
  const float* gain;     // [M][G][K]
  const float* shape;    // [M][G][K][d]
  const u4* frag;        // [M*G][NT][2][64] (multi-stage only)
  const int* sig;        // [M*G]
  uint32_t* codes;       // [N][words] or null
  float* residual;       // [N][D] or null
  int byte_codes;        // b == 8: plain byte stores, else atomic OR
  int lds_codes;         // byte codes of 4 whole subspaces per block: LDS-staged
  int vec_rows;          // d == 8 and 16-byte aligned rows: vector loads
  const uint32_t* ptag;  // prepared codebook header to check, or null
  PrepTag etag;          // the header this call expects
  int64_t chunk_rows;    // rows per workgroup (a multiple of RB)
};

// A row's subvector from row-major X, loaded raw (prefetch) and widened
// later.  VEC: d == 8 with 16-byte aligned rows (vector loads); otherwise d
// scalar loads with clamped indices.  Neither form branches.
template <typename T, bool VEC> struct RowRaw {
  T v[8];
  __device__ __forceinline__ void load(const T* p, int d) {
    if (VEC) {
      if (sizeof(T) == 2) {
        *(u4*)v = *(const u4*)p;
      } else {
        ((u4*)v)[0] = ((const u4*)p)[0];
        ((u4*)v)[1] = ((const u4*)p)[1];
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = p[j < d ? j : 0];
    }
  }
  __device__ __forceinline__ void get(float (&x)[8], int d, bool valid) const {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (valid && (VEC || j < d)) ? (float)v[j] : 0.f;
  }
  __device__ __forceinline__ u4 raw16(const float (&x)[8], bool valid) const {
    // the exact float16 operand: the loaded bits when they are the whole
    // (valid, 8-wide) row, else rebuilt from the masked float copy
    if (VEC && sizeof(T) == 2) {
      const u4 r = *(const u4*)v;
      return valid ? r : (u4){0u, 0u, 0u, 0u};
    }
    _Float16 hv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) hv[j] = (_Float16)x[j];
    return pack_h8(hv);
  }
};

// Stage-fused encoder: a workgroup encodes a chunk of rows for ENC_SUBS
// consecutive subspaces, three waves per subspace; the residual of a 32-row
// block stays in registers through all M stages.  The waves of a subspace
// claim its blocks one at a time from an LDS counter, one block ahead (a
// static split left the youngest wave of each SIMD running alone at the
// end of every workgroup).  A single-stage launch keeps the subspaces'
// codebooks in LDS and each wave's operand tiles in registers for the whole
// launch; a multi-stage launch reloads each stage's tiles from a table.
template <typename T, bool MULTI, bool VEC>
__global__ void __launch_bounds__(ENC_WAVES * 64, WAVES_PER_SIMD) encode_kernel(EncodeArgs a) {
  constexpr bool F16IN = sizeof(T) == 2;
  __shared__ float cbl[MULTI ? 1 : ENC_SUBS * KMAX * (DP + 1)];
  // byte codes of this chunk, [stage][row][subspace]; written out at the end
  // so that no global store sits in the loop (stores share vmcnt with loads)
  __shared__ uint32_t codes_l[ENC_CODES_WORDS];
  __shared__ int next_blk[ENC_SUBS];
  const int lane = wave_lane(), wave = threadIdx.x >> 6;
  const int sg = wave % ENC_SUBS;   // this wave's subspace within the group
  const int g = blockIdx.y * ENC_SUBS + sg;
  const int i = lane & 31, h = lane >> 5;
  const int d = a.d, K = a.K, G = a.G;
  const bool gvalid = g < G;
  const int64_t row_begin = (int64_t)blockIdx.x * a.chunk_rows;
  const int64_t row_end = row_begin + a.chunk_rows < a.N ? row_begin + a.chunk_rows : a.N;
  const int nblk = (int)((row_end - row_begin + RB - 1) / RB);
  float* mg = cbl + (MULTI ? 0 : sg * KMAX * (DP + 1));   // gains [KMAX]
  float* ms = mg + KMAX;                                    // shapes [KMAX][DP]
  // waves sg, sg + ENC_SUBS, ... start with blocks 0, 1, ...
  if (threadIdx.x < ENC_SUBS) next_blk[threadIdx.x] = ENC_WAVES / ENC_SUBS;
  Tiles tl;
  int ex0 = 0;
  if (!MULTI) {
    // the group's codebooks into LDS (the first wave of each subspace);
    // sigma from the subspace's largest gain
    const int gc = gvalid ? g : 0;
    if (wave < ENC_SUBS) {
      for (int k = lane; k < KMAX; k += 64) {
        float gv, sv[DP];
        read_codeword(a.gain + (size_t)gc * K, a.shape + (size_t)gc * K * d, d, K, k, false, gv,
                      sv);
        mg[k] = gv;
#pragma unroll
        for (int j = 0; j < DP; ++j) ms[k * DP + j] = sv[j];
      }
    }
    __syncthreads();
    float m = 0.f;
    for (int k = lane; k < KMAX; k += 64) m = fmaxf(m, mg[k]);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    ex0 = sigma_exp(m);
    build_tiles(tl, mg, ms, K, ex0, false, lane);
  } else {
    __syncthreads();   // the block counters
  }
  const bool lds_codes = a.lds_codes != 0;
  if (MULTI && a.ptag) {
    // a prepared codebook whose header does not match this call: every code
    // field of the block's rows is set to all ones and the residual to NaN
    bool ok = true;
#pragma unroll
    for (int w = 0; w < PREP_WORDS; ++w) ok &= a.ptag[w] == a.etag.w[w];
    if (!ok) {
      if (gvalid && wave < ENC_SUBS && lane < 32) {
        for (int64_t row = row_begin + lane; row < row_end; row += 32) {
          if (a.codes) {
            for (int m = 0; m < a.M; ++m) {
              const int64_t bit = ((int64_t)m * G + g) * a.b;
              if (a.byte_codes) {
                ((uint8_t*)(a.codes + row * a.words))[bit / 8] = 0xffu;
              } else {   // words zeroed beforehand
                uint32_t* wp = a.codes + row * a.words + bit / 32;
                const int off = (int)(bit % 32);
                const uint32_t ones = (1u << a.b) - 1u;
                atomicOr(wp, ones << off);
                if (off + a.b > 32) atomicOr(wp + 1, ones >> (32 - off));
              }
            }
          }
          if (a.residual) {
            float* dst = a.residual + row * (int64_t)(G * d) + (int64_t)g * d;
            for (int j = 0; j < d; ++j) dst[j] = __builtin_nanf("");
          }
        }
      }
      return;   // uniform over the workgroup (every wave reads the same header)
    }
  }
  if (!gvalid) {
    // the flush at the end needs every wave at its barrier
    __syncthreads();
    goto flush;
  }
  {
  const T* X = (const T*)a.x;
  RowRaw<T, VEC> nx;
  auto fetch = [&](int rb) {
    int64_t row = row_begin + (int64_t)rb * RB + i;
    row = row < row_end ? row : row_begin;
    nx.load(X + row * a.ldx + (int64_t)g * d, d);
  };
  auto claim = [&]() {
    int v = 0;
    if (lane == 0) v = atomicAdd(&next_blk[sg], 1);
    return __builtin_amdgcn_readfirstlane(v);
  };
  int rb = wave / ENC_SUBS;
  if (rb < nblk) fetch(rb);
  // a single stage keeps its tables in registers for every row block
  if (MULTI && a.M == 1) {
    const u4* fr = a.frag + (size_t)g * NT * 2 * 64;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tl.a1[t] = fr[(t * 2 + 0) * 64 + lane];
      tl.a2[t] = fr[(t * 2 + 1) * 64 + lane];
    }
    ex0 = a.sig[g];
  }
  int rb_next = rb < nblk ? claim() : nblk;
  while (rb < nblk) {
    const int64_t r0 = row_begin + (int64_t)rb * RB;
    const int64_t row = r0 + i;
    const bool valid = row < row_end;
    float x[8];
    nx.get(x, d, valid);
    const u4 raw = nx.raw16(x, valid);
    if (rb_next < nblk) fetch(rb_next);
    const int rb_after = rb_next < nblk ? claim() : nblk;
    for (int m = 0; m < a.M; ++m) {
      const int cb = m * G + g;
      int ex = ex0;
      if (MULTI && a.M > 1) {
        const u4* fr = a.frag + (size_t)cb * NT * 2 * 64;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          tl.a1[t] = fr[(t * 2 + 0) * 64 + lane];
          tl.a2[t] = fr[(t * 2 + 1) * 64 + lane];
        }
        ex = a.sig[cb];
      }
      h8 b1, b2;
      float rr, ss;
      bool need_exact;
      // after the first stage the residual is no longer float16-exact
      if (F16IN && m == 0)
        make_b<true>(x, raw, ex, h, b1, b2, rr, need_exact, ss);
      else
        make_b<false>(x, raw, ex, h, b1, b2, rr, need_exact, ss);
      const int key = min_key(tl, b1, b2);
      float dhat;
      int kstar = reduce_rows(key, h, dhat);
      need_exact = need_exact || !(dhat <= ldexpf(rr, SA + 1)) || kstar >= K;
      const unsigned long long fb = __ballot(valid && need_exact && h == 0);
      if (MULTI) {
        const float* gcb = a.gain + (size_t)cb * K;
        const float* scb = a.shape + (size_t)cb * K * d;
        if (fb) exact_rows(fb, x, d, d, K, gcb, scb, false, kstar);
        if (kstar >= K) kstar = K - 1;   // only tail rows past N can get here
        const float gk = gcb[kstar];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j < d) x[j] = fmaf(-gk, scb[(size_t)kstar * d + j], x[j]);
      } else {
        if (fb) exact_rows(fb, x, d, DP, K, mg, ms, false, kstar);
        if (kstar >= K) kstar = K - 1;
        if (a.residual) {
          const float gk = mg[kstar];
#pragma unroll
          for (int j = 0; j < 8; ++j) x[j] = fmaf(-gk, ms[kstar * DP + j], x[j]);
        }
      }
      if (valid && h == 0 && a.codes) {
        const int64_t t = (int64_t)m * G + g;
        if (lds_codes) {
          ((uint8_t*)(codes_l + m * a.chunk_rows + (row - row_begin)))[sg] = (uint8_t)kstar;
        } else if (a.byte_codes) {
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
    if (valid && a.residual && h == 0) {
      float* dst = a.residual + row * (int64_t)(G * d) + (int64_t)g * d;
      for (int j = 0; j < d; ++j) dst[j] = x[j];
    }
    rb = rb_next;
    rb_next = rb_after;
  }
  __syncthreads();
  }
flush:
  if (lds_codes) {
    // one 32-bit word per (stage, row): the codes of this block's four
    // consecutive subspaces
    const int64_t g0 = (int64_t)blockIdx.y * ENC_SUBS;
    const int nrows = (int)(row_end - row_begin);
    for (int e = threadIdx.x; e < a.M * nrows; e += blockDim.x) {
      const int m = e / nrows, r = e % nrows;
      uint32_t* dst = (uint32_t*)((uint8_t*)(a.codes + (row_begin + r) * a.words) + m * G + g0);
      *dst = codes_l[m * a.chunk_rows + r];
    }
  }
}

// Latency encoder for a few rows with a prepared codebook (the tokens
// appended to a cache at each decoding step): one wave per (32-row block,
// subspace), no LDS, no barriers and no block claiming, so a launch of 1 to
// a few hundred rows costs little more than its loads: the header and the
// rows in one round trip, then (the header matching) the first stage's
// operand tables in a second; the arithmetic is the stage-fused encoder's (same operand tables, same
// keys, same float64 re-scoring and residual update), so codes and residuals
// agree with it bit for bit.
template <typename T, bool VEC>
__global__ void __launch_bounds__(ENC_SMALL_WAVES * 64) encode_small_kernel(EncodeArgs a) {
  constexpr bool F16IN = sizeof(T) == 2;
  const int lane = wave_lane();
  const int G = a.G, d = a.d, K = a.K;
  const int wid =
      __builtin_amdgcn_readfirstlane((int)blockIdx.x * ENC_SMALL_WAVES + (int)(threadIdx.x >> 6));
  const int g = wid % G, rb = wid / G;
  const int nblk = (int)((a.N + RB - 1) / RB);
  if (rb >= nblk) return;   // uniform over the wave; no barrier follows
  const int i = lane & 31, h = lane >> 5;
  const int64_t row = (int64_t)rb * RB + i;
  const bool valid = row < a.N;
  RowRaw<T, VEC> nx;
  nx.load((const T*)a.x + (valid ? row : 0) * a.ldx + (int64_t)g * d, d);
  // the header first, fetched with the row: a buffer prepared for another
  // shape may be smaller than this shape's tables, so nothing else is read
  // from it before the header matches (a mismatch gives all-ones code fields
  // and a NaN residual)
  uint32_t tag[PREP_WORDS];
#pragma unroll
  for (int w = 0; w < PREP_WORDS; ++w) tag[w] = a.ptag[w];
  {
    // one wait for the row and the header together (left to itself the
    // compiler issues the row after the branch, or waits for it before it
    // fetches the header)
    uint32_t* rw = (uint32_t*)nx.v;
#pragma unroll
    for (int j = 0; j < (int)sizeof(nx.v) / 4; ++j) asm volatile("" : "+v"(rw[j]));
#pragma unroll
    for (int w = 0; w < PREP_WORDS; ++w) asm volatile("" : "+v"(tag[w]));
  }
  bool ok = true;
#pragma unroll
  for (int w = 0; w < PREP_WORDS; ++w) ok &= tag[w] == a.etag.w[w];
  if (!ok) {   // uniform over the wave: every lane read the same header
    if (valid && h == 0) {
      for (int m = 0; m < a.M; ++m) {
        if (!a.codes) break;
        const int64_t bit = ((int64_t)m * G + g) * a.b;
        if (a.byte_codes) {
          ((uint8_t*)(a.codes + row * a.words))[bit / 8] = 0xffu;
        } else {   // words zeroed beforehand
          uint32_t* wp = a.codes + row * a.words + bit / 32;
          const int off = (int)(bit % 32);
          const uint32_t ones = (1u << a.b) - 1u;
          atomicOr(wp, ones << off);
          if (off + a.b > 32) atomicOr(wp + 1, ones >> (32 - off));
        }
      }
      if (a.residual) {
        float* dst = a.residual + row * (int64_t)(G * d) + (int64_t)g * d;
        for (int j = 0; j < d; ++j) dst[j] = __builtin_nanf("");
      }
    }
    return;
  }
  // then the first stage's tables and sigma, all in flight together
  Tiles tl;
  {
    const u4* fr = a.frag + (size_t)g * NT * 2 * 64;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tl.a1[t] = fr[(t * 2 + 0) * 64 + lane];
      tl.a2[t] = fr[(t * 2 + 1) * 64 + lane];
    }
  }
  int ex = a.sig[g];
  float x[8];
  nx.get(x, d, valid);
  const u4 raw = nx.raw16(x, valid);
  for (int m = 0; m < a.M; ++m) {
    const int cb = m * G + g;
    if (m > 0) {
      const u4* fr = a.frag + (size_t)cb * NT * 2 * 64;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        tl.a1[t] = fr[(t * 2 + 0) * 64 + lane];
        tl.a2[t] = fr[(t * 2 + 1) * 64 + lane];
      }
      ex = a.sig[cb];
    }
    h8 b1, b2;
    float rr, ss;
    bool need_exact;
    if (F16IN && m == 0)
      make_b<true>(x, raw, ex, h, b1, b2, rr, need_exact, ss);
    else
      make_b<false>(x, raw, ex, h, b1, b2, rr, need_exact, ss);
    const int key = min_key(tl, b1, b2);
    float dhat;
    int kstar = reduce_rows(key, h, dhat);
    need_exact = need_exact || !(dhat <= ldexpf(rr, SA + 1)) || kstar >= K;
    const unsigned long long fb = __ballot(valid && need_exact && h == 0);
    const float* gcb = a.gain + (size_t)cb * K;
    const float* scb = a.shape + (size_t)cb * K * d;
    if (fb) {
      ExactCodebook xc;
      // VEC implies d == 8; a prepared buffer's shapes are 256-byte aligned
      xc.load<VEC>(gcb, scb, d, K);
      xc.rows(fb, x, d, K, kstar);
    }
    if (kstar >= K) kstar = K - 1;   // only rows past N can get here
    if (a.residual || m + 1 < a.M) {
      const float gk = gcb[kstar];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < d) x[j] = fmaf(-gk, scb[(size_t)kstar * d + j], x[j]);
    }
    if (valid && h == 0 && a.codes) {
      const int64_t t = (int64_t)m * G + g;
      const uint32_t code = (uint32_t)kstar;
      if (a.byte_codes) {
        ((uint8_t*)(a.codes + row * a.words))[t] = (uint8_t)code;
      } else {   // words zeroed beforehand
        const int64_t bit = t * a.b;
        uint32_t* wp = a.codes + row * a.words + bit / 32;
        const int off = (int)(bit % 32);
        atomicOr(wp, code << off);
        if (off + a.b > 32) atomicOr(wp + 1, code >> (32 - off));
      }
    }
  }
  if (valid && a.residual && h == 0) {
    float* dst = a.residual + row * (int64_t)(G * d) + (int64_t)g * d;
    for (int j = 0; j < d; ++j) dst[j] = x[j];
  }
}

struct DecodeArgs {
  const uint32_t* codes;
  int64_t N, ldo;
  int d, K, G, M_use, b, words;
  const float* gain;
  const float* shape;
  void* out;
  int gpw, gblocks;      // LDS kernel: subspaces per workgroup, subspace blocks
  int64_t rows_per_wg;   // LDS kernel: rows per workgroup
  int tab_bytes;         // LDS kernel: table bytes (staged code words follow)
  int vec;               // LDS kernel: 8-element vector stores are aligned
};

// Gather-sum decoder, generic fallback: one thread per (row, subspace),
// codewords read from global memory.  Used when a subspace's codeword table
// does not fit the LDS kernel below.
template <typename TO>
__global__ void decode_global_kernel(DecodeArgs a) {
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
      {
        // the codeword g s is rounded to float32 before the stage sum
#pragma clang fp contract(off)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j < a.d) acc[j] += gk * s[j];
      }
    }
    TO* dst = (TO*)a.out + row * a.ldo + (int64_t)g * a.d;
    for (int j = 0; j < a.d; ++j) dst[j] = (TO)acc[j];
  }
}

constexpr int DEC_THREADS = 1024;
constexpr int DEC_TABLE_BYTES = 65536;     // codeword table per workgroup
constexpr int DEC_ROW_BATCH = 4;           // rows in flight per thread
constexpr int DEC_FILL_BATCH = 4;          // table entries in flight per thread
constexpr int DEC_CODE_PT = 16;            // staged code words per thread, at most

template <typename TO> struct OutVec;
template <> struct OutVec<_Float16> {
  static __device__ __forceinline__ void store(_Float16* p, const float (&v)[8]) {
    h8 h;
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = (_Float16)v[j];
    *(u4*)p = __builtin_bit_cast(u4, h);
  }
};
template <> struct OutVec<float> {
  static __device__ __forceinline__ void store(float* p, const float (&v)[8]) {
    ((f4*)p)[0] = (f4){v[0], v[1], v[2], v[3]};
    ((f4*)p)[1] = (f4){v[4], v[5], v[6], v[7]};
  }
};

// Codeword table entry c = g s of DP elements, stored as float32, or as
// float16 when a single stage is decoded to float16 (the product is then
// rounded once, exactly as the store would round it).
template <typename TT> struct TabEntry;
template <> struct TabEntry<float> {
  static __device__ __forceinline__ void put(float* t, const float (&c)[8]) {
    ((f4*)t)[0] = (f4){c[0], c[1], c[2], c[3]};
    ((f4*)t)[1] = (f4){c[4], c[5], c[6], c[7]};
  }
  static __device__ __forceinline__ void add(const float* t, float (&acc)[8]) {
    const f4 lo = ((const f4*)t)[0], hi = ((const f4*)t)[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) { acc[j] += lo[j]; acc[4 + j] += hi[j]; }
  }
};
template <> struct TabEntry<_Float16> {
  static __device__ __forceinline__ void put(_Float16* t, const float (&c)[8]) {
    h8 h;
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = (_Float16)c[j];
    *(u4*)t = __builtin_bit_cast(u4, h);
  }
  static __device__ __forceinline__ void add(const _Float16* t, float (&acc)[8]) {
    const h8 h = as_h8(*(const u4*)t);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += (float)h[j];
  }
};

// Code words of subspaces [g0, g0 + ngr) of stage m within a row: the
// word range [lo, lo + n) holding their b-bit fields.
__device__ __forceinline__ void stage_words(int m, int G, int g0, int ngr, int b, int& lo,
                                            int& n) {
  const int64_t first = ((int64_t)m * G + g0) * b;
  const int64_t last = first + (int64_t)ngr * b - 1;
  lo = (int)(first >> 5);
  n = (int)(last >> 5) - lo + 1;
}

// Gather-sum decoder with the codeword table in LDS.  A workgroup owns `gpw`
// consecutive subspaces and a contiguous range of rows; its table holds the
// codewords g s of those subspaces for the first M_use stages, laid out
// [gpw][M_use][K][8].  The code words of its rows and subspaces are staged
// in LDS too ([rows][words of stage 0, stage 1, ...]), loaded together with
// the table, so the output loop issues no global loads: its stores stream
// without waiting on loads (a wait on a load also waits for every store
// issued before it).  Threads map to (row, subspace) with the subspace
// fastest, so each row's output slice of gpw * d elements is written
// contiguously, and every thread keeps DEC_ROW_BATCH rows in flight.
// Workgroups that share rows (and so share code words) are numbered to land
// on the same XCD, whose L2 then serves the shared code lines.
template <typename TO, typename TT>
__global__ void __launch_bounds__(DEC_THREADS) decode_lds_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) unsigned char dec_smem[];
  TT* tab = (TT*)dec_smem;
  uint32_t* cwl = (uint32_t*)(dec_smem + a.tab_bytes);
  const int gpw = a.gpw, gblocks = a.gblocks;
  const int id = blockIdx.x;
  const int xcd = id % 8, slot = id / 8;
  const int gb = slot % gblocks;
  const int rc = (slot / gblocks) * 8 + xcd;
  const int64_t r_begin = (int64_t)rc * a.rows_per_wg;
  if (r_begin >= a.N) return;
  int64_t r_end = r_begin + a.rows_per_wg;
  if (r_end > a.N) r_end = a.N;
  const int nrows = (int)(r_end - r_begin);
  const int g0 = gb * gpw;
  const int ngr = min(gpw, a.G - g0);
  const int K = a.K, M = a.M_use, d = a.d, G = a.G, b = a.b;
  const int tid = threadIdx.x;
  // staged code words per row (host-checked: nrows * rs <= DEC_CODE_PT * DEC_THREADS)
  int rs = 0;
  for (int m = 0; m < M; ++m) {
    int lo, n;
    stage_words(m, G, g0, ngr, b, lo, n);
    rs += n;
  }
  const int ncw = nrows * rs;
  const uint32_t* crow = a.codes + r_begin * a.words;
  uint32_t cw[DEC_CODE_PT];
#pragma unroll
  for (int q = 0; q < DEC_CODE_PT; ++q) {
    if (q * DEC_THREADS < ncw) {           // uniform per q
      const int e = min(q * DEC_THREADS + tid, ncw - 1);
      const int row = e / rs;
      int j = e - row * rs, m = 0, lo, n;
      stage_words(0, G, g0, ngr, b, lo, n);
      while (j >= n) {
        j -= n;
        ++m;
        stage_words(m, G, g0, ngr, b, lo, n);
      }
      cw[q] = crow[(int64_t)row * a.words + lo + j];
    }
  }
  // table fill: every load of a batch is issued before the first use
  const int entries = ngr * M * K;
  for (int e0 = 0; e0 < entries; e0 += DEC_THREADS * DEC_FILL_BATCH) {
    float g[DEC_FILL_BATCH], c[DEC_FILL_BATCH][8];
#pragma unroll
    for (int q = 0; q < DEC_FILL_BATCH; ++q) {
      const int e = min(e0 + q * DEC_THREADS + tid, entries - 1);
      // K = 2^b; no integer division unless several stages are decoded
      const int k = e & (K - 1), q2 = e >> b;
      const int m = M == 1 ? 0 : q2 % M, gi = M == 1 ? q2 : q2 / M;
      const size_t cb = (size_t)m * G + g0 + gi;
      read_codeword(a.gain + cb * K, a.shape + cb * K * d, d, K, k, false, g[q], c[q]);
    }
#pragma unroll
    for (int q = 0; q < DEC_FILL_BATCH; ++q) {
      const int e = e0 + q * DEC_THREADS + tid;
      if (e < entries) {
#pragma unroll
        for (int j = 0; j < 8; ++j) c[q][j] *= g[q];
        TabEntry<TT>::put(tab + (size_t)e * 8, c[q]);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < DEC_CODE_PT; ++q) {
    const int e = q * DEC_THREADS + tid;
    if (e < ncw) cwl[e] = cw[q];
  }
  __syncthreads();
  const int gi = tid % gpw;
  if (gi >= ngr) return;
  const int rstep = DEC_THREADS / gpw;
  const int g = g0 + gi;
  const TT* tg = tab + (size_t)gi * M * K * 8;
  for (int r0 = tid / gpw; r0 < nrows; r0 += DEC_ROW_BATCH * rstep) {
    float acc[DEC_ROW_BATCH][8];
#pragma unroll
    for (int q = 0; q < DEC_ROW_BATCH; ++q)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[q][j] = 0.f;
    int off = 0;                            // staged words of the stages before m
    for (int m = 0; m < M; ++m) {
      int lo, n;
      stage_words(m, G, g0, ngr, b, lo, n);
      const int p = (int)(((int64_t)m * G + g) * b - (int64_t)lo * 32);
      const int wi = off + (p >> 5), sh = p & 31;
      const bool two = sh + b > 32;
      int k[DEC_ROW_BATCH];
#pragma unroll
      for (int q = 0; q < DEC_ROW_BATCH; ++q) {
        int row = r0 + q * rstep;
        row = row < nrows ? row : 0;       // in-range row; its result is not stored
        const uint32_t* w = cwl + row * rs + wi;
        uint64_t v = w[0];
        if (two) v |= (uint64_t)w[1] << 32;
        k[q] = (int)((v >> sh) & ((1u << b) - 1));
      }
#pragma unroll
      for (int q = 0; q < DEC_ROW_BATCH; ++q)
        TabEntry<TT>::add(tg + ((size_t)m * K + k[q]) * 8, acc[q]);
      off += n;
    }
#pragma unroll
    for (int q = 0; q < DEC_ROW_BATCH; ++q) {
      const int row = r0 + q * rstep;
      if (row >= nrows) break;
      TO* dst = (TO*)a.out + (r_begin + row) * a.ldo + (int64_t)g * d;
      if (a.vec) {
        OutVec<TO>::store(dst, acc[q]);
      } else {
        for (int j = 0; j < d; ++j) dst[j] = (TO)acc[q][j];
      }
    }
  }
}

// Input check of gsrq_train_stage (flag GSRQ_CHECK_INPUTS).  Bits of *bad:
// 1 a weight that is negative or not finite, 2 an element of X that is not
// finite, 4 a seed row whose subvector is zero (GSKM seeding needs a
// direction: Alg. 1 starts from shapes on the unit sphere).  Every block
// walks rows; the threads of a block stride over the row's D elements.
constexpr uint32_t CHK_WEIGHT = 1u, CHK_NONFINITE = 2u, CHK_ZERO_SEED = 4u;

__device__ __forceinline__ bool finite_bits(float v) {
  return (__float_as_uint(v) & 0x7f800000u) != 0x7f800000u;
}
__device__ __forceinline__ bool finite_bits(_Float16 v) {
  return (__builtin_bit_cast(uint16_t, v) & 0x7c00u) != 0x7c00u;
}

template <typename T>
__global__ void __launch_bounds__(256) check_inputs_kernel(const T* __restrict__ X, int64_t ldx,
                                                           int64_t N, int D, int d,
                                                           const float* __restrict__ w,
                                                           const int32_t* __restrict__ seeds,
                                                           int nseeds, int K,
                                                           uint32_t* __restrict__ bad) {
  uint32_t flags = 0;
  for (int64_t r = blockIdx.x; r < N; r += gridDim.x) {
    const T* row = X + r * ldx;
    for (int c = threadIdx.x; c < D; c += blockDim.x)
      if (!finite_bits(row[c])) flags |= CHK_NONFINITE;
    if (threadIdx.x == 0 && w) {
      const float v = w[r];
      if (!finite_bits(v) || v < 0.f) flags |= CHK_WEIGHT;
    }
  }
  // seed subvectors: entry e = g K + k names row seeds[e] of subspace g
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < nseeds;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int g = (int)(e / K);
    const T* sub = X + (int64_t)seeds[e] * ldx + (int64_t)g * d;
    bool zero = true;
    for (int j = 0; j < d; ++j) zero &= (float)sub[j] == 0.f;
    if (zero) flags |= CHK_ZERO_SEED;
  }
  if (flags) atomicOr(bad, flags);
}

// ------------------------------------------------------------- host side

// Optional launch timing (off by default): HIP events bracket every launch
// of the instrumented kernels on the launch's own stream.
gsrq_status check_shape(const gsrq_shape* s, bool need_m) {
  if (!s) return GSRQ_E_ARG;
  if (s->N < 1 || s->D < 1 || s->d < 1 || s->D % s->d != 0) return GSRQ_E_ARG;
  if (s->K < 2 || s->K > 65536 || !is_pow2(s->K)) return GSRQ_E_ARG;
  if (need_m && s->M < 1) return GSRQ_E_ARG;
  return GSRQ_OK;
}

// Shapes of the narrow family (this file); gsrq_wide::serves() names the
// shapes of the wide one.
bool narrow(const gsrq_shape* s) { return s->d <= DP && s->K <= KMAX; }

gsrq_status check_supported(const gsrq_shape* s) {
  if (narrow(s) || gsrq_wide::serves(s)) return GSRQ_OK;
  return GSRQ_E_UNSUPPORTED;
}

struct TrainLayout {
  size_t xt, part, assign, done, iters, wxx, seednorm, seeds, cbg[2], cbs[2], total;
  int chunks, chunk_rows;
};

TrainLayout train_layout(const gsrq_shape* s, size_t elt) {
  TrainLayout L;
  const int64_t G = s->D / s->d;
  // about one workgroup per CU in all: chunks per subspace from the CU
  // count, within the per-workgroup row limits
  int64_t chunks = (TRAIN_SLOTS + G - 1) / G;
  const int64_t lo = (s->N + TRAIN_CHUNK_MAX - 1) / TRAIN_CHUNK_MAX;
  const int64_t hi = (s->N + TRAIN_CHUNK_MIN - 1) / TRAIN_CHUNK_MIN;
  chunks = chunks < hi ? chunks : hi;
  chunks = chunks > lo ? chunks : lo;
  int64_t rows = (s->N + chunks - 1) / chunks;
  rows = (rows + RB - 1) / RB * RB;
  L.chunk_rows = (int)rows;
  L.chunks = (int)((s->N + rows - 1) / rows);
  size_t off = 0;
  L.xt = off; off = align256(off + (size_t)G * s->N * 8 * elt);
  L.part = off; off = align256(off + (size_t)G * L.chunks * PSTRIDE * sizeof(double));
  L.assign = off; off = align256(off + (size_t)G * s->N * sizeof(uint16_t));
  L.done = off; off = align256(off + (size_t)G * sizeof(int));
  L.iters = off; off = align256(off + (size_t)G * sizeof(int));
  L.wxx = off; off = align256(off + (size_t)G * sizeof(double));
  L.seednorm = off; off = align256(off + (size_t)G * s->K * sizeof(float));
  L.seeds = off; off = align256(off + (size_t)G * s->K * sizeof(int32_t));
  // codebooks of consecutive iterations (updates fused into the assignment
  // launches write one while the next launch reads the other)
  for (int b = 0; b < 2; ++b) {
    L.cbg[b] = off; off = align256(off + (size_t)G * s->K * sizeof(float));
    L.cbs[b] = off; off = align256(off + (size_t)G * s->K * s->d * sizeof(float));
  }
  L.total = off;
  return L;
}

// multi-stage encode keeps per-stage operand tiles in the workspace
size_t encode_ws(const gsrq_shape* s) {
  const int64_t G = s->D / s->d;
  if (s->M <= 1) return 256;
  return align256((size_t)s->M * G * NT * 2 * 64 * sizeof(u4)) +
         align256((size_t)s->M * G * sizeof(int));
}

// Layout of a prepared codebook: header, sigma exponents [M G], operand
// tiles [M G][NT][2][64], then copies of the gains [M][G][K] and shapes
// [M][G][K][d] it was built from.
struct PrepLayout {
  size_t sig, frag, gain, shape, total;
};

PrepLayout prep_layout(const gsrq_shape* s) {
  const int64_t ncb = (int64_t)s->M * (s->D / s->d);
  PrepLayout P;
  size_t off = 256;
  P.sig = off; off = align256(off + ncb * sizeof(int));
  P.frag = off; off = align256(off + ncb * NT * 2 * 64 * sizeof(u4));
  P.gain = off; off = align256(off + ncb * s->K * sizeof(float));
  P.shape = off; off = align256(off + ncb * s->K * s->d * sizeof(float));
  P.total = off;
  return P;
}

template <typename T>
gsrq_status encode_launch(const gsrq_shape* s, const void* X, int64_t ldx, const float* gain,
                          const float* shape, int M, uint32_t* codes, float* residual, void* ws,
                          hipStream_t st, const void* prepared = nullptr) {
  EncodeArgs a;
  a.x = X; a.ldx = ldx; a.N = s->N; a.d = s->d; a.K = s->K; a.G = s->D / s->d; a.M = M;
  a.b = log2i(s->K);
  a.words = (int)((M * (int64_t)a.G * a.b + 31) / 32);
  a.gain = gain; a.shape = shape; a.frag = nullptr; a.sig = nullptr;
  a.codes = codes; a.residual = residual;
  a.byte_codes = (a.b == 8) && ((M * (int64_t)a.G) % 4 == 0);
  a.lds_codes = codes && a.byte_codes && (a.G % ENC_SUBS == 0) && M <= ENC_MAX_STAGES;
  const size_t esz = sizeof(T);
  a.vec_rows = (s->d == 8) && ((uintptr_t)X % 16 == 0) && ((ldx * esz) % 16 == 0);
  a.ptag = nullptr;
  a.etag = prep_tag(M, a.G, s->d, s->K);
  gsrq_status e;
  // prepared codebook: tables and codebook from the buffer, header checked
  const bool multi = M > 1 || prepared;
  if (prepared) {
    const PrepLayout P = prep_layout(s);
    const char* pb = (const char*)prepared;
    a.ptag = (const uint32_t*)pb;
    a.sig = (const int*)(pb + P.sig);
    a.frag = (const u4*)(pb + P.frag);
    a.gain = (const float*)(pb + P.gain);
    a.shape = (const float*)(pb + P.shape);
  }
  if (codes && !a.byte_codes) {
    if ((e = fill_u32(codes, (size_t)s->N * a.words, 0u, st))) return e;
  }
  if (M > 1 && !prepared) {
    u4* frag = (u4*)ws;
    int* sig = (int*)((char*)ws + align256((size_t)M * a.G * NT * 2 * 64 * sizeof(u4)));
    tiles_kernel<<<(unsigned)(M * a.G), 64, 0, st>>>(gain, shape, s->d, s->K, frag, sig, nullptr,
                                                     a.etag);
    if ((e = launch_ok())) return e;
    a.frag = frag;
    a.sig = sig;
  }
  if (prepared && s->N <= ENC_SMALL_ROWS) {
    // a few rows: one wave per (row block, subspace), nothing shared
    const int64_t waves = (s->N + RB - 1) / RB * a.G;
    const unsigned wgs = (unsigned)((waves + ENC_SMALL_WAVES - 1) / ENC_SMALL_WAVES);
    TimedLaunch tl(GSRQ_KERNEL_ENCODE, st);
    if (a.vec_rows)
      encode_small_kernel<T, true><<<wgs, ENC_SMALL_WAVES * 64, 0, st>>>(a);
    else
      encode_small_kernel<T, false><<<wgs, ENC_SMALL_WAVES * 64, 0, st>>>(a);
    return launch_ok();
  }
  // about one workgroup per CU: rows split into chunks so that the groups
  // of ENC_SUBS subspaces times the chunks fill the 256 CUs once; a chunk's
  // LDS-staged codes (M words per row) bound its rows
  const int64_t groups = (a.G + ENC_SUBS - 1) / ENC_SUBS;
  int64_t chunks = std::max<int64_t>(1, (256 + groups - 1) / groups);
  int64_t cr = (s->N + chunks - 1) / chunks;
  cr = (cr + RB - 1) / RB * RB;
  const int64_t cap = (int64_t)ENC_CODES_WORDS / std::max(1, M) / RB * RB;
  if (cr > cap) cr = cap;
  a.chunk_rows = cr;
  chunks = (s->N + cr - 1) / cr;
  if (chunks > 0x7fffffff) return GSRQ_E_UNSUPPORTED;
  dim3 grid((unsigned)chunks, (unsigned)groups);
  TimedLaunch tl(GSRQ_KERNEL_ENCODE, st);
  if (multi) {
    if (a.vec_rows)
      encode_kernel<T, true, true><<<grid, ENC_WAVES * 64, 0, st>>>(a);
    else
      encode_kernel<T, true, false><<<grid, ENC_WAVES * 64, 0, st>>>(a);
  } else {
    if (a.vec_rows)
      encode_kernel<T, false, true><<<grid, ENC_WAVES * 64, 0, st>>>(a);
    else
      encode_kernel<T, false, false><<<grid, ENC_WAVES * 64, 0, st>>>(a);
  }
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
    TimedLaunch tl(GSRQ_KERNEL_TRANSPOSE, st);
    transpose_kernel<T><<<grid_for(work, 256), 256, 0, st>>>((const T*)X, ldx, s->N, d, G, xt);
    if ((e = launch_ok())) return e;
  }
  if ((e = fill_u32(done, G, 0u, st))) return e;
  if ((e = fill_u32(iters, G, 0u, st))) return e;
  if (trace && T_ > 0 && (e = fill_u32(trace, (size_t)G * T_ * 2, 0u, st))) return e;

  AssignArgs aa = {};
  aa.xt = xt; aa.N = s->N; aa.d = d; aa.K = K; aa.G = G; aa.w = w;
  aa.gain = gain; aa.shape = shape; aa.assign = assign;
  aa.done = done; aa.iters = iters; aa.part = part;
  aa.seednorm = seednorm; aa.trace = trace;
  aa.wxx = (double*)(base + L.wxx);
  aa.want_wxx = trace != nullptr;   // the first pass computes it
  aa.chunks = L.chunks; aa.chunk_rows = L.chunk_rows; aa.force_changed = 0; aa.t = 0; aa.T = T_;
  aa.no_early_stop = (flags & GSRQ_NO_EARLY_STOP) ? 1 : 0;
  aa.kmeans = (flags & GSRQ_KMEANS) ? 1 : 0;
  float* bufg[2] = {(float*)(base + L.cbg[0]), (float*)(base + L.cbg[1])};
  float* bufs[2] = {(float*)(base + L.cbs[0]), (float*)(base + L.cbs[1])};
  aa.buf_gain[0] = bufg[0]; aa.buf_gain[1] = bufg[1];
  aa.buf_shape[0] = bufs[0]; aa.buf_shape[1] = bufs[1];
  aa.fin_gain = gain; aa.fin_shape = shape;
  const dim3 agrid((unsigned)L.chunks, (unsigned)G);

  if (!resume) {
    if (hipMemcpyAsync(dseeds, seeds, (size_t)G * K * sizeof(int32_t), hipMemcpyHostToDevice,
                       st) != hipSuccess)
      return GSRQ_E_HIP;
    seed_kernel<T><<<G, 256, 0, st>>>(xt, s->N, d, K, dseeds, shape, seednorm, aa.kmeans, gain);
    if ((e = launch_ok())) return e;
  }
  // GSKM from seed rows: an initial assignment with unit gains; its gains
  // (eq. 8) are computed at the start of the first iteration's launch
  const bool seeded_gskm = !resume && !aa.kmeans;
  int prev_wxx = 0;   // the last pass accumulated sum w ||x||^2
  if (!resume && aa.kmeans) {
    // K-means starts from the seed centroids; there is no previous assignment
    aa.force_changed = 1;
  } else if (seeded_gskm) {
    {
      TimedLaunch tl(GSRQ_KERNEL_ASSIGN, st);
      assign_accumulate_kernel<T, MODE_INIT><<<agrid, TRAIN_WAVES * 64, 0, st>>>(aa);
    }
    if ((e = launch_ok())) return e;
    prev_wxx = aa.want_wxx;
    aa.want_wxx = 0;
    if (T_ == 0) {
      // initialisation only: the gains straight into the caller's arrays
      aa.old_shape = shape;
      aa.upd_has_wxx = prev_wxx;
      TimedLaunch tl(GSRQ_KERNEL_FINALIZE, st);
      update_kernel<MODE_INIT><<<G, UPD_THREADS, 0, st>>>(aa);
      return launch_ok();
    }
  } else {
    aa.force_changed = (flags & GSRQ_ASSIGN_IN) ? 0 : 1;
  }
  // where codebook C_j (the one iteration j + 1 scores with) lives: C_0 in
  // the caller's arrays (seeded K-means, resume) or, computed by the first
  // launch, in buffer 0; later ones alternate between the two buffers
  auto cb_gain = [&](int j) -> float* { return (j == 0 && !seeded_gskm) ? gain : bufg[j & 1]; };
  auto cb_shape = [&](int j) -> float* { return (j == 0 && !seeded_gskm) ? shape : bufs[j & 1]; };
  for (int t = 1; t <= T_; ++t) {
    aa.t = t;
    aa.upd_has_wxx = prev_wxx;
    if (t == 1 && !seeded_gskm) {
      aa.upd = UPD_NONE;
      aa.gain = gain;
      aa.shape = shape;
    } else {
      aa.upd = t == 1 ? UPD_INIT : UPD_ITER;
      aa.old_gain = t == 1 ? nullptr : cb_gain(t - 2);
      aa.old_shape = t == 1 ? shape : cb_shape(t - 2);   // seed shapes for the first
      aa.new_gain = cb_gain(t - 1);
      aa.new_shape = cb_shape(t - 1);
    }
    {
      TimedLaunch tl(GSRQ_KERNEL_ASSIGN, st);
      assign_accumulate_kernel<T, MODE_ITER><<<agrid, TRAIN_WAVES * 64, 0, st>>>(aa);
    }
    if ((e = launch_ok())) return e;
    prev_wxx = aa.want_wxx;
    aa.force_changed = 0;
    aa.want_wxx = 0;
  }
  if (T_ > 0) {
    // the last iteration's update into the caller's arrays; subspaces that
    // stopped earlier get their final codebook copied there
    aa.upd_has_wxx = prev_wxx;
    aa.old_gain = cb_gain(T_ - 1);
    aa.old_shape = cb_shape(T_ - 1);
    aa.copy_done = 1;
    TimedLaunch tl(GSRQ_KERNEL_FINALIZE, st);
    update_kernel<MODE_ITER><<<G, UPD_THREADS, 0, st>>>(aa);
  }
  if ((e = launch_ok())) return e;
  if (R_next) {
    gsrq_shape s1 = *s;
    s1.M = 1;
    return encode_launch<T>(&s1, X, ldx, gain, shape, 1, nullptr, R_next, nullptr, st);
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
  *bytes = narrow(s) ? train_layout(s, sizeof(float)).total
                     : gsrq_wide::train_workspace_bytes(s, 0);
  return GSRQ_OK;
}

gsrq_status gsrq_encode_workspace_bytes(const gsrq_shape* s, size_t* bytes) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!bytes) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  *bytes = narrow(s) ? encode_ws(s) : gsrq_wide::encode_workspace_bytes(s);
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
  if (flags & ~(uint32_t)(GSRQ_RESUME | GSRQ_ASSIGN_IN | GSRQ_NO_EARLY_STOP | GSRQ_KMEANS |
                          GSRQ_CHECK_INPUTS))
    return GSRQ_E_ARG;
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
      std::sort(tmp, tmp + s->K);
      bool dup = false;
      for (int a = 1; a < s->K; ++a) dup |= tmp[a] == tmp[a - 1];
      delete[] tmp;
      if (dup) return GSRQ_E_ARG;
    }
  }
  const size_t elt = x_dtype == GSRQ_F16 ? sizeof(_Float16) : sizeof(float);
  const size_t need = narrow(s) ? train_layout(s, elt).total
                                : gsrq_wide::train_workspace_bytes(s, elt);
  if (ws_bytes < need) return GSRQ_E_WORKSPACE;
  if (flags & GSRQ_CHECK_INPUTS) {
    // the check runs before anything else and uses the start of the
    // workspace (a status word, then a device copy of the seed table); the
    // call waits for it, and on a failed check returns with no output touched
    const bool seeded = !(flags & GSRQ_RESUME) && !(flags & GSRQ_KMEANS);
    const size_t nseeds = seeded ? (size_t)G * s->K : 0;
    if (need < 256 + nseeds * sizeof(int32_t)) return GSRQ_E_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    uint32_t* bad = (uint32_t*)workspace;
    int32_t* dseeds = (int32_t*)((char*)workspace + 256);
    if ((e = fill_u32(bad, 1, 0u, st))) return e;
    if (nseeds && hipMemcpyAsync(dseeds, seed_rows, nseeds * sizeof(int32_t),
                                 hipMemcpyHostToDevice, st) != hipSuccess)
      return GSRQ_E_HIP;
    const int grid = (int)std::min<int64_t>(s->N, 2048);
    if (x_dtype == GSRQ_F16)
      check_inputs_kernel<_Float16><<<grid, 256, 0, st>>>((const _Float16*)X, ldx, s->N, s->D,
                                                          s->d, w, dseeds, (int)nseeds, s->K, bad);
    else
      check_inputs_kernel<float><<<grid, 256, 0, st>>>((const float*)X, ldx, s->N, s->D, s->d,
                                                       w, dseeds, (int)nseeds, s->K, bad);
    if ((e = launch_ok())) return e;
    uint32_t hbad = 0;
    if (hipMemcpyAsync(&hbad, bad, sizeof(hbad), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
      return GSRQ_E_HIP;
    if (hbad) return GSRQ_E_ARG;
  }
  if (!narrow(s))
    return gsrq_wide::train_stage(s, X, x_dtype, ldx, w, T, seed_rows, flags, gain, shape,
                                  R_next, assign_io, iters_run, obj_trace, workspace, stream);
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
  if (!narrow(s)) {
    if (ws_bytes < gsrq_wide::encode_workspace_bytes(s)) return GSRQ_E_WORKSPACE;
    return gsrq_wide::encode(s, X, x_dtype, ldx, gain, shape, codes, residual, workspace, stream);
  }
  if (ws_bytes < encode_ws(s)) return GSRQ_E_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  if (x_dtype == GSRQ_F16)
    return encode_launch<_Float16>(s, X, ldx, gain, shape, s->M, codes, residual, workspace, st);
  return encode_launch<float>(s, X, ldx, gain, shape, s->M, codes, residual, workspace, st);
}

gsrq_status gsrq_prepared_bytes(const gsrq_shape* s, size_t* bytes) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!bytes) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  if (!narrow(s)) return GSRQ_E_UNSUPPORTED;
  *bytes = prep_layout(s).total;
  return GSRQ_OK;
}

gsrq_status gsrq_encode_prepare(const gsrq_shape* s, const float* gain, const float* shape,
                                void* prepared, size_t bytes, void* stream) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!gain || !shape || !prepared) return GSRQ_E_ARG;
  if (((uintptr_t)prepared & 255) != 0) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  if (!narrow(s)) return GSRQ_E_UNSUPPORTED;
  const PrepLayout P = prep_layout(s);
  if (bytes < P.total) return GSRQ_E_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  char* pb = (char*)prepared;
  const int64_t ncb = (int64_t)s->M * (s->D / s->d);
  if (hipMemcpyAsync(pb + P.gain, gain, ncb * s->K * sizeof(float), hipMemcpyDeviceToDevice,
                     st) != hipSuccess ||
      hipMemcpyAsync(pb + P.shape, shape, ncb * s->K * s->d * sizeof(float),
                     hipMemcpyDeviceToDevice, st) != hipSuccess)
    return GSRQ_E_HIP;
  tiles_kernel<<<(unsigned)ncb, 64, 0, st>>>((const float*)(pb + P.gain),
                                             (const float*)(pb + P.shape), s->d, s->K,
                                             (u4*)(pb + P.frag), (int*)(pb + P.sig),
                                             (uint32_t*)pb,
                                             prep_tag(s->M, (int)(s->D / s->d), s->d, s->K));
  return launch_ok();
}

gsrq_status gsrq_encode_prepared(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype,
                                 int64_t ldx, const void* prepared, uint32_t* codes,
                                 float* residual, void* stream) {
  gsrq_status e = check_shape(s, true);
  if (e) return e;
  if (!X || !prepared || (!codes && !residual)) return GSRQ_E_ARG;
  if (x_dtype != GSRQ_F32 && x_dtype != GSRQ_F16) return GSRQ_E_ARG;
  if (ldx < s->D || ((uintptr_t)prepared & 255) != 0) return GSRQ_E_ARG;
  if ((e = check_supported(s))) return e;
  if (!narrow(s) || s->M > ENC_MAX_STAGES) return GSRQ_E_UNSUPPORTED;
  hipStream_t st = (hipStream_t)stream;
  if (x_dtype == GSRQ_F16)
    return encode_launch<_Float16>(s, X, ldx, nullptr, nullptr, s->M, codes, residual, nullptr,
                                   st, prepared);
  return encode_launch<float>(s, X, ldx, nullptr, nullptr, s->M, codes, residual, nullptr, st,
                              prepared);
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
  if (!narrow(s))
    return gsrq_wide::decode(s, codes, M_use, gain, shape, Xhat, out_dtype, ldo, stream);
  DecodeArgs a;
  a.codes = codes; a.N = s->N; a.ldo = ldo; a.d = s->d; a.K = s->K; a.G = s->D / s->d;
  a.M_use = M_use; a.b = log2i(s->K);
  a.words = (int)((s->M * (int64_t)a.G * a.b + 31) / 32);
  a.gain = gain; a.shape = shape; a.out = Xhat;
  hipStream_t st = (hipStream_t)stream;
  TimedLaunch tl(GSRQ_KERNEL_DECODE, st);
  // single-stage float16 output: the table holds float16 products
  const bool half_tab = M_use == 1 && out_dtype == GSRQ_F16;
  const int64_t per_group = (int64_t)M_use * s->K * 8 * (half_tab ? 2 : 4);  // table bytes
  if (per_group <= DEC_TABLE_BYTES) {
    int gpw = 1;   // a power of two, so (row, subspace) threads tile the workgroup
    while (gpw * 2 <= 64 && gpw * 2 * per_group <= DEC_TABLE_BYTES && gpw < a.G) gpw *= 2;
    a.gpw = gpw;
    a.gblocks = (a.G + gpw - 1) / gpw;
    // staged code words per row: the most any subspace block needs
    int64_t rs = 1;
    for (int gb = 0; gb < a.gblocks; ++gb) {
      const int64_t g0 = (int64_t)gb * gpw, ngr = std::min<int64_t>(gpw, a.G - g0);
      int64_t n = 0;
      for (int m = 0; m < M_use; ++m) {
        const int64_t first = (m * (int64_t)a.G + g0) * a.b, last = first + ngr * a.b - 1;
        n += (last >> 5) - (first >> 5) + 1;
      }
      rs = std::max(rs, n);
    }
    // about one workgroup per CU, each streaming a contiguous row range (the
    // table fill is paid once per workgroup), with at most DEC_CODE_PT
    // staged code words per thread
    int64_t rchunks = (256 + a.gblocks - 1) / a.gblocks;
    const int64_t min_rows = 256;
    if (rchunks * min_rows > s->N) rchunks = (s->N + min_rows - 1) / min_rows;
    if (rchunks < 1) rchunks = 1;
    const int64_t max_rows = (int64_t)DEC_CODE_PT * DEC_THREADS / rs;
    if (max_rows < 1) return GSRQ_E_UNSUPPORTED;
    a.rows_per_wg = (s->N + rchunks - 1) / rchunks;
    if (a.rows_per_wg > max_rows) a.rows_per_wg = max_rows;
    rchunks = (s->N + a.rows_per_wg - 1) / a.rows_per_wg;
    if (8 * a.gblocks * ((rchunks + 7) / 8) > INT32_MAX) return GSRQ_E_UNSUPPORTED;
    const int blocks = (int)(8 * a.gblocks * ((rchunks + 7) / 8));
    const size_t esz = out_dtype == GSRQ_F16 ? 2 : 4;
    a.vec = (s->d == 8) && ((uintptr_t)Xhat % 16 == 0) && ((ldo * esz) % 16 == 0);
    a.tab_bytes = (int)(gpw * per_group);
    const size_t lds = (size_t)a.tab_bytes + (size_t)a.rows_per_wg * rs * sizeof(uint32_t);
    auto launch = [&](const void* fn, auto kern) -> gsrq_status {
      if (lds > 65536 &&
          hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
              hipSuccess)
        return GSRQ_E_HIP;
      kern<<<blocks, DEC_THREADS, lds, st>>>(a);
      return GSRQ_OK;
    };
    gsrq_status e;
    if (out_dtype == GSRQ_F16 && half_tab)
      e = launch((const void*)decode_lds_kernel<_Float16, _Float16>,
                 decode_lds_kernel<_Float16, _Float16>);
    else if (out_dtype == GSRQ_F16)
      e = launch((const void*)decode_lds_kernel<_Float16, float>,
                 decode_lds_kernel<_Float16, float>);
    else
      e = launch((const void*)decode_lds_kernel<float, float>, decode_lds_kernel<float, float>);
    if (e) return e;
  } else {
    const int grid = grid_for(s->N * a.G, 256);
    if (out_dtype == GSRQ_F16)
      decode_global_kernel<_Float16><<<grid, 256, 0, st>>>(a);
    else
      decode_global_kernel<float><<<grid, 256, 0, st>>>(a);
  }
  return launch_ok();
}

gsrq_status gsrq_timing_enable_kinds(uint32_t kinds) {
  g_gsrq_timing.on = kinds != 0;
  g_gsrq_timing.kinds = kinds;
  if (kinds) g_gsrq_timing.n = 0;   // switching off keeps the records for reading
  return GSRQ_OK;
}

gsrq_status gsrq_timing_enable(int on) {
  return gsrq_timing_enable_kinds(on ? ~0u : 0u);
}

gsrq_status gsrq_timing_read(double* total_ms, int64_t* launches, int n_kinds) {
  if (!total_ms || !launches || n_kinds < 0) return GSRQ_E_ARG;
  for (int k = 0; k < n_kinds; ++k) { total_ms[k] = 0.0; launches[k] = 0; }
  for (int i = 0; i < g_gsrq_timing.n; ++i) {
    const auto& r = g_gsrq_timing.recs[i];
    if (hipEventSynchronize(r.b) != hipSuccess) return GSRQ_E_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return GSRQ_E_HIP;
    if (r.kind < n_kinds) { total_ms[r.kind] += ms; launches[r.kind] += 1; }
  }
  g_gsrq_timing.n = 0;
  return GSRQ_OK;
}

}  // extern "C"
