// Wide-subspace kernel family of the GSRQ hot path for AMD MI355X (gfx950):
// subvectors of d = 8 C elements (C = 1, 2, 4, 8, 16 or 32 groups of eight) and
// codebooks of any power-of-two size K.  It serves the shapes the narrow
// family in gsrq.hip cannot hold in registers (d > 8 or K > 256).
//
// What is computed is the same as in the narrow family (arXiv 2607.01065:
// gain-shape scoring of eq. 5, argmin with ties to the lowest index, the
// weighted updates of eqs. 6-8 with the safeguards of Sec. 5.2, greedy
// residual encoding of Sec. 3 / 5.1, gather-sum decoding).  How:
//  * Operand fragments.  For every codebook and 32-codeword tile a small
//    kernel writes the A operands of each MFMA of the distance contraction
//    (hi/lo float16 split of a = -2 g s 2^SA / sigma, and the bias terms) to
//    a table in the workspace.  The scoring kernel stages the table through
//    LDS: whole when it fits (resident), else chunk by chunk, double
//    buffered (streamed), so the codebook side is read from L2 once per
//    workgroup and from LDS by every wave.
//  * Rows are the B operands and stay in registers across all tiles.
//    Float16 stage inputs enter exactly; float32 ones (residuals) as a hi/lo
//    pair scaled by a per-row power of two.
//  * Argmin.  Per tile, packed keys with a 4-bit slot (v_min3), then the
//    tile index of the smallest key; the two lane halves holding a row are
//    combined at the end.  Rows whose operands leave the float16 range, or
//    whose best distance exceeds twice their energy, are re-scored exactly
//    in float64.
//  * Training accumulation is a kernel of its own: a workgroup owns a slice
//    of codewords and a chunk of rows, collects the chunk's members of its
//    slice from the assignment, and sums them in float64 LDS accumulators;
//    a finalize kernel reduces the per-chunk partials in a fixed order and
//    applies eqs. 7 and 8 and the stop test.
//  * Multi-stage encode runs one scoring launch per stage; the float32
//    residual passes between stages through HBM (a d = 128 residual does
//    not fit in registers next to the operands).
#include <algorithm>
#include <type_traits>

#include "gsrq_common.h"
#include "gsrq_wide.h"

namespace {

constexpr int W_WAVES = 8;
constexpr int W_THREADS = W_WAVES * 64;
constexpr int W_ROWS = W_WAVES * RB;            // rows per workgroup round
constexpr int W_CMAX = 32;                      // d <= 256
constexpr int W_RESIDENT_BYTES = 63 * 1024;     // fragment tables kept whole in LDS
constexpr int W_STREAM_BYTES = 30720;           // one staging buffer when streamed
constexpr int W_SREG = (W_STREAM_BYTES / 16 + W_THREADS - 1) / W_THREADS;  // staged u4 per thread
constexpr int W_ACC_LDS_BYTES = 98304;          // accumulator slice in LDS
constexpr int W_ACC_BATCH = 4;                  // rows per thread per collection pass
constexpr int W_ACC_MEMBERS = 8;                // member rows per lane group in flight
constexpr int W_BUCKET_KMAX = 16384;            // codewords the bucketing histogram holds
// Sorted sums: a codeword's wave takes its first W_SORT_Q members; the rest of
// the bucketed rows is cut into windows of W_SORT_Q positions, each summed by
// a wave of its own (a window meets the overflow of at most one codeword:
// two overflows are at least W_SORT_Q positions apart)
constexpr int W_SORT_Q = 128;
__host__ __device__ inline int w_sort_windows(int64_t N) {
  return (int)((N + W_SORT_Q - 1) / W_SORT_Q);
}
constexpr int W_FUSED_ROUNDS = 4;               // row rounds a stage-fused encode workgroup keeps
constexpr int W_DEC_TABLE_BYTES = 131072;        // codeword table per workgroup, at most
constexpr int W_DEC_LDS_BYTES = 152 * 1024;      // table + staged code words
constexpr int W_DEC_CODE_PT = 16;               // staged code words per thread, at most
constexpr int W_DEC_THREADS = 1024;

enum { W_TRAIN = 0, W_ENCODE = 1 };

// Group pairs of a subvector: lane half h holds group 2p + h of pair p.
__host__ __device__ constexpr int w_pairs(int C) { return (C + 1) / 2; }
// Fragments per tile: HI_p, LO_p for every pair, then the bias fragment.
__host__ __device__ constexpr int w_frags(int C) { return 2 * w_pairs(C) + 1; }
// Row blocks a wave scores per round: two for the streamed single pass
// while their operands fit the register budget (d <= 128), else one.
__host__ __device__ constexpr int w_row_blocks(int C, bool resident, bool sp, bool ind) {
  return (sp && !ind && !resident && C <= 16) ? 2 : 1;
}
// Staged u4 per thread of a streamed chunk: a chunk holds at least one whole
// tile (33 fragments at d = 256 exceed the W_STREAM_BYTES budget).
__host__ __device__ constexpr int w_sreg(int C) {
  return W_SREG > (w_frags(C) * 64 + W_THREADS - 1) / W_THREADS
             ? W_SREG
             : (w_frags(C) * 64 + W_THREADS - 1) / W_THREADS;
}
static_assert(w_sreg(W_CMAX) * W_THREADS >= w_frags(W_CMAX) * 64, "staging holds one tile");
// Waves of a scoring workgroup.  With a streamed table at d <= 128 (the
// hi/lo pass, the single pass and the pass over listed rows) it runs four:
// each workgroup then scores one round of rows and streams the table once
// for them, and two or three workgroups share a CU, so that one's row loads
// and barriers overlap another's MFMAs (eight-wave workgroups held a CU
// alone).  Resident tables keep eight.
__host__ __device__ constexpr int w_score_waves(int C, bool resident, bool sp, bool ind) {
  return (!resident && C <= 16) ? 4 : W_WAVES;
}
// Tiles per streamed chunk of the hi/lo pass, and the staged u4 per thread
// for a workgroup of nth threads.
__host__ __device__ constexpr int w_stream_tiles(int C) {
  return W_STREAM_BYTES / (w_frags(C) * 1024) > 1 ? W_STREAM_BYTES / (w_frags(C) * 1024) : 1;
}
__host__ __device__ constexpr int w_sreg_n(int C, int nth) {
  return (w_stream_tiles(C) * w_frags(C) * 64 + nth - 1) / nth;
}
// The single pass stages P + 1 fragments per tile through larger chunks
// (fewer barriers per round); two workgroups per CU still fit in LDS.
constexpr int W_SP_STREAM_BYTES = 36864;
// a four-wave single-pass workgroup stages half-size chunks (five staged
// u4 per thread; full-size ones measured no faster and spill in one
// instantiation); its registers allow two such workgroups per CU
__host__ __device__ constexpr int w_sp_stream_bytes(int nw) {
  return nw == W_WAVES ? W_SP_STREAM_BYTES : W_SP_STREAM_BYTES / 2;
}
__host__ __device__ constexpr int w_sp_sreg_n(int C, int nw) {
  return (w_sp_stream_bytes(nw) / 16 + nw * 64 - 1) / (nw * 64) >
                 ((w_pairs(C) + 1) * 64 + nw * 64 - 1) / (nw * 64)
             ? (w_sp_stream_bytes(nw) / 16 + nw * 64 - 1) / (nw * 64)
             : ((w_pairs(C) + 1) * 64 + nw * 64 - 1) / (nw * 64);
}
__host__ __device__ constexpr int w_sp_sreg(int C) {
  return (W_SP_STREAM_BYTES / 16 + W_THREADS - 1) / W_THREADS >
                 ((w_pairs(C) + 1) * 64 + W_THREADS - 1) / W_THREADS
             ? (W_SP_STREAM_BYTES / 16 + W_THREADS - 1) / W_THREADS
             : ((w_pairs(C) + 1) * 64 + W_THREADS - 1) / W_THREADS;
}

// ------------------------------------------------------------------ kernels

// Per-codebook state the fragment launch writes besides the tables: smallest
// gain and largest gain ([2][ncb]), and the deferred-row counters it clears.
struct WDeferPtrs {
  float* gmin;
  int* xcount;
  int* xchanged;
  double* xobj;
  int* hcount;   // null: no single pass
};

// Operand fragments of one 32-codeword tile (grid: tiles x codebooks, one
// wave).  Lane = codeword c (0..31) + 32 h; lane half h covers the 8-element
// group 2p + h of pair p.  With a_j = -2 g s_j 2^SA / sigma and
// gg = (g / sigma)^2 2^SA, the tile's fragments are, per lane, in order:
//   HI_p (p < P)   hi(a[16p + 8h, 16p + 8h + 8))
//   bias           h0 [hi(gg) lo(gg) 2^SA 2^SA 0 0 0 0], h1 zero
//   LO_p (p < P)   lo(a[16p + 8h, 16p + 8h + 8))
// so the single-pass scoring kernel stages the first P + 1 of them only.
// Padding codewords (k >= K) have a = 0 and a float16-max g^2 slot.  P is
// a template argument so that all of a lane's shape loads are issued
// together (a runtime pair loop waited for each pair's loads in turn).
template <int P>
__global__ void __launch_bounds__(64) w_frag_kernel(const float* __restrict__ gain,
                                                    const float* __restrict__ shape, int d, int K,
                                                    int unit_gain, int* __restrict__ sig,
                                                    const int* __restrict__ done, int G, int cb0,
                                                    u4* __restrict__ frag, WDeferPtrs X) {
  const int t = blockIdx.x, tiles = gridDim.x;
  const int cbl = blockIdx.y, cb = cb0 + cbl;
  if (done && done[cbl % G]) return;
  const int lane = threadIdx.x, c = lane & 31, h = lane >> 5;
  const int k = t * CW + c;
  const bool real = k < K;
  const int kk = real ? k : K - 1;
  const float g = real ? (unit_gain ? 1.f : gain[(size_t)cb * K + kk]) : 0.f;
  const float* s = shape + ((size_t)cb * K + kk) * d;
  // sigma (from the largest gain) and the smallest gain, found by every
  // wave of the codebook (max and min are exact in any order, so all agree);
  // the wave of tile 0 records them and clears the deferred-row state
  float m = 0.f, n = INFINITY;
  for (int q0 = 0; q0 < K; q0 += 8 * 64) {
    // eight loads in flight per lane; indexes past K repeat gain K - 1,
    // which changes neither extreme
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int q = min(q0 + 64 * u + lane, K - 1);
      v[u] = unit_gain ? 1.f : gain[(size_t)cb * K + q];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      m = fmaxf(m, v[u]);
      n = fminf(n, v[u]);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    m = fmaxf(m, __shfl_xor(m, off));
    n = fminf(n, __shfl_xor(n, off));
  }
  const int ex = sigma_exp(m);
  if (t == 0 && lane == 0) {
    sig[cb] = ex;
    X.gmin[cbl] = n;
    X.gmin[gridDim.y + cbl] = m;
    X.xcount[cbl] = 0;
    X.xchanged[cbl] = 0;
    X.xobj[cbl] = 0.0;
    if (X.hcount) X.hcount[cbl] = 0;
  }
  u4* out = frag + ((size_t)cbl * tiles + t) * (2 * P + 1) * 64;
  float sv[P][8];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int e = 16 * p + 8 * h + j;
      sv[p][j] = s[min(e, d - 1)];            // in bounds; masked below
    }
#pragma unroll
  for (int p = 0; p < P; ++p) {
    _Float16 hi[8], lo[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int e = 16 * p + 8 * h + j;
      const float av = ldexpf(-2.f * g * ((real && e < d) ? sv[p][j] : 0.f), SA - ex);
      hi[j] = (_Float16)av;
      lo[j] = (_Float16)(av - (float)hi[j]);
    }
    out[p * 64 + lane] = pack_h8(hi);
    out[(P + 1 + p) * 64 + lane] = pack_h8(lo);
  }
  const float gs = ldexpf(g, -ex);
  const float gg = ldexpf(gs * gs, SA);
  out[P * 64 + lane] = h ? (u4){0u, 0u, 0u, 0u} : bias_codeword(real, gg);
}

// Seed shapes s_k = x_r / (||x_r|| + eps) from rows of the row-major input.
// K-means seeding (kmeans != 0): the centroid is the seed row itself, held
// as gain ||x_r|| and shape x_r / ||x_r|| (0 for a zero row).
template <typename T>
__global__ void w_seed_kernel(const T* __restrict__ X, int64_t ldx, int d, int K,
                              const int32_t* __restrict__ seeds, float* __restrict__ shape,
                              float* __restrict__ seednorm, int kmeans,
                              float* __restrict__ gain) {
  const int g = blockIdx.y;
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  const int64_t row = seeds[(size_t)g * K + k];
  const T* x = X + row * ldx + (int64_t)g * d;
  double ss = 0.0;
  for (int j = 0; j < d; ++j) { const double v = to_f(x[j]); ss = fma(v, v, ss); }
  const double nrm = sqrt(ss);
  const double den = kmeans ? (nrm > 0.0 ? nrm : 1.0) : nrm + (double)Y_EPS;
  float* sk = shape + ((size_t)g * K + k) * d;
  for (int j = 0; j < d; ++j) sk[j] = (float)((double)to_f(x[j]) / den);
  seednorm[(size_t)g * K + k] = (float)nrm;
  if (kmeans) gain[(size_t)g * K + k] = (float)nrm;
}

struct WScoreArgs {
  const void* x;          // stage input rows [N][ldx]
  int64_t ldx, N;
  int d, K, G, tiles, QF;
  int cb0;                // codebook index (gain, shape, sig) of subspace 0: m G
  int fcb0;               // codebook index of fragment-table entry 0
  const u4* frag;         // [ncb][tiles][QF][64]
  const float* gmin;      // [ncb] smallest gain (same indexing as frag), then [ncb] largest
  int* xcount;            // [G] rows deferred to the exact kernel (reset with sigma)
  int* xrows;             // [G][N] their row indices
  int* xchanged;          // [G] exact kernel: some deferred row changed code
  double* xobj;           // [G] exact kernel: their weighted distortion
  int* hcount;            // [G] rows the single pass lists for the hi/lo pass
  int* hrows;             // [G][N] their row indices
  unsigned long long* hbest;  // [G][N] hi/lo pass: best (distance key, codeword) per listed row
  float* hrr;             // [G][N] hi/lo pass: the row term rr, or -1 if it needs float64
  int nslice, tps;        // hi/lo pass: tile slices and tiles per slice
  const int* sig;         // [ncb]
  const float* gain;      // [ncb][K]
  const float* shape;     // [ncb][K][d]
  int unit_gain;          // score with unit gains (equal-gain initial assignment)
  // training outputs
  const float* w;         // [N] or null (all ones)
  const int* done;        // [G] or null
  uint16_t* assign;       // [G][N]: old assignment in, new one out
  int* changed;           // [G][nwg]
  double* obj;            // [G][nwg] or null
  // encode outputs
  uint32_t* codes;        // [N][words], zeroed beforehand, or null
  int words, b, m;
  float* res_out;         // [N][G d] float32 residual or null
  // launch geometry
  int nwg, rounds, tpc, map_xcd, lg;
};

// Raw elements of this lane's half of a row: the groups 2p + h (elements
// [16p + 8h, 16p + 8h + 8)), in the stage input's type.  The loads never
// branch (indices clamped into the subvector, values masked later), so a
// prefetch stays in flight.
template <typename T, int P> struct WRaw {
  static constexpr int NV = sizeof(T) == 2 ? P : 2 * P;
  u4 v[NV];
  __device__ __forceinline__ void load(const T* xp, int d, bool vec, int h) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int e0 = 16 * p + 8 * h;
      if (vec) {
        // a lone last group (d = 8) leaves lane half 1 empty: read group 0
        const int q = e0 < d ? 2 * p + h : 0;
        if (sizeof(T) == 2) {
          v[p] = ((const u4*)xp)[q];
        } else {
          v[2 * p] = ((const u4*)xp)[2 * q];
          v[2 * p + 1] = ((const u4*)xp)[2 * q + 1];
        }
      } else {
        T t[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) t[j] = xp[min(e0 + j, d - 1)];
        if (sizeof(T) == 2) {
          v[p] = *(const u4*)t;
        } else {
          v[2 * p] = ((const u4*)t)[0];
          v[2 * p + 1] = ((const u4*)t)[1];
        }
      }
    }
  }
  // element j of pair p (as float), zero past d or for an invalid row
  __device__ __forceinline__ float at(int p, int j, int d, int h, bool valid) const {
    const int e = 16 * p + 8 * h + j;
    float x;
    if (sizeof(T) == 2) {
      const uint32_t w = v[p][j >> 1];
      x = (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> (16 * (j & 1))));
    } else {
      x = __uint_as_float(v[2 * p + (j >> 2)][j & 3]);
    }
    return (valid && e < d) ? x : 0.f;
  }
};

// Row-side operands of one row (this lane's row) for all tiles, built from
// the raw elements; lane half h holds the groups 2p + h.
// F16 rows (the exact float16 stage input, rho = 1):
//   bx[p] = x of the group;  bias (h0) [sigma sigma hi(rr) lo(rr) 0 0 0 0],
//   rr = ||x||^2 / sigma, giving D = 2^SA dist / sigma.
// F32 rows: rho = 2^er >= max|x|, b = x 2^SB / rho:
//   bx[p] = hi(b), blo[p] = lo(b) of the group,
//   bias (h0) [2^SB sigma / rho (twice) hi(rr) lo(rr) 0 0 0 0],
//   rr = 2^SB ||x||^2 / (sigma rho), giving D = 2^(SA+SB) dist / (sigma rho).
// need_exact flags rows whose operands leave the float16 range.
template <typename T, int P>
__device__ __forceinline__ void w_make_b(const WRaw<T, P>& raw, int d, bool valid, int ex, int h,
                                         u4 (&bx)[P], u4 (&blo)[P], u4& bias, float& rr,
                                         bool& need_exact, float& eD) {
  constexpr bool F16 = sizeof(T) == 2;
  int sr;
  if (F16) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    float ss = 0.f;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const bool live = valid && 16 * p + 8 * h < d;   // d is a multiple of 8
      bx[p] = live ? raw.v[p] : (u4){0u, 0u, 0u, 0u};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // copy the element first: a bit_cast of a vector element reads the
        // wrong element with this compiler
        const uint32_t wj = bx[p][j];
        const h2 v2 = __builtin_bit_cast(h2, wj);
        ss = __builtin_amdgcn_fdot2(v2, v2, ss, false);
      }
    }
    ss += __shfl_xor(ss, 32);
    sr = ex;
    rr = ldexpf(ss, -ex);
    need_exact = ex > 15 || ex < -14 || !(rr < 32768.f);
    // single-pass error bound in D units: 2^-10 g ||x|| 2^SA / sigma, g <= sigma
    eD = ldexpf(sqrtf(ss), SA - 10) * (1.f + 0x1p-9f);
  } else {
    float mx = 0.f, ss = 0.f;
#pragma unroll
    for (int p = 0; p < P; ++p)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float v = raw.at(p, j, d, h, valid);
        mx = fmaxf(mx, fabsf(v));
        ss = fmaf(v, v, ss);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    ss += __shfl_xor(ss, 32);
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
    // single-pass error bound in D units: 2^-9 g ||x|| 2^(SA+SB) / (sigma rho)
    eD = ldexpf(sqrtf(ss), SA + SB - 9 - er) * (1.f + 0x1p-9f);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      _Float16 hi[8], lo[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float v = ldexpf(raw.at(p, j, d, h, valid), SB - er);
        hi[j] = (_Float16)v;
        lo[j] = (_Float16)(v - (float)hi[j]);
      }
      bx[p] = pack_h8(hi);
      blo[p] = pack_h8(lo);
    }
  }
  rr = fminf(rr, 32768.f);
  sr = sr < -14 ? -14 : (sr > 15 ? 15 : sr);
  bias = h ? (u4){0u, 0u, 0u, 0u} : bias_row(sr, rr);
}

// Elements [e0, e0 + 8) of a float32 row as float (zero past d or for an
// invalid row): two vector loads when vec (d a multiple of 8, 16-byte
// aligned), else element loads with clamped indices.
__device__ __forceinline__ void w_row_group(const float* xp, int e0, int d, bool vec, bool valid,
                                            float (&xv)[8]) {
  const bool live = valid && e0 < d;
  if (vec) {
    const int q = e0 < d ? e0 : 0;   // a lone last group (d = 8): read group 0
    const f4 a = *(const f4*)(xp + q), b = *(const f4*)(xp + q + 4);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      xv[u] = live ? a[u] : 0.f;
      xv[4 + u] = live ? b[u] : 0.f;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int e = e0 + j;
      xv[j] = (valid && e < d) ? xp[e < d ? e : 0] : 0.f;
    }
  }
}
__device__ __forceinline__ void w_row_group(const _Float16* xp, int e0, int d, bool vec,
                                            bool valid, float (&xv)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int e = e0 + j;
    xv[j] = (valid && e < d) ? (float)xp[e < d ? e : 0] : 0.f;
  }
}

// The same operands loaded straight from memory (no prefetch): fewer live
// registers for wide rows, where a workgroup scores a single round.
template <typename T, int P>
__device__ __forceinline__ void w_make_b_direct(const T* xp, int d, bool vec, bool valid, int ex, int h,
                                         u4 (&bx)[P], u4 (&blo)[P], u4& bias, float& rr,
                                         bool& need_exact, float& eD) {
  constexpr bool F16 = sizeof(T) == 2;
  int sr;
  if constexpr (F16) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    float ss = 0.f;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int e0 = 16 * p + 8 * h;
      if (vec) {
        // a lone last group (d = 8) leaves lane half 1 empty
        bx[p] = e0 < d ? ((const u4*)xp)[2 * p + h] : (u4){0u, 0u, 0u, 0u};
      } else {
        _Float16 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = e0 + j < d ? (_Float16)xp[e0 + j] : (_Float16)0.f;
        bx[p] = pack_h8(v);
      }
      if (!valid) bx[p] = (u4){0u, 0u, 0u, 0u};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // copy the element first: a bit_cast of a vector element reads the
        // wrong element with this compiler
        const uint32_t wj = bx[p][j];
        const h2 v2 = __builtin_bit_cast(h2, wj);
        ss = __builtin_amdgcn_fdot2(v2, v2, ss, false);
      }
    }
    ss += __shfl_xor(ss, 32);
    sr = ex;
    rr = ldexpf(ss, -ex);
    need_exact = ex > 15 || ex < -14 || !(rr < 32768.f);
    // single-pass error bound in D units: 2^-10 g ||x|| 2^SA / sigma, g <= sigma
    eD = ldexpf(sqrtf(ss), SA - 10) * (1.f + 0x1p-9f);
  } else if constexpr (P <= 8) {
    // pass 1: the row's scale, from vector loads (element loads came back a
    // few at a time and made this the slowest part of a float32-row launch)
    float mx = 0.f, ss = 0.f;
    // the vector / element choice is made once per pass, so that a pass's
    // loads share one basic block and are issued together
    auto scale_pass = [&](auto vec_c) {
#pragma unroll
      for (int p = 0; p < P; ++p) {
        float xv[8];
        w_row_group(xp, 16 * p + 8 * h, d, decltype(vec_c)::value, valid, xv);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          mx = fmaxf(mx, fabsf(xv[j]));
          ss = fmaf(xv[j], xv[j], ss);
        }
        // at most four groups' loads in flight (bounds the registers)
        if (p % 4 == 3) asm volatile("" ::: "memory");
      }
    };
    if (vec) scale_pass(std::true_type{});
    else scale_pass(std::false_type{});
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    ss += __shfl_xor(ss, 32);
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
    // single-pass error bound in D units: 2^-9 g ||x|| 2^(SA+SB) / (sigma rho)
    eD = ldexpf(sqrtf(ss), SA + SB - 9 - er) * (1.f + 0x1p-9f);
    // pass 2 re-reads the row (cache hits): holding pass 1's values across
    // the reduction would take 8 P registers per row block
    asm volatile("" ::: "memory");
    auto split_pass = [&](auto vec_c) {
#pragma unroll
      for (int p = 0; p < P; ++p) {
        float xv[8];
        w_row_group(xp, 16 * p + 8 * h, d, decltype(vec_c)::value, valid, xv);
        _Float16 hi[8], lo[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float v = ldexpf(xv[j], SB - er);
          hi[j] = (_Float16)v;
          lo[j] = (_Float16)(v - (float)hi[j]);
        }
        bx[p] = pack_h8(hi);
        blo[p] = pack_h8(lo);
        if (p % 4 == 3) asm volatile("" ::: "memory");
      }
    };
    if (vec) split_pass(std::true_type{});
    else split_pass(std::false_type{});
    } else {
    // wider rows (d = 256): element loads keep the registers of a pass low
    // pass 1: the row's scale; pass 2 re-reads the (cached) row and splits it
    float mx = 0.f, ss = 0.f;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int e0 = 16 * p + 8 * h;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int e = e0 + j;
        const float v = (valid && e < d) ? (float)xp[e < d ? e : 0] : 0.f;
        mx = fmaxf(mx, fabsf(v));
        ss = fmaf(v, v, ss);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    ss += __shfl_xor(ss, 32);
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
    // single-pass error bound in D units: 2^-9 g ||x|| 2^(SA+SB) / (sigma rho)
    eD = ldexpf(sqrtf(ss), SA + SB - 9 - er) * (1.f + 0x1p-9f);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int e0 = 16 * p + 8 * h;
      _Float16 hi[8], lo[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int e = e0 + j;
        const float x = (valid && e < d) ? (float)xp[e < d ? e : 0] : 0.f;
        const float v = ldexpf(x, SB - er);
        hi[j] = (_Float16)v;
        lo[j] = (_Float16)(v - (float)hi[j]);
      }
      bx[p] = pack_h8(hi);
      blo[p] = pack_h8(lo);
    }
    }
  rr = fminf(rr, 32768.f);
  sr = sr < -14 ? -14 : (sr > 15 ? 15 : sr);
  bias = h ? (u4){0u, 0u, 0u, 0u} : bias_row(sr, rr);
}

// Distances of one tile: the MFMA chain over the tile's fragments at `ta`
// (this lane's entry of fragment 0; fragments are 64 u4 apart).  Per pair:
// hi(a) x + lo(a) x (float16 rows) or hi(a) hi(b) + lo(a) hi(b) + hi(a) lo(b)
// (float32 rows); then the bias terms.
template <bool F16, int P>
__device__ __forceinline__ f16v w_tile(const u4* ta, const u4 (&bx)[P], const u4 (&blo)[P],
                                       u4 bias) {
  // the fragments of pair p + AH are read while pair p's MFMAs run (with
  // the reads next to their MFMAs, two read registers exposed an LDS round
  // trip every two or three MFMAs)
  constexpr int AH = P < 2 ? P : 2;
  u4 fh[P], fl[P], fb;
#pragma unroll
  for (int q = 0; q < AH; ++q) {
    fh[q] = ta[q * 64];
    fl[q] = ta[(P + 1 + q) * 64];
  }
  if (AH == P) fb = ta[P * 64];
  f16v acc = {};
#pragma unroll
  for (int p = 0; p < P; ++p) {
    if (p + AH < P) {
      fh[p + AH] = ta[(p + AH) * 64];
      fl[p + AH] = ta[(P + 1 + p + AH) * 64];
    } else if (p + AH == P && AH < P) {
      fb = ta[P * 64];
    }
    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(fh[p]), as_h8(bx[p]), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(fl[p]), as_h8(bx[p]), acc, 0, 0, 0);
    if (!F16) acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(fh[p]), as_h8(blo[p]), acc, 0, 0, 0);
  }
  acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(fb), as_h8(bias), acc, 0, 0, 0);
  // the schedule: the first AH pairs' reads, then per pair its MFMAs and two
  // reads ahead (left alone the scheduler moves each read next to its MFMA)
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * AH, 0);
#pragma unroll
  for (int p = 0; p < P; ++p) {
    __builtin_amdgcn_sched_group_barrier(0x008, F16 ? 2 : 3, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  return acc;
}

// Single-pass distances of one tile: hi(a) against the row's float16
// operand (the row itself, or hi(b) of a float32 row) per pair, then the
// bias terms (P + 1 MFMAs instead of 2P + 1 or 3P + 1).  The dropped lo
// parts bound the error: |D~ - D| <= 2^-10 (1 + 2^-11) sum |a_j b_j| for
// float16 rows, 2^-9 (1 + 2^-12) sum |a_j b_j| for float32 rows.
template <int P>
__device__ __forceinline__ f16v w_tile_sp(const u4* ta, const u4 (&bx)[P], u4 bias) {
  f16v acc = {};
#pragma unroll
  for (int p = 0; p < P; ++p)
    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(ta[p * 64]), as_h8(bx[p]), acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(ta[P * 64]), as_h8(bias), acc, 0, 0, 0);
}

// Single-pass distances of one tile for two row blocks: each fragment is
// read from LDS once and feeds both blocks' MFMA chains, which halves the
// LDS traffic per MFMA (with one block per wave the fragment reads alone
// would take the whole LDS bandwidth at full MFMA rate).
template <int P>
__device__ __forceinline__ void w_tile_sp2(const u4* ta, const u4 (&bx0)[P], const u4 (&bx1)[P],
                                           u4 bias0, u4 bias1, f16v& c0, f16v& c1) {
  f16v a0 = {}, a1 = {};
  // fragment p + 1 is read while fragment p's two MFMAs run (one read
  // register set alone would expose every LDS read's latency)
  h8 f = as_h8(ta[0]);
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const h8 fn = as_h8(ta[(p + 1) * 64]);
    a0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(f, as_h8(bx0[p]), a0, 0, 0, 0);
    a1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(f, as_h8(bx1[p]), a1, 0, 0, 0);
    f = fn;
  }
  c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(f, as_h8(bias0), a0, 0, 0, 0);
  c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(f, as_h8(bias1), a1, 0, 0, 0);
}

// Smallest packed key of a tile: the low 4 bits of each distance carry its
// slot j (lane l holds codewords 8 (j / 4) + 4 h + j % 4 of row l % 32).
__device__ __forceinline__ int w_tile_key(const f16v& c) {
  constexpr int MASK = ~15;
  int m = min3i((__float_as_int(c[0]) & MASK) | 0, (__float_as_int(c[1]) & MASK) | 1,
                (__float_as_int(c[2]) & MASK) | 2);
#pragma unroll
  for (int j = 3; j < 15; j += 2)
    m = min3i(m, (__float_as_int(c[j]) & MASK) | j, (__float_as_int(c[j + 1]) & MASK) | (j + 1));
  return min(m, (__float_as_int(c[15]) & MASK) | 15);
}

// Running best over tiles in increasing order: a later tile replaces the
// best only with a strictly smaller distance, so ties keep the lower index.
__device__ __forceinline__ void w_take(int key, int t, int& best, int& bt) {
  if (key < (best & ~15)) { best = key; bt = t; }
}

__device__ __forceinline__ int med3i(int a, int b, int c) {
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// The two smallest packed keys of a tile (b <= s), streamed: each key
// moves the second smallest to med3(b, s, key) and the smallest to
// min(b, key).
__device__ __forceinline__ void w_tile_key2(const f16v& c, int& b, int& s) {
  constexpr int MASK = ~15;
  const int k0 = __float_as_int(c[0]) & MASK, k1 = (__float_as_int(c[1]) & MASK) | 1;
  b = min(k0, k1);
  s = max(k0, k1);
#pragma unroll
  for (int j = 2; j < 16; ++j) {
    const int k = (__float_as_int(c[j]) & MASK) | j;
    s = med3i(b, s, k);
    b = min(b, k);
  }
}

// Running best (with its tile) and second-smallest key over tiles: the
// second smallest of {best, second, b, s} is med3(best, b, min(second, s))
// when best <= second and b <= s.
__device__ __forceinline__ void w_take2(int b, int s, int t, int& best, int& bt, int& second) {
  second = med3i(best, b, min(second, s));
  w_take(b, t, best, bt);
}

// Staging of a chunk of fragment tiles: thread slot r holds element
// e = r W_THREADS + tid of the chunk, i.e. entry o of its tile tr (both
// fixed per thread, computed once).  The loads never branch: a slot past
// the chunk's last tile reads that tile again and is never stored, so the
// loads stay in flight while the current chunk is scored.
template <int QU, int SR, int NTH = W_THREADS> struct WStage {
  int tr[SR], o[SR];
  __device__ __forceinline__ WStage() {
#pragma unroll
    for (int r = 0; r < SR; ++r) {
      const int e = r * NTH + (int)threadIdx.x;
      tr[r] = e / (QU * 64);
      o[r] = e - tr[r] * (QU * 64);
    }
  }
  __device__ __forceinline__ void load(const u4* ftab, int QF, int t0, int nt,
                                       u4 (&reg)[SR]) const {
#pragma unroll
    for (int r = 0; r < SR; ++r)
      reg[r] = ftab[(uint32_t)((t0 + min(tr[r], nt - 1)) * QF * 64 + o[r])];
  }
};
template <int SR, int NTH = W_THREADS>
__device__ __forceinline__ void w_stage_store(u4* buf, int n, const u4 (&reg)[SR]) {
#pragma unroll
  for (int r = 0; r < SR; ++r) {
    const int e = r * NTH + (int)threadIdx.x;
    if (e < n) buf[e] = reg[r];
  }
}

// Four consecutive elements of a stage-input row as float32 (vector load:
// 16 bytes of float32, 8 bytes of float16).
__device__ __forceinline__ f4 w_load4(const float* p) { return *(const f4*)p; }
__device__ __forceinline__ f4 w_load4(const _Float16* p) {
  typedef _Float16 h4 __attribute__((ext_vector_type(4)));
  const h4 v = *(const h4*)p;
  return (f4){(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}

// Residual r = x - g s over n consecutive elements (a lane half's share of
// a row), written to dst when dst is non-null; returns ||r||^2 (float32).
// vec: n % 4 == 0 and x, s, dst 16-byte (float16 x: 8-byte) aligned, so
// every access is a vector access; otherwise element by element.
template <typename T, bool BATCH = false>
__device__ __forceinline__ float w_residual(const T* xp, const float* sk, float gk, int n,
                                            bool vec, float* dst) {
  float dist = 0.f;
  if (vec) {
    int j0 = 0;
    if constexpr (BATCH) {
      // eight vector loads of each operand in flight per batch (one load
      // pair per iteration waited for each pair in turn: the encode
      // epilogue's slowest part)
      for (; j0 + 32 <= n; j0 += 32) {
        f4 x[8], sv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          x[u] = w_load4(xp + j0 + 4 * u);
          sv[u] = *(const f4*)(sk + j0 + 4 * u);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          f4 r;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            r[q] = fmaf(-gk, sv[u][q], x[u][q]);
            dist = fmaf(r[q], r[q], dist);
          }
          if (dst) *(f4*)(dst + j0 + 4 * u) = r;
        }
      }
    }
    for (int j = j0; j < n; j += 4) {
      const f4 x = w_load4(xp + j), sv = *(const f4*)(sk + j);
      f4 r;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        r[u] = fmaf(-gk, sv[u], x[u]);
        dist = fmaf(r[u], r[u], dist);
      }
      if (dst) *(f4*)(dst + j) = r;
    }
  } else {
    for (int j = 0; j < n; ++j) {
      const float r = fmaf(-gk, sk[j], (float)xp[j]);
      dist = fmaf(r, r, dist);
      if (dst) dst[j] = r;
    }
  }
  return dist;
}

// Writes code k into the b-bit field at `bit` of a row's words (zeroed
// beforehand): byte and half-word fields are stored, others OR'd in.
__device__ __forceinline__ void w_put_code(uint32_t* wp, int64_t bit, int b, int k) {
  if (b == 8) {
    ((uint8_t*)wp)[bit >> 3] = (uint8_t)k;
  } else if (b == 16) {
    ((uint16_t*)wp)[bit >> 4] = (uint16_t)k;
  } else {
    const int off = (int)(bit & 31);
    atomicOr(wp + (bit >> 5), (uint32_t)k << off);
    if (off + b > 32) atomicOr(wp + (bit >> 5) + 1, (uint32_t)k >> (32 - off));
  }
}

// Scoring kernel: assignment (eq. 5) of every row of a chunk for one
// subspace, then the mode's outputs (training: assignment, changed flag,
// objective; encode: code bits and residual).  Grid: G x nwg workgroups,
// numbered so that subspaces whose rows share cache lines run on one XCD.
// Waves per SIMD: four (two workgroups per CU) with a resident table and
// narrow rows; two when d >= 64 (row operands up to 68 VGPRs) or when the
// table is streamed (staging registers).
// SP (single pass, d >= 64): P + 1 MFMAs per tile on the float16 operands
// (w_tile_sp); the two smallest keys of every row are kept, and a row whose
// second-best distance lies within twice the error bound of its best (or
// whose keys cannot separate a 1e-4 margin) is listed for the hi/lo pass
// instead of being decided here.
// IND (indirect, the hi/lo pass after SP): the rows are the subspace's
// listed ones (hrows, hcount) and the codebook is split into slices of tps
// tiles, each kept whole in LDS by its workgroups; workgroup (g, slice, r0)
// scores rounds r0, r0 + nwg, ... of the list against its slice and merges
// every row's best (distance key, codeword) into hbest with a 64-bit
// atomic minimum (lowest codeword on equal keys); w_listed_finish_kernel
// then writes the outputs.
template <typename T, int C, int MODE, bool RESIDENT, bool SP, bool IND>
__global__ void __launch_bounds__(w_score_waves(C, RESIDENT, SP, IND) * 64, (RESIDENT && C <= 4) ? 4 : 2)
    w_score_kernel(WScoreArgs a) {
  constexpr int NW = w_score_waves(C, RESIDENT, SP, IND);
  constexpr int NTH = NW * 64;
  constexpr int WR = NW * RB;   // rows of a round per row block of the waves
  extern __shared__ __align__(16) u4 wtab[];
  __shared__ double red_obj[NW];
  __shared__ int red_changed;
  constexpr bool F16 = sizeof(T) == 2;
  constexpr int P = w_pairs(C);
  constexpr int QU = SP ? P + 1 : w_frags(C);
  // R row blocks per wave and round (two for the streamed single pass:
  // every fragment read from LDS feeds two MFMAs); with one, two tiles'
  // MFMA chains in flight, and the next round's row prefetched, while the
  // row operands are small enough to leave registers for both
  constexpr int R = w_row_blocks(C, RESIDENT, SP, IND);
  constexpr bool PAIR_TILES = (C <= 4 || SP) && R == 1;
  constexpr bool PREFETCH = C <= 2 && !IND;
  static_assert(!PREFETCH || R == 1, "the row prefetch holds one row block");

  int g, rc, slice = 0;
  {
    const int id = blockIdx.x;
    if (IND) {
      g = id % a.G;
      slice = (id / a.G) % a.nslice;
      rc = id / (a.G * a.nslice);
    } else if (a.map_xcd) {
      const int xcd = id & 7, slot = id >> 3, gpx = a.G >> 3;
      const int j = slot % gpx;
      rc = slot / gpx;
      g = ((j / a.lg) * 8 + xcd) * a.lg + (j % a.lg);
    } else {
      g = id % a.G;
      rc = id / a.G;
    }
  }
  if (a.done && a.done[g]) return;
  // indirect rows: this workgroup takes rounds rc, rc + nwg, ... of the list
  const int hcnt = IND ? a.hcount[g] : 0;
  if (IND && rc * WR >= hcnt) return;
  const int nrounds = IND ? (hcnt - rc * WR + a.nwg * WR - 1) / (a.nwg * WR)
                          : a.rounds;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = lane & 31, h = lane >> 5;
  const int d = a.d, K = a.K;
  // this workgroup's tiles: all, or (IND) its slice
  const int tb = IND ? slice * a.tps : 0;
  const int tiles = IND ? min(a.tiles - tb, a.tps) : a.tiles;
  const int cb = a.cb0 + g;
  const int ex = a.sig[cb];
  const u4* ftab = a.frag + ((size_t)(cb - a.fcb0) * a.tiles + tb) * a.QF * 64;
  const float* gcb = a.gain + (size_t)cb * K;
  const float* scb = a.shape + (size_t)cb * K * d;
  const T* X = (const T*)a.x;
  const bool vec = (d == 8 * C) && ((a.ldx * (int64_t)sizeof(T)) % 16 == 0) &&
                   (((uintptr_t)X) % 16 == 0);
  // vector accesses in the residual / objective epilogue: row, codeword and
  // residual output aligned (d is a multiple of 8)
  const bool rvec = vec && (((uintptr_t)scb) % 16 == 0) &&
                    (a.res_out == nullptr || ((uintptr_t)a.res_out) % 16 == 0);
  if (tid == 0) red_changed = 0;
  if (RESIDENT) {
    const int n = tiles * QU * 64;
    for (int e = tid; e < n; e += NTH) {
      const int t = e / (QU * 64), o = e - t * (QU * 64);
      wtab[e] = ftab[(size_t)t * a.QF * 64 + o];
    }
  }
  __syncthreads();

  double obj = 0.0;
  bool any_changed = false;
  // this lane's row of round rd, row block r of the wave (valid: below N,
  // or within the list)
  auto row_of = [&](int rd, int r, bool& valid) -> int64_t {
    if (IND) {
      const int idx = (rc + rd * a.nwg) * WR + wave * RB + i;
      valid = idx < hcnt;
      return a.hrows[(size_t)g * a.N + (valid ? idx : 0)];
    }
    const int64_t row = ((int64_t)rc * a.rounds + rd) * (WR * R) +
                        (int64_t)(wave * R + r) * RB + i;
    valid = row < a.N;
    return row;
  };
  auto row_ptr = [&](int64_t row) -> const T* {
    return X + (row < a.N ? row : 0) * a.ldx + (int64_t)g * d;
  };
  WRaw<T, P> raw;
  if (PREFETCH) {
    bool v0;
    raw.load(row_ptr(row_of(0, 0, v0)), d, vec, h);
  }
  for (int rd = 0; rd < nrounds; ++rd) {
    bool valid[R];
    int64_t row[R];
    const T* xp[R];
    u4 bx[R][P], blo[R][P], bias[R];
    float rr[R], eD[R];
    bool need_exact[R];
    auto make_block = [&](int r) {
      row[r] = row_of(rd, r, valid[r]);
      xp[r] = row_ptr(row[r]);
      if (PREFETCH)
        w_make_b<T, P>(raw, d, valid[r], ex, h, bx[r], blo[r], bias[r], rr[r], need_exact[r],
                       eD[r]);
      else
        w_make_b_direct<T, P>(xp[r], d, vec, valid[r], ex, h, bx[r], blo[r], bias[r], rr[r],
                              need_exact[r], eD[r]);
    };
    make_block(0);
    if constexpr (R == 2) make_block(1);
    // the next round's row is fetched while this one is scored
    if (PREFETCH && rd + 1 < nrounds) {
      bool v1;
      raw.load(row_ptr(row_of(rd + 1, 0, v1)), d, vec, h);
    }

    int best[R], bt[R], second[R];
    best[0] = 0x7fffffff, bt[0] = 0, second[0] = 0x7fffffff;
    if constexpr (R == 2) best[R - 1] = 0x7fffffff, bt[R - 1] = 0, second[R - 1] = 0x7fffffff;
    // scores of tiles t and t + 1 (when present) into the running best
    auto score = [&](const u4* ta, int t, bool pair) {
      if constexpr (SP && R == 2) {
        f16v c0, c1;
        w_tile_sp2<P>(ta, bx[0], bx[R - 1], bias[0], bias[R - 1], c0, c1);
        int b0, s0, b1, s1;
        w_tile_key2(c0, b0, s0);
        w_take2(b0, s0, t, best[0], bt[0], second[0]);
        w_tile_key2(c1, b1, s1);
        w_take2(b1, s1, t, best[R - 1], bt[R - 1], second[R - 1]);
      } else if constexpr (SP) {
        if (pair) {
          const f16v c0 = w_tile_sp<P>(ta, bx[0], bias[0]);
          const f16v c1 = w_tile_sp<P>(ta + QU * 64, bx[0], bias[0]);
          int b0, s0, b1, s1;
          w_tile_key2(c0, b0, s0);
          w_take2(b0, s0, t, best[0], bt[0], second[0]);
          w_tile_key2(c1, b1, s1);
          w_take2(b1, s1, t + 1, best[0], bt[0], second[0]);
        } else {
          const f16v c0 = w_tile_sp<P>(ta, bx[0], bias[0]);
          int b0, s0;
          w_tile_key2(c0, b0, s0);
          w_take2(b0, s0, t, best[0], bt[0], second[0]);
        }
      } else {
        const f16v c0 = w_tile<F16, P>(ta, bx[0], blo[0], bias[0]);
        if (pair) {
          const f16v c1 = w_tile<F16, P>(ta + QU * 64, bx[0], blo[0], bias[0]);
          w_take(w_tile_key(c0), t, best[0], bt[0]);
          w_take(w_tile_key(c1), t + 1, best[0], bt[0]);
        } else {
          w_take(w_tile_key(c0), t, best[0], bt[0]);
        }
      }
    };
    if (RESIDENT) {
      for (int t = 0; t < tiles; t += (PAIR_TILES ? 2 : 1))
        score(wtab + (size_t)t * QU * 64 + lane, tb + t, PAIR_TILES && t + 1 < tiles);
    } else {
      const int tpc = a.tpc;
      const int nch = (tiles + tpc - 1) / tpc;
      const int chunk_u4 = tpc * QU * 64;
      constexpr int SR = SP ? w_sp_sreg_n(C, NW) : (NW == W_WAVES ? w_sreg(C) : w_sreg_n(C, NTH));
      const WStage<QU, SR, NTH> stg;
      u4 reg[SR];
      {
        const int nt0 = min(tpc, tiles);
        stg.load(ftab, a.QF, 0, nt0, reg);
        w_stage_store<SR, NTH>(wtab, nt0 * QU * 64, reg);
      }
      __syncthreads();
      for (int c = 0; c < nch; ++c) {
        const int t0 = c * tpc;
        const int nt = min(tpc, tiles - t0);
        const int nt_next = (c + 1 < nch) ? min(tpc, tiles - t0 - tpc) : 0;
        const int n_next = nt_next * QU * 64;
        if (n_next) stg.load(ftab, a.QF, t0 + tpc, nt_next, reg);
        const u4* buf = wtab + (size_t)(c & 1) * chunk_u4;
        for (int tt = 0; tt < nt; tt += (PAIR_TILES ? 2 : 1))
          score(buf + (size_t)tt * QU * 64 + lane, tb + t0 + tt, PAIR_TILES && tt + 1 < nt);
        if (n_next) w_stage_store<SR, NTH>(wtab + (size_t)((c + 1) & 1) * chunk_u4, n_next, reg);
        __syncthreads();
      }
    }

    // per row block: combine the two lane halves of each row, then the
    // mode's outputs
    auto finish_block = [&](int r) {
      // combine the two lane halves of each row: smallest distance, then the
      // lowest codeword index
      int kstar;
      float dhat;
      bool ambiguous = false;
      {
        const int j = best[r] & 15;
        const int kidx = bt[r] * CW + (j >> 2) * 8 + h * 4 + (j & 3);
        const int hv = best[r] >> 4;
        const auto sh = __builtin_amdgcn_permlane32_swap(hv, hv, false, false);
        const auto sk = __builtin_amdgcn_permlane32_swap(kidx, kidx, false, false);
        const long long v0 = (long long)(int)sh[0] * 4294967296ll + (long long)(unsigned)sk[0];
        const long long v1 = (long long)(int)sh[1] * 4294967296ll + (long long)(unsigned)sk[1];
        const long long v = v0 < v1 ? v0 : v1;
        dhat = __int_as_float((int)(v >> 32) << 4);
        kstar = (int)(v & 0xffffffffll);
        if (SP) {
          // second smallest over both halves: med3(b0, b1, min(s0, s1)); a
          // row is decided when it lies beyond twice the error bound (the
          // single-pass bound, float32 accumulation and key truncation)
          // The bound of a codeword scales with its gain (eD is the bound at
          // g = sigma): the best's own gain on its side, the codebook's
          // largest gain for every other codeword.
          const auto sb = __builtin_amdgcn_permlane32_swap(best[r], best[r], false, false);
          const auto ss2 = __builtin_amdgcn_permlane32_swap(second[r], second[r], false, false);
          const int srow = med3i(sb[0], sb[1], min(ss2[0], ss2[1]));
          const float sv = __int_as_float(srow & ~15);
          const float gb = a.unit_gain ? 1.f : gcb[kstar < K ? kstar : K - 1];
          const float gx = a.unit_gain ? 1.f : a.gmin[a.G + (cb - a.fcb0)];
          const float md = ldexpf(eD[r] * (gb + gx), -ex) * 1.0625f +
                           ldexpf(dhat + ldexpf(rr[r], SA + 1), -15) + 0x1p-3f;
          ambiguous = !(sv - dhat > md);
        }
      }
      if (IND) {
        // this slice's best into the row's running minimum; the finish kernel
        // decides the row (64-bit keys: the distance key with its sign bit
        // flipped, so signed order is unsigned order, then the codeword)
        if (valid[r] && h == 0) {
          const size_t idx = (size_t)g * a.N + (size_t)((rc + rd * a.nwg) * WR + wave * RB + i);
          const uint32_t hv = (uint32_t)(__float_as_int(dhat) >> 4) ^ 0x80000000u;
          atomicMin(a.hbest + idx, ((unsigned long long)hv << 32) | (uint32_t)kstar);
          if (slice == 0) a.hrr[idx] = need_exact[r] ? -1.f : rr[r];
        }
        return;
      }
      need_exact[r] = need_exact[r] || !(dhat <= ldexpf(rr[r], SA + 1)) || kstar >= K;
      // rows the key cannot decide go to the subspace's list for the exact
      // kernel, which also writes their outputs; here they are skipped
      const bool defer = valid[r] && need_exact[r];
      {
        const unsigned long long fb = __ballot(defer && h == 0);
        if (fb) {
          const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(fb >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)fb, 0u));
          int base = 0;
          if (lane == 0) base = atomicAdd(a.xcount + g, __popcll(fb));
          base = __shfl(base, 0);
          if (defer && h == 0) a.xrows[(size_t)g * a.N + base + rank] = (int)row[r];
        }
      }
      // single pass: rows within the error bound go to the hi/lo pass
      const bool relist = SP && valid[r] && !defer && ambiguous;
      if (SP) {
        const unsigned long long fb = __ballot(relist && h == 0);
        if (fb) {
          const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(fb >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)fb, 0u));
          int base = 0;
          if (lane == 0) base = atomicAdd(a.hcount + g, __popcll(fb));
          base = __shfl(base, 0);
          if (relist && h == 0) {
            a.hrows[(size_t)g * a.N + base + rank] = (int)row[r];
            a.hbest[(size_t)g * a.N + base + rank] = ~0ull;
          }
        }
      }
      if (kstar >= K) kstar = K - 1;   // deferred rows and rows past N only
      const bool own = valid[r] && !defer && !relist;

      const float gk = a.unit_gain ? 1.f : gcb[kstar];
      const float* sk = scb + (size_t)kstar * d;
      if (MODE == W_TRAIN) {
        if (own && h == 0) {
          uint16_t* ap = a.assign + (size_t)g * a.N + row[r];
          if (*ap != (uint16_t)kstar) any_changed = true;
          *ap = (uint16_t)kstar;
        }
        if (a.obj) {
          // weighted distortion of this assignment under the scoring codebook;
          // each lane half sums half of the elements
          const int jb = h * (d / 2);
          float dist = w_residual<T, (P <= 8)>(xp[r] + jb, sk + jb, gk, d / 2, rvec, nullptr);
          dist += __shfl_xor(dist, 32);
          if (own && h == 0) obj += (double)(a.w ? a.w[row[r]] : 1.f) * (double)dist;
        }
      } else {
        if (own && h == 0 && a.codes)
          w_put_code(a.codes + row[r] * a.words, ((int64_t)a.m * a.G + g) * a.b, a.b, kstar);
        if (own && a.res_out) {
          // each lane half writes its half of the row's residual
          const int jb = h * (d / 2);
          float* dst = a.res_out + row[r] * ((int64_t)a.G * d) + (int64_t)g * d + jb;
          w_residual<T, (P <= 8)>(xp[r] + jb, sk + jb, gk, d / 2, rvec, dst);
        }
      }
    };
    finish_block(0);
    if constexpr (R == 2) finish_block(1);
  }
  if (MODE == W_TRAIN && !IND) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) obj += __shfl_xor(obj, off);
    if (lane == 0) red_obj[wave] = obj;
    if (__ballot(any_changed) && lane == 0) atomicOr(&red_changed, 1);
    __syncthreads();
    if (tid == 0) {
      double s = 0.0;
      for (int w = 0; w < NW; ++w) s += red_obj[w];
      a.changed[(size_t)g * a.nwg + rc] = red_changed;
      if (a.obj) a.obj[(size_t)g * a.nwg + rc] = s;
    }
  }
}

// Stage-fused encode for narrow wide rows (d <= 16) with resident fragment
// tables: a workgroup keeps the float32 residuals of its W_FUSED_ROUNDS x
// W_ROWS rows in registers (lane half h holds elements [8h, 8h + 8) of its
// row) through all M stages.  Per stage the stage's table is copied into
// LDS and every round is scored (float32 operand path, packed-key argmin);
// rows the key cannot decide are re-scored in float64 by the whole wave
// (eq. 5 form, every codeword; rare at these shapes); the code is written
// and the winning codeword fetched, and after the stage's last round the
// codewords are subtracted (the fetches overlap the later rounds' scoring).
// The residual leaves the registers only at the end, when it is requested.
struct WFusedArgs {
  const void* x;          // [N][ldx] input rows
  int64_t ldx, N;
  int d, K, G, M, tiles, QF, b, words;
  const u4* frag;         // [M G][tiles][QF][64]
  const int* sig;         // [M G]
  const float* gain;      // [M][G][K]
  const float* shape;     // [M][G][K][d]
  uint32_t* codes;        // [N][words], zeroed beforehand, or null
  float* res_out;         // [N][G d] or null
  int res_vec;            // res_out 16-byte aligned
  int svec;               // shape 16-byte aligned
  int nwg, map_xcd, lg;
};

template <typename T, int C>
__global__ void __launch_bounds__(W_THREADS, 2) w_encode_fused_kernel(WFusedArgs a) {
  extern __shared__ __align__(16) u4 wtab[];
  static_assert(C <= 2, "one 16-element group pair per row");
  constexpr int R = W_FUSED_ROUNDS;
  constexpr int QU = w_frags(C);
  int g, rc;
  {
    const int id = blockIdx.x;
    if (a.map_xcd) {
      const int xcd = id & 7, slot = id >> 3, gpx = a.G >> 3;
      const int j = slot % gpx;
      rc = slot / gpx;
      g = ((j / a.lg) * 8 + xcd) * a.lg + (j % a.lg);
    } else {
      g = id % a.G;
      rc = id / a.G;
    }
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = lane & 31, h = lane >> 5;
  const int d = a.d, K = a.K, G = a.G;
  const T* X = (const T*)a.x;
  float r[R][8];
  int64_t rows[R];
  const bool xvec = ((a.ldx * (int64_t)sizeof(T)) % 16 == 0) && (((uintptr_t)X) % 16 == 0);
#pragma unroll
  for (int rd = 0; rd < R; ++rd) {
    rows[rd] = ((int64_t)rc * R + rd) * W_ROWS + (int64_t)wave * RB + i;
    const bool valid = rows[rd] < a.N;
    const T* xp = X + (valid ? rows[rd] : 0) * a.ldx + (int64_t)g * d;
    WRaw<T, 1> raw;
    raw.load(xp, d, xvec, h);
#pragma unroll
    for (int j = 0; j < 8; ++j) r[rd][j] = raw.at(0, j, d, h, valid);
  }
  for (int m = 0; m < a.M; ++m) {
    const int cb = m * G + g;
    const int ex = a.sig[cb];
    const float* gcb = a.gain + (size_t)cb * K;
    const float* scb = a.shape + (size_t)cb * K * d;
    {
      const u4* ftab = a.frag + (size_t)cb * a.tiles * a.QF * 64;
      const int n = a.tiles * QU * 64;
      __syncthreads();                      // the previous stage's table is no longer read
      for (int e = tid; e < n; e += W_THREADS) {
        const int t = e / (QU * 64), o = e - t * (QU * 64);
        wtab[e] = ftab[(size_t)t * a.QF * 64 + o];
      }
      __syncthreads();
    }
    float gsel[R];
    f4 ssel[R][2];
#pragma unroll
    for (int rd = 0; rd < R; ++rd) {
      const int64_t row = rows[rd];
      const bool valid = row < a.N;
      WRaw<float, 1> raw;
      raw.v[0] = (u4){__float_as_uint(r[rd][0]), __float_as_uint(r[rd][1]),
                      __float_as_uint(r[rd][2]), __float_as_uint(r[rd][3])};
      raw.v[1] = (u4){__float_as_uint(r[rd][4]), __float_as_uint(r[rd][5]),
                      __float_as_uint(r[rd][6]), __float_as_uint(r[rd][7])};
      u4 bx[1], blo[1], bias;
      float rr;
      bool need_exact;
      float eD;
      w_make_b<float, 1>(raw, d, valid, ex, h, bx, blo, bias, rr, need_exact, eD);
      int best = 0x7fffffff, bt = 0;
      for (int t = 0; t < a.tiles; t += 2) {
        const u4* ta = wtab + (size_t)t * QU * 64 + lane;
        const f16v c0 = w_tile<false, 1>(ta, bx, blo, bias);
        if (t + 1 < a.tiles) {
          const f16v c1 = w_tile<false, 1>(ta + QU * 64, bx, blo, bias);
          w_take(w_tile_key(c0), t, best, bt);
          w_take(w_tile_key(c1), t + 1, best, bt);
        } else {
          w_take(w_tile_key(c0), t, best, bt);
        }
      }
      int kstar;
      float dhat;
      {
        const int j = best & 15;
        const int kidx = bt * CW + (j >> 2) * 8 + h * 4 + (j & 3);
        const int hv = best >> 4;
        const auto sh = __builtin_amdgcn_permlane32_swap(hv, hv, false, false);
        const auto sk = __builtin_amdgcn_permlane32_swap(kidx, kidx, false, false);
        const long long v0 = (long long)(int)sh[0] * 4294967296ll + (long long)(unsigned)sk[0];
        const long long v1 = (long long)(int)sh[1] * 4294967296ll + (long long)(unsigned)sk[1];
        const long long v = v0 < v1 ? v0 : v1;
        dhat = __int_as_float((int)(v >> 32) << 4);
        kstar = (int)(v & 0xffffffffll);
      }
      need_exact = need_exact || !(dhat <= ldexpf(rr, SA + 1)) || kstar >= K;
      unsigned long long fb = __ballot(valid && need_exact && h == 0);
      while (fb) {
        // the whole wave re-scores row L in float64: g^2 - 2 g s.x over all K
        const int L = __ffsll((long long)fb) - 1;
        fb &= fb - 1;
        double xr[16];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          xr[j] = (double)__shfl(r[rd][j], L);
          xr[8 + j] = (double)__shfl(r[rd][j], L + 32);
        }
        double bd = INFINITY;
        int bk = 0x7fffffff;
        for (int k = lane; k < K; k += 64) {
          const double gk = (double)gcb[k];
          double dot = 0.0;
          for (int j = 0; j < d; ++j) dot = fma(xr[j], (double)scb[(size_t)k * d + j], dot);
          const double dist = fma(-2.0 * gk, dot, gk * gk);
          if (dist < bd) { bd = dist; bk = k; }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const double od = __shfl_xor(bd, off);
          const int ok = __shfl_xor(bk, off);
          if (od < bd || (od == bd && ok < bk)) { bd = od; bk = ok; }
        }
        if (i == L) kstar = bk;
      }
      if (kstar >= K) kstar = K - 1;        // rows past N only
      if (valid && h == 0 && a.codes)
        w_put_code(a.codes + row * a.words, ((int64_t)m * G + g) * a.b, a.b, kstar);
      // the codeword is fetched now and subtracted after the stage's last
      // round, so the loads overlap the next rounds' scoring
      const int e0 = 8 * h < d ? 8 * h : 0;   // d = 8: lane half 1 holds no elements
      gsel[rd] = gcb[kstar] * ((8 * h < d) ? 1.f : 0.f);
      const float* sp = scb + (size_t)kstar * d + e0;
      if (a.svec) {
        ssel[rd][0] = ((const f4*)sp)[0];
        ssel[rd][1] = ((const f4*)sp)[1];
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          ssel[rd][0][j] = sp[j];
          ssel[rd][1][j] = sp[4 + j];
        }
      }
    }
#pragma unroll
    for (int rd = 0; rd < R; ++rd)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        r[rd][j] = fmaf(-gsel[rd], ssel[rd][0][j], r[rd][j]);
        r[rd][4 + j] = fmaf(-gsel[rd], ssel[rd][1][j], r[rd][4 + j]);
      }
  }
  if (a.res_out) {
#pragma unroll
    for (int rd = 0; rd < R; ++rd) {
      const int64_t row = rows[rd];
      if (row >= a.N || 8 * h >= d) continue;
      float* dst = a.res_out + row * ((int64_t)G * d) + (int64_t)g * d + 8 * h;
      if (a.res_vec) {
        ((f4*)dst)[0] = (f4){r[rd][0], r[rd][1], r[rd][2], r[rd][3]};
        ((f4*)dst)[1] = (f4){r[rd][4], r[rd][5], r[rd][6], r[rd][7]};
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) dst[j] = r[rd][j];
      }
    }
  }
}

// Stage-fused encode for d = 64 and 128 with the hi/lo pass (K <= 512): a
// wave keeps the float32 residual of its 32-row block in registers through
// all M stages (lane half h holds groups 2p + h of its row: elements
// [16p + 8h, 16p + 8h + 8)), so no residual crosses HBM between stages.
// Per stage the stage's whole fragment table is copied into LDS, every
// tile scored (float32 operand path, two tiles' MFMA chains in flight), the
// row's code written, and the winning codeword subtracted in place; rows
// the key cannot decide are re-scored in float64 by the whole wave (eq. 5
// form over every codeword; rare).  The residual leaves the registers only
// at the end, when it is requested.
constexpr int W_FW_LDS_MAX = 144 * 1024;   // a stage's fragment table, at most
constexpr int W_FW_KMAX = 512;             // codewords of the float64 re-score, at most
// eight waves share a stage's table: two per SIMD, so one wave's argmin and
// table reads overlap another's MFMA chains even when the table leaves room
// for a single workgroup per CU, and each table copy serves 256 rows
constexpr int W_FW_WAVES = 8;
constexpr int W_FW_THREADS = W_FW_WAVES * 64;
constexpr int W_FW_ROWS = W_FW_WAVES * RB;
template <typename T, int C>
__global__ void __launch_bounds__(W_FW_THREADS, 1) w_encode_fused_wide_kernel(WFusedArgs a) {
  extern __shared__ __align__(16) u4 wtab[];
  static_assert(C == 8 || C == 16, "d = 64 or 128");
  constexpr int P = w_pairs(C);
  constexpr int QU = w_frags(C);
  int g, rc;
  {
    const int id = blockIdx.x;
    if (a.map_xcd) {
      const int xcd = id & 7, slot = id >> 3, gpx = a.G >> 3;
      const int j = slot % gpx;
      rc = slot / gpx;
      g = ((j / a.lg) * 8 + xcd) * a.lg + (j % a.lg);
    } else {
      g = id % a.G;
      rc = id / a.G;
    }
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = lane & 31, h = lane >> 5;
  const int d = a.d, K = a.K, G = a.G;
  const int64_t row = (int64_t)rc * W_FW_ROWS + (int64_t)wave * RB + i;
  const bool valid = row < a.N;
  float r[P][8];
  {
    const T* xp = (const T*)a.x + (valid ? row : 0) * a.ldx + (int64_t)g * d + 8 * h;
    const bool xvec = ((a.ldx * (int64_t)sizeof(T)) % 16 == 0) && (((uintptr_t)a.x) % 16 == 0);
#pragma unroll
    for (int p = 0; p < P; ++p) {
      float v[8];
      if (xvec) {
        if (sizeof(T) == 2) {
          const h8 x8 = as_h8(*(const u4*)(xp + 16 * p));
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = (float)x8[j];
        } else {
          const f4 lo = *(const f4*)(xp + 16 * p), hi = *(const f4*)(xp + 16 * p + 4);
#pragma unroll
          for (int j = 0; j < 4; ++j) { v[j] = lo[j]; v[4 + j] = hi[j]; }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (float)xp[16 * p + j];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) r[p][j] = valid ? v[j] : 0.f;
    }
  }
  for (int m = 0; m < a.M; ++m) {
    const int cb = m * G + g;
    const int ex = a.sig[cb];
    const float* gcb = a.gain + (size_t)cb * K;
    const float* scb = a.shape + (size_t)cb * K * d;
    {
      const u4* ftab = a.frag + (size_t)cb * a.tiles * a.QF * 64;
      const int n = a.tiles * QU * 64;
      constexpr int UN = 4;                 // loads in flight per thread
      __syncthreads();                      // the previous stage's table is no longer read
      for (int e0 = tid; e0 < n; e0 += UN * W_FW_THREADS) {
        u4 v[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
          const int e = e0 + u * W_FW_THREADS;
          const int t = e / (QU * 64), o = e - t * (QU * 64);
          if (e < n) v[u] = ftab[(size_t)t * a.QF * 64 + o];
        }
#pragma unroll
        for (int u = 0; u < UN; ++u)
          if (e0 + u * W_FW_THREADS < n) wtab[e0 + u * W_FW_THREADS] = v[u];
      }
      __syncthreads();
    }
    u4 bx[P], blo[P], bias;
    float rr, eD;
    bool need_exact;
    {
      WRaw<float, P> raw;
#pragma unroll
      for (int p = 0; p < P; ++p) {
        raw.v[2 * p] = (u4){__float_as_uint(r[p][0]), __float_as_uint(r[p][1]),
                            __float_as_uint(r[p][2]), __float_as_uint(r[p][3])};
        raw.v[2 * p + 1] = (u4){__float_as_uint(r[p][4]), __float_as_uint(r[p][5]),
                                __float_as_uint(r[p][6]), __float_as_uint(r[p][7])};
      }
      w_make_b<float, P>(raw, d, valid, ex, h, bx, blo, bias, rr, need_exact, eD);
    }
    int best = 0x7fffffff, bt = 0;
    for (int t = 0; t < a.tiles; t += 2) {
      const u4* ta = wtab + (size_t)t * QU * 64 + lane;
      const f16v c0 = w_tile<false, P>(ta, bx, blo, bias);
      if (t + 1 < a.tiles) {
        const f16v c1 = w_tile<false, P>(ta + QU * 64, bx, blo, bias);
        w_take(w_tile_key(c0), t, best, bt);
        w_take(w_tile_key(c1), t + 1, best, bt);
      } else {
        w_take(w_tile_key(c0), t, best, bt);
      }
    }
    int kstar;
    float dhat;
    {
      const int j = best & 15;
      const int kidx = bt * CW + (j >> 2) * 8 + h * 4 + (j & 3);
      const int hv = best >> 4;
      const auto sh = __builtin_amdgcn_permlane32_swap(hv, hv, false, false);
      const auto sk = __builtin_amdgcn_permlane32_swap(kidx, kidx, false, false);
      const long long v0 = (long long)(int)sh[0] * 4294967296ll + (long long)(unsigned)sk[0];
      const long long v1 = (long long)(int)sh[1] * 4294967296ll + (long long)(unsigned)sk[1];
      const long long v = v0 < v1 ? v0 : v1;
      dhat = __int_as_float((int)(v >> 32) << 4);
      kstar = (int)(v & 0xffffffffll);
    }
    need_exact = need_exact || !(dhat <= ldexpf(rr, SA + 1)) || kstar >= K;
    unsigned long long fb = __ballot(valid && need_exact && h == 0);
    while (fb) {
      // the whole wave re-scores row L in float64: g^2 - 2 g s.x over all
      // K codewords (lane l takes codewords l, l + 64, ...), the row's
      // elements broadcast one at a time from lanes L and L + 32
      const int L = __ffsll((long long)fb) - 1;
      fb &= fb - 1;
      constexpr int KQ = W_FW_KMAX / 64;
      double dot[KQ];
#pragma unroll
      for (int q = 0; q < KQ; ++q) dot[q] = 0.0;
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const double xj = (double)__shfl(r[p][j & 7], L + 32 * (j >> 3));
          const int e = 16 * p + j;
#pragma unroll
          for (int q = 0; q < KQ; ++q) {
            const int k = lane + 64 * q;
            if (k < K) dot[q] = fma(xj, (double)scb[(size_t)k * d + e], dot[q]);
          }
        }
      double bd = INFINITY;
      int bk = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < KQ; ++q) {
        const int k = lane + 64 * q;
        if (k < K) {
          const double gk = (double)gcb[k];
          const double dist = fma(-2.0 * gk, dot[q], gk * gk);
          if (dist < bd) { bd = dist; bk = k; }
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const double od = __shfl_xor(bd, off);
        const int ok = __shfl_xor(bk, off);
        if (od < bd || (od == bd && ok < bk)) { bd = od; bk = ok; }
      }
      if (i == L) kstar = bk;
    }
    if (kstar >= K) kstar = K - 1;        // rows past N only
    if (valid && h == 0 && a.codes)
      w_put_code(a.codes + row * a.words, ((int64_t)m * G + g) * a.b, a.b, kstar);
    // subtract the codeword: this lane half's groups of g s
    const float gk = gcb[kstar];
    const float* sp = scb + (size_t)kstar * d + 8 * h;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      float sv[8];
      if (a.svec) {
        const f4 lo = *(const f4*)(sp + 16 * p), hi = *(const f4*)(sp + 16 * p + 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) { sv[j] = lo[j]; sv[4 + j] = hi[j]; }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) sv[j] = sp[16 * p + j];
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) r[p][j] = fmaf(-gk, sv[j], r[p][j]);
    }
  }
  if (a.res_out && valid) {
    float* dst = a.res_out + row * ((int64_t)G * d) + (int64_t)g * d + 8 * h;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      if (a.res_vec) {
        ((f4*)(dst + 16 * p))[0] = (f4){r[p][0], r[p][1], r[p][2], r[p][3]};
        ((f4*)(dst + 16 * p))[1] = (f4){r[p][4], r[p][5], r[p][6], r[p][7]};
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) dst[16 * p + j] = r[p][j];
      }
    }
  }
}

// Outputs of the rows the single pass listed, after the sliced hi/lo pass:
// each row's best (distance key, codeword) from hbest is checked like a row
// of the scoring kernel (operands in the float16 range, best distance at
// most twice the row's energy) and either appended to the exact kernel's
// list or written out: training the assignment, the stop flag (xchanged)
// and the weighted distortion (xobj); encode the code bits and the
// residual.  One wave per listed row, grid-stride over the list.
template <typename T, int MODE>
__global__ void __launch_bounds__(256) w_listed_finish_kernel(WScoreArgs a) {
  const int g = blockIdx.y;
  if (a.done && a.done[g]) return;
  const int cnt = a.hcount[g];
  const int lane = threadIdx.x & 63, wpb = blockDim.x >> 6;
  const int d = a.d, K = a.K;
  const int cb = a.cb0 + g;
  const float* gcb = a.gain + (size_t)cb * K;
  const float* scb = a.shape + (size_t)cb * K * d;
  const T* X = (const T*)a.x;
  for (int idx = blockIdx.x * wpb + (int)(threadIdx.x >> 6); idx < cnt; idx += gridDim.x * wpb) {
    const size_t li = (size_t)g * a.N + idx;
    const int64_t row = a.hrows[li];
    const unsigned long long key = a.hbest[li];
    const float rr = a.hrr[li];
    const int kstar = (int)(uint32_t)key;
    const float dhat = __int_as_float((int)((uint32_t)(key >> 32) ^ 0x80000000u) << 4);
    if (!(rr >= 0.f) || !(dhat <= ldexpf(rr, SA + 1)) || kstar >= K) {
      if (lane == 0) {
        const int pos = atomicAdd(a.xcount + g, 1);
        a.xrows[(size_t)g * a.N + pos] = (int)row;
      }
      continue;
    }
    const float gk = a.unit_gain ? 1.f : gcb[kstar];
    const float* sk = scb + (size_t)kstar * d;
    const T* xp = X + row * a.ldx + (int64_t)g * d;
    if (MODE == W_TRAIN) {
      if (a.obj) {
        float dist = 0.f;
        for (int j = lane; j < d; j += 64) {
          const float r = fmaf(-gk, sk[j], (float)xp[j]);
          dist = fmaf(r, r, dist);
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) dist += __shfl_xor(dist, off);
        if (lane == 0) atomicAdd(a.xobj + g, (double)(a.w ? a.w[row] : 1.f) * (double)dist);
      }
      if (lane == 0) {
        uint16_t* ap = a.assign + (size_t)g * a.N + row;
        if (*ap != (uint16_t)kstar) a.xchanged[g] = 1;
        *ap = (uint16_t)kstar;
      }
    } else {
      if (lane == 0 && a.codes)
        w_put_code(a.codes + row * a.words, ((int64_t)a.m * a.G + g) * a.b, a.b, kstar);
      if (a.res_out) {
        float* dst = a.res_out + row * ((int64_t)a.G * d) + (int64_t)g * d;
        for (int j = lane; j < d; j += 64) dst[j] = fmaf(-gk, sk[j], (float)xp[j]);
      }
    }
  }
}

// Deferred exact rows: the eq. (5) argmin in float64 (ties to the lowest
// index) for the rows the scoring kernel listed, and their outputs.  Grid:
// (workgroups, G); a workgroup takes batches of 16 listed rows of its
// subspace.  Candidates are pruned by gain per batch, which is exact: with
// E_k = ||x||^2 + g_k^2 - 2 g_k s_k.x and |s_k.x| <= ||x|| (shapes of norm at
// most 1), (g_k - ||x||)^2 <= E_k <= (g_k + ||x||)^2, so a codeword with
// g_k > gmin + 2 max ||x|| (1e-5 relative slack) wins for no row of the
// batch.  The survivors' s_k.x are accumulated in float64, one codeword per
// lane at a time spread over all four waves (a batch of a few rows, the
// usual case, then costs one pass over each codeword's elements instead of
// a 4 x 4 block walk by one wave); each lane keeps the dot products of the
// batch's rows (in groups of four, only the groups the batch fills) in
// element order 0 .. d - 1, streaming its codeword in double-buffered
// 32-element blocks against rows held in LDS as float64.  The per-row
// minimum (lowest index on ties) is taken over lanes, then over waves.
constexpr int W_XROWS = 16;
constexpr int W_XTHREADS = 256;
constexpr int W_XKMAX = 4096;    // candidate list capacity (codewords)

template <typename T, int MODE>
__global__ void __launch_bounds__(W_XTHREADS) w_exact_kernel(WScoreArgs a) {
  __shared__ __align__(16) double xsd[W_XROWS][8 * W_CMAX];
  __shared__ double xn[W_XROWS], xq[W_XROWS];
  __shared__ double wbd[W_XTHREADS / 64][W_XROWS];
  __shared__ int wbk[W_XTHREADS / 64][W_XROWS];
  __shared__ double bestd[W_XROWS];
  __shared__ int bestk[W_XROWS];
  __shared__ int rows[W_XROWS];
  __shared__ int olda[W_XROWS];
  __shared__ int cand[W_XKMAX];
  __shared__ int ncand;
  const int g = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, K = a.K;
  const int cb = a.cb0 + g;
  const float* gcb = a.gain + (size_t)cb * K;
  const float* scb = a.shape + (size_t)cb * K * d;
  const T* X = (const T*)a.x;
  // A launch is mostly latency.  The workgroup of a subspace's first batch
  // (the others are usually empty) fetches what does not depend on the list
  // together with its count: that batch's row ids, read before the count is
  // known (entries past it are in bounds and unused), and with
  // K <= W_XTHREADS the gain of codeword tid for the candidate test.
  const bool small = K <= W_XTHREADS;
  const bool ahead = blockIdx.x == 0;
  float gpre = 1.f;
  if (small && ahead && !a.unit_gain) gpre = gcb[min(tid, K - 1)];
  int rid = 0;
  if (ahead && tid < W_XROWS) rid = a.xrows[(size_t)g * a.N + min((int64_t)tid, a.N - 1)];
  const int cnt = a.xcount[g];
  if (a.done && a.done[g]) return;
  const double gmin = (double)a.gmin[cb - a.fcb0];
  bool first = true;
  for (int b0 = blockIdx.x * W_XROWS; b0 < cnt; b0 += gridDim.x * W_XROWS) {
    const int nb = min(W_XROWS, cnt - b0);
    if (!(first && ahead) && tid < W_XROWS)
      rid = a.xrows[(size_t)g * a.N + b0 + min(tid, nb - 1)];
    // slots past nb repeat the last row (wave 0 holds all W_XROWS ids)
    {
      const int r = __shfl(rid, min(lane, nb - 1));
      if (tid < W_XROWS) rows[tid] = r;
    }
    if (tid == 0) ncand = 0;
    __syncthreads();
    {
      // the rows' d elements (slots past nb repeat the last row), eight
      // unconditional loads in flight per thread, and the rows' previous
      // assignments: the batch is latency-bound
      int oa = 0;
      if (MODE == W_TRAIN && tid < W_XROWS) oa = a.assign[(size_t)g * a.N + rows[tid]];
      const int ld = 31 - __clz(d), n = W_XROWS << ld;
      constexpr int UN = 8;
      for (int e0 = tid; e0 < n; e0 += UN * W_XTHREADS) {
        float v[UN];
#pragma unroll
        for (int u = 0; u < UN; ++u) {
          const int e = min(e0 + u * W_XTHREADS, n - 1);
          v[u] = to_f(X[(int64_t)rows[e >> ld] * a.ldx + (int64_t)g * d + (e & (d - 1))]);
        }
#pragma unroll
        for (int u = 0; u < UN; ++u) {
          const int e = e0 + u * W_XTHREADS;
          if (e < n) xsd[e >> ld][e & (d - 1)] = (double)v[u];
        }
      }
      if (MODE == W_TRAIN && tid < W_XROWS) olda[tid] = oa;
    }
    __syncthreads();
    // row norms: wave w sums rows 4w .. 4w + 3 across its lanes
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const double* xr = xsd[wave * 4 + r];
      double q = 0.0;
      for (int j = lane; j < d; j += 64) q = fma(xr[j], xr[j], q);
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) q += __shfl_xor(q, off);
      if (lane == 0) {
        xq[wave * 4 + r] = q;
        xn[wave * 4 + r] = sqrt(q);
      }
    }
    __syncthreads();
    double xmax = 0.0;
    for (int i = 0; i < W_XROWS; ++i) xmax = fmax(xmax, xn[i]);
    const double thr = (gmin + 2.0 * xmax) * (1.0 + 1e-5);
    // candidate list (any order; ties are broken by index below): codewords
    // with g > g_min + 2 max ||x|| cannot win
    for (int k0 = 0; k0 < K; k0 += W_XTHREADS) {
      const int k = k0 + tid;
      const double gk = a.unit_gain ? 1.0
                                    : (double)(small && ahead && first ? gpre
                                                                       : gcb[min(k, K - 1)]);
      const bool c = k < K && gk <= thr;
      const unsigned long long m = __ballot(c);
      const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      int base = 0;
      if (lane == 0 && m) base = atomicAdd(&ncand, __popcll(m));
      base = __shfl(base, 0);
      if (c && base + rank < W_XKMAX) cand[base + rank] = k;
    }
    __syncthreads();
    // a list that overflowed falls back to every codeword
    const int nc = ncand <= W_XKMAX ? ncand : K;
    const bool all = ncand > W_XKMAX;
    const int nr4 = (nb + 3) >> 2;          // row groups of four the batch fills
    constexpr int JB = 32;                  // codeword elements per block
    double bd[4][4];
    int bk[4][4];
#pragma unroll
    for (int rg = 0; rg < 4; ++rg)
#pragma unroll
      for (int r = 0; r < 4; ++r) { bd[rg][r] = INFINITY; bk[rg][r] = 0x7fffffff; }
    for (int c0 = wave * 64 + lane; c0 - lane < nc; c0 += W_XTHREADS) {
      const bool live = c0 < nc;
      const int kq = all ? min(c0, K - 1) : cand[min(c0, nc - 1)];
      const double gq = a.unit_gain ? 1.0 : (double)gcb[kq];
      const float* sp = scb + (size_t)kq * d;
      double acc[4][4];
#pragma unroll
      for (int rg = 0; rg < 4; ++rg)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[rg][r] = 0.0;
      auto block = [&](const f4 (&buf)[JB / 4], int jb) {
        const int je = min(JB, d - jb);
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          if (rg >= nr4) break;
#pragma unroll
          for (int v = 0; v < JB / 4; ++v) {
            if (4 * v >= je) break;
            const double c0d = (double)buf[v][0], c1d = (double)buf[v][1];
            const double c2d = (double)buf[v][2], c3d = (double)buf[v][3];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const double* xr = &xsd[rg * 4 + r][jb + 4 * v];
              const double2 xa = *(const double2*)xr, xb = *(const double2*)(xr + 2);
              double t = acc[rg][r];
              t = fma(xa.x, c0d, t);
              t = fma(xa.y, c1d, t);
              t = fma(xb.x, c2d, t);
              t = fma(xb.y, c3d, t);
              acc[rg][r] = t;
            }
          }
        }
      };
      f4 ca[JB / 4], cz[JB / 4];             // the two block buffers
      const int nbk = (d + JB - 1) / JB;
      auto load = [&](f4 (&buf)[JB / 4], int jb) {
#pragma unroll
        for (int v = 0; v < JB / 4; ++v) {
          const int j = min(jb + 4 * v, d - 4);          // in bounds; unused past d
          buf[v] = *(const f4*)(sp + j);
        }
      };
      load(ca, 0);
      for (int bi = 0; bi < nbk; bi += 2) {
        if (bi + 1 < nbk) load(cz, (bi + 1) * JB);
        block(ca, bi * JB);
        if (bi + 1 < nbk) {
          if (bi + 2 < nbk) load(ca, (bi + 2) * JB);
          block(cz, (bi + 1) * JB);
        }
      }
      if (live) {
#pragma unroll
        for (int rg = 0; rg < 4; ++rg)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            // eq. (5) up to the row constant ||x||^2: g^2 - 2 g s.x
            const double e = fma(-2.0 * gq, acc[rg][r], gq * gq);
            if (e < bd[rg][r] || (e == bd[rg][r] && kq < bk[rg][r])) {
              bd[rg][r] = e;
              bk[rg][r] = kq;
            }
          }
      }
    }
    first = false;
    // minimum per row over the wave's lanes, then over the four waves
#pragma unroll
    for (int rg = 0; rg < 4; ++rg) {
      if (rg >= nr4) break;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        double b = bd[rg][r];
        int k = bk[rg][r];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const double od = __shfl_xor(b, off);
          const int ok = __shfl_xor(k, off);
          if (od < b || (od == b && ok < k)) { b = od; k = ok; }
        }
        if (lane == 0) {
          wbd[wave][rg * 4 + r] = b;
          wbk[wave][rg * 4 + r] = k;
        }
      }
    }
    __syncthreads();
    if (tid < nb) {
      double b = wbd[0][tid];
      int k = wbk[0][tid];
      for (int w2 = 1; w2 < W_XTHREADS / 64; ++w2) {
        const double od = wbd[w2][tid];
        const int ok = wbk[w2][tid];
        if (od < b || (od == b && ok < k)) { b = od; k = ok; }
      }
      bestk[tid] = k < K ? k : 0;           // (a non-empty list always sets k)
      bestd[tid] = b;
    }
    __syncthreads();
    // outputs: wave w writes rows w, w + 4, w + 8, w + 12
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = wave + 4 * r;
      if (i >= nb) break;
      const int64_t row = rows[i];
      const int k = bestk[i];
      if (MODE == W_TRAIN) {
        if (lane == 0) {
          // weighted distortion ||x - g s||^2 = ||x||^2 + (g^2 - 2 g s.x)
          // of the chosen codeword, both terms in float64
          if (a.obj)
            atomicAdd(a.xobj + g, (double)(a.w ? a.w[row] : 1.f) * (xq[i] + bestd[i]));
          if (olda[i] != k) a.xchanged[g] = 1;
          a.assign[(size_t)g * a.N + row] = (uint16_t)k;
        }
      } else {
        if (lane == 0 && a.codes)
          w_put_code(a.codes + row * a.words, ((int64_t)a.m * a.G + g) * a.b, a.b, k);
        if (a.res_out) {
          const float gk = gcb[k];
          float* dst = a.res_out + row * ((int64_t)a.G * d) + (int64_t)g * d;
          for (int j = lane; j < d; j += 64)
            dst[j] = fmaf(-gk, scb[(size_t)k * d + j], (float)xsd[i][j]);
        }
      }
    }
    __syncthreads();
  }
}

struct WAccArgs {
  const void* x;
  int64_t ldx, N;
  int d, K, G;
  const float* w;          // [N] or null
  const uint16_t* assign;  // [G][N]
  const int* done;         // [G] or null
  double* part;            // [G][rchunks][K][2d+2]
  int ks, slices, rchunks;
  int64_t rows_per_chunk;
  const int* sorted;       // [G][N] rows bucketed by codeword, or null
  const int* boff;         // [G][K + 1] bucket offsets into sorted
  double* ovf;             // [G][nwin][2d+2] window partials (sorted sums), or null
  const int* wk;           // [G][nwin] the codeword whose overflow meets window i, or -1
  int nwin;
};

// Rows of each subspace bucketed by codeword, a counting sort in three
// launches over row chunks of bch rows (one workgroup per chunk and
// subspace, so the whole GPU takes part; w_bucket_rows sizes the chunks):
//   count:   cnt[g][c][k] = members of codeword k in chunk c (LDS histogram);
//   scan:    boff[g][k] = first position of codeword k's members in
//            sorted[g] (boff[g][K] = N), and cnt[g][c][k] becomes the first
//            position of chunk c's members of k;
//   scatter: every row of chunk c goes to the next position of its codeword.
// Buckets hold their members chunk by chunk; within a chunk the order is
// that of LDS atomics (the sums built from it are then exact up to float64
// rounding order).
constexpr int W_BCH = 2048;
// Rows per bucketing chunk: W_BCH, doubled while the scan's chunks x K
// entries per subspace exceed 32768 (the scan is one workgroup per subspace).
inline int64_t w_bucket_rows(int64_t N, int K) {
  int64_t bch = W_BCH;
  while (bch < N && ((N + bch - 1) / bch) * (int64_t)K > 32768) bch *= 2;
  return bch;
}
__global__ void __launch_bounds__(256) w_bucket_count_kernel(const uint16_t* __restrict__ assign,
                                                             int64_t N, int K, int64_t bch,
                                                             const int* __restrict__ done,
                                                             int* __restrict__ cnt) {
  extern __shared__ int hist[];
  const int g = blockIdx.y, c = blockIdx.x;
  if (done && done[g]) return;
  const int tid = threadIdx.x;
  for (int k = tid; k < K; k += 256) hist[k] = 0;
  __syncthreads();
  const uint16_t* asg = assign + (size_t)g * N;
  const int64_t r1 = min(N, (int64_t)(c + 1) * bch);
  for (int64_t r = (int64_t)c * bch + tid; r < r1; r += 256) atomicAdd(&hist[asg[r]], 1);
  __syncthreads();
  int* out = cnt + ((size_t)g * gridDim.x + c) * K;
  for (int k = tid; k < K; k += 256) out[k] = hist[k];
}

__global__ void __launch_bounds__(1024) w_bucket_scan_kernel(int64_t N, int K, int chunks,
                                                             const int* __restrict__ done,
                                                             int* __restrict__ cnt,
                                                             int* __restrict__ boff,
                                                             int nwin, int* __restrict__ wk) {
  extern __shared__ int sc[];               // [chunks][K] counts, staged
  __shared__ int wsum[16];
  const int g = blockIdx.x;
  if (done && done[g]) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int* cg = cnt + (size_t)g * chunks * K;
  {
    // the counts into LDS, eight loads in flight per thread
    const int n = chunks * K;
    constexpr int UN = 8;
    for (int e0 = tid; e0 < n; e0 += UN * 1024) {
      int v[UN];
#pragma unroll
      for (int u = 0; u < UN; ++u) v[u] = cg[min(e0 + u * 1024, n - 1)];
#pragma unroll
      for (int u = 0; u < UN; ++u)
        if (e0 + u * 1024 < n) sc[e0 + u * 1024] = v[u];
    }
  }
  int* wkg = wk ? wk + (size_t)g * nwin : nullptr;
  if (wkg)
    for (int i = tid; i < nwin; i += 1024) wkg[i] = -1;
  __syncthreads();
  // thread tid owns bins [b, e): their totals over the chunks, then an
  // exclusive scan of the totals over the workgroup
  const int per = (K + 1023) / 1024;
  const int b = min(K, tid * per), e = min(K, b + per);
  int tot = 0;
  for (int k = b; k < e; ++k)
    for (int c = 0; c < chunks; ++c) tot += sc[c * K + k];
  int inc = tot;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(inc, off);
    if (lane >= off) inc += v;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int base = inc - tot;
  for (int w2 = 0; w2 < wave; ++w2) base += wsum[w2];
  int* bo = boff + (size_t)g * (K + 1);
  for (int k = b; k < e; ++k) {
    const int m0 = base;
    bo[k] = base;
    for (int c = 0; c < chunks; ++c) {
      const int n = sc[c * K + k];
      cg[(size_t)c * K + k] = base;
      base += n;
    }
    // the windows that codeword k's members past its first W_SORT_Q meet
    if (wkg && base - m0 > W_SORT_Q)
      for (int i = (m0 + W_SORT_Q) / W_SORT_Q; i <= (base - 1) / W_SORT_Q; ++i) wkg[i] = k;
  }
  if (tid == 0) bo[K] = (int)N;
}

__global__ void __launch_bounds__(256) w_bucket_scatter_kernel(const uint16_t* __restrict__ assign,
                                                               int64_t N, int K, int64_t bch,
                                                               const int* __restrict__ done,
                                                               const int* __restrict__ cnt,
                                                               int* __restrict__ sorted) {
  extern __shared__ int cur[];
  const int g = blockIdx.y, c = blockIdx.x;
  if (done && done[g]) return;
  const int tid = threadIdx.x;
  const int* in = cnt + ((size_t)g * gridDim.x + c) * K;
  for (int k = tid; k < K; k += 256) cur[k] = in[k];
  __syncthreads();
  const uint16_t* asg = assign + (size_t)g * N;
  int* srt = sorted + (size_t)g * N;
  const int64_t r1 = min(N, (int64_t)(c + 1) * bch);
  for (int64_t r = (int64_t)c * bch + tid; r < r1; r += 256)
    srt[atomicAdd(&cur[asg[r]], 1)] = (int)r;
}

// Batched member loop of the accumulation: members [0, n), member `it` is
// row row_of(it) of codeword asg[row] in [k0, k0 + ks).  Lane groups of d / E
// lanes take one member each (E elements per lane), W_ACC_MEMBERS members
// per lane group in flight: every load of a batch is issued before the
// first use (past the end a lane group re-reads its first member and adds
// nothing).
template <typename T, int E, typename RowOf>
__device__ __forceinline__ void w_acc_members(const WAccArgs& a, int g, int k0, double* wacc,
                                              int n, RowOf row_of) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, S = 2 * d + 2;
  const int L = d / E;                 // lanes per member row (power of two, <= 64)
  const int per_wave = 64 / L;
  const int sub = lane / L, li = lane % L;
  const uint16_t* asg = a.assign + (size_t)g * a.N;
  const T* X = (const T*)a.x;
  const int stride = W_WAVES * per_wave;
  for (int it0 = wave * per_wave + sub; it0 < n; it0 += W_ACC_MEMBERS * stride) {
    float xv[W_ACC_MEMBERS][E], wt[W_ACC_MEMBERS];
    int k[W_ACC_MEMBERS];
#pragma unroll
    for (int u = 0; u < W_ACC_MEMBERS; ++u) {
      const int it = it0 + u * stride < n ? it0 + u * stride : it0;
      const int64_t row = row_of(it);
      k[u] = asg[row];
      const T* xr = X + row * a.ldx + (int64_t)g * d;
#pragma unroll
      for (int e = 0; e < E; ++e) xv[u][e] = (float)xr[E * li + e];
      wt[u] = a.w ? a.w[row] : 1.f;
    }
#pragma unroll
    for (int u = 0; u < W_ACC_MEMBERS; ++u) {
      float ss = xv[u][E - 1] * xv[u][E - 1];
#pragma unroll
      for (int e = E - 2; e >= 0; --e) ss = fmaf(xv[u][e], xv[u][e], ss);
      for (int off = L / 2; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      if (it0 + u * stride >= n) continue;   // uniform within the lane group
      const float inv = __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(ss) + Y_EPS);
      double* ak = wacc + (size_t)(k[u] - k0) * S;
#pragma unroll
      for (int e = 0; e < E; ++e)
        unsafeAtomicAdd(ak + E * li + e, (double)(xv[u][e] * (wt[u] * inv)));
#pragma unroll
      for (int e = 0; e < E; ++e) unsafeAtomicAdd(ak + d + E * li + e, (double)(xv[u][e] * wt[u]));
      if (li == 0) {
        unsafeAtomicAdd(ak + 2 * d, (double)wt[u]);
        unsafeAtomicAdd(ak + 2 * d + 1, 1.0);
      }
    }
  }
}

// Weighted sums of eqs. 6-8 for one (codeword slice, row chunk, subspace):
// sum w y and sum w x (y = x / (||x|| + eps)), sum w and the member count
// per codeword, accumulated in float64 LDS and written as one partial.
// Members: with one slice, every row of the chunk; with bucketed rows, the
// chunk's share of the slice's buckets; otherwise the chunk's members of
// the slice, collected into an LDS list first.  E elements per lane: 2, or
// 4 for d = 256 (a lane group is at most one wave).
template <typename T, int E>
__global__ void __launch_bounds__(W_THREADS) w_accumulate_kernel(WAccArgs a) {
  extern __shared__ double wacc[];
  __shared__ int list[W_THREADS * W_ACC_BATCH];
  __shared__ int nlist;
  const int g = blockIdx.y;
  if (a.done && a.done[g]) return;
  const int slice = blockIdx.x % a.slices, rc = blockIdx.x / a.slices;
  const int tid = threadIdx.x, lane = tid & 63;
  const int d = a.d, S = 2 * d + 2;
  const int k0 = slice * a.ks, k1 = min(a.K, k0 + a.ks);
  for (int e = tid; e < a.ks * S; e += W_THREADS) wacc[e] = 0.0;
  __syncthreads();
  if (a.sorted) {
    const int* bo = a.boff + (size_t)g * (a.K + 1);
    const int m0 = bo[k0], m1 = bo[k1];
    const int mb = m0 + (int)((int64_t)(m1 - m0) * rc / a.rchunks);
    const int me = m0 + (int)((int64_t)(m1 - m0) * (rc + 1) / a.rchunks);
    const int* srt = a.sorted + (size_t)g * a.N + mb;
    w_acc_members<T, E>(a, g, k0, wacc, me - mb, [&](int it) { return (int64_t)srt[it]; });
    __syncthreads();
  } else {
    const int64_t r0 = (int64_t)rc * a.rows_per_chunk;
    const int64_t r1 = min(a.N, r0 + a.rows_per_chunk);
    if (a.slices == 1) {
      w_acc_members<T, E>(a, g, k0, wacc, (int)(r1 - r0), [&](int it) { return r0 + it; });
      __syncthreads();
    } else {
      const uint16_t* asg = a.assign + (size_t)g * a.N;
      for (int64_t base = r0; base < r1; base += (int64_t)W_THREADS * W_ACC_BATCH) {
        if (tid == 0) nlist = 0;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < W_ACC_BATCH; ++q) {
          // one LDS atomic per wave: members are placed by their rank in the wave
          const int64_t row = base + (int64_t)q * W_THREADS + tid;
          const int k = row < r1 ? (int)asg[row] : -1;
          const bool in = k >= k0 && k < k1;
          const unsigned long long m = __ballot(in);
          const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
          int base_idx = 0;
          if (lane == 0 && m) base_idx = atomicAdd(&nlist, __popcll(m));
          base_idx = __shfl(base_idx, 0);
          if (in) list[base_idx + rank] = (int)(row - r0);
        }
        __syncthreads();
        w_acc_members<T, E>(a, g, k0, wacc, nlist, [&](int it) { return r0 + list[it]; });
        __syncthreads();
      }
    }
  }
  double* out = a.part + (((size_t)g * a.rchunks + rc) * a.K + k0) * S;
  const int n = (k1 - k0) * S;
  for (int e = tid; e < n; e += W_THREADS) out[e] = wacc[e];
}

// Weighted sums of eqs. 6-8 from the rows bucketed by codeword (d >= 64):
// one wave per codeword walks the codeword's members in bucket order and
// keeps the sums in float64 registers, written once as the single partial
// of the subspace (no LDS atomics: in bucket order consecutive members share
// a codeword, so atomics into one LDS slice all hit the same addresses).
// Lane groups of 16 lanes take one member each (four members side by side,
// w_smembers(E) per group in flight), lane i of a group holding elements
// [E i, E i + E) of the row (E = d / 16, vector loads); a member's norm is
// a 16-lane reduction, and the four groups' sums are added once at the end.
// The per-member products are formed as in w_acc_members.
// members per lane group in flight: eight up to d = 128, four at d = 256
// (where eight would leave two waves per SIMD)
__host__ __device__ constexpr int w_smembers(int E) { return E <= 8 ? 8 : 4; }
template <typename T> struct WVec;
template <> struct WVec<_Float16> {
  // E consecutive float16 elements (E a multiple of 4) as float
  template <int E> static __device__ __forceinline__ void load(const _Float16* p, float (&v)[E]) {
    typedef _Float16 h4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int q = 0; q < E / 4; ++q) {
      const h4 x = ((const h4*)p)[q];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[4 * q + u] = (float)x[u];
    }
  }
};
template <> struct WVec<float> {
  template <int E> static __device__ __forceinline__ void load(const float* p, float (&v)[E]) {
#pragma unroll
    for (int q = 0; q < E / 4; ++q) {
      const f4 x = ((const f4*)p)[q];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[4 * q + u] = x[u];
    }
  }
};

template <typename T, int E>
__global__ void __launch_bounds__(256) w_accumulate_sorted_kernel(WAccArgs a) {
  constexpr int SM = w_smembers(E);
  const int g = blockIdx.y;
  if (a.done && a.done[g]) return;
  const int lane = threadIdx.x & 63, grp = lane >> 4, li = lane & 15;
  // the wave's codeword, or its window of the bucketed rows past the
  // codeword blocks, in scalar registers (the bounds are then scalar loads)
  const int d = a.d, S = 2 * d + 2;
  const int* bo = a.boff + (size_t)g * (a.K + 1);
  const int nkb = (a.K + 3) / 4;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int m0, m1, mall;
  double* out;
  if ((int)blockIdx.x < nkb) {
    const int k = blockIdx.x * 4 + wv;
    if (k >= a.K) return;   // uniform per wave
    m0 = bo[k];
    mall = bo[k + 1];
    m1 = a.ovf ? min(mall, m0 + W_SORT_Q) : mall;
    out = a.part + ((size_t)g * a.rchunks * a.K + k) * S;
  } else {
    const int i = ((int)blockIdx.x - nkb) * 4 + wv;
    if (i >= a.nwin) return;
    const int k = a.wk[(size_t)g * a.nwin + i];
    if (k < 0) return;
    m0 = max(i * W_SORT_Q, bo[k] + W_SORT_Q);
    m1 = min(i * W_SORT_Q + W_SORT_Q, bo[k + 1]);
    mall = m1;
    out = a.ovf + ((size_t)g * a.nwin + i) * S;
  }
  const int* srt = a.sorted + (size_t)g * a.N;
  const T* X = (const T*)a.x + (int64_t)g * d + E * li;
  double sy[E], sx[E], wsum = 0.0;
#pragma unroll
  for (int e = 0; e < E; ++e) sy[e] = sx[e] = 0.0;
  constexpr int STEP = 4 * SM;   // members per batch and wave
  // member m + 4 u + grp of a batch (past the bucket's end a slot re-reads
  // the last member and adds nothing); the next batch's member ids are read
  // while this batch's rows are in flight, so a batch costs one memory round
  // trip (a crowded codeword is walked by its one wave alone)
  int rid[SM];
  if (m0 < m1) {
#pragma unroll
    for (int u = 0; u < SM; ++u) rid[u] = srt[min(m0 + 4 * u + grp, m1 - 1)];
  }
  for (int m = m0; m < m1; m += STEP) {
    float xv[SM][E], wt[SM];
#pragma unroll
    for (int u = 0; u < SM; ++u) {
      const int64_t row = rid[u];
      WVec<T>::template load<E>(X + row * a.ldx, xv[u]);
      wt[u] = a.w ? a.w[row] : 1.f;
    }
    if (m + STEP < m1) {
#pragma unroll
      for (int u = 0; u < SM; ++u) rid[u] = srt[min(m + STEP + 4 * u + grp, m1 - 1)];
    }
#pragma unroll
    for (int u = 0; u < SM; ++u) {
      float ss = xv[u][E - 1] * xv[u][E - 1];
#pragma unroll
      for (int e = E - 2; e >= 0; --e) ss = fmaf(xv[u][e], xv[u][e], ss);
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      if (m + 4 * u + grp < m1) {
        const float inv = __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(ss) + Y_EPS);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          sy[e] += (double)(xv[u][e] * (wt[u] * inv));
          sx[e] += (double)(xv[u][e] * wt[u]);
        }
        wsum += (double)wt[u];
      }
    }
  }
  // the four lane groups' sums (members of the same codeword)
#pragma unroll
  for (int off = 16; off < 64; off <<= 1) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      sy[e] += __shfl_xor(sy[e], off);
      sx[e] += __shfl_xor(sx[e], off);
    }
    wsum += __shfl_xor(wsum, off);
  }
  if (grp == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      out[E * li + e] = sy[e];
      out[d + E * li + e] = sx[e];
    }
    if (li == 0) {
      out[2 * d] = wsum;
      out[2 * d + 1] = (double)(mall - m0);
    }
  }
}

struct WFinArgs {
  int d, K, G, rchunks, T;
  int t;                  // iteration (1-based); 0 for the initial gains
  int no_early_stop, force_changed, nwg;
  const double* part;     // [G][rchunks][K][2d+2]
  const int* changed;     // [G][nwg]
  const double* obj;      // [G][nwg] or null
  const float* seednorm;  // [G][K]
  float* gain;            // [G][K]
  float* shape;           // [G][K][d]
  int* done;              // [G]: 0 running, else the iteration that stopped
  int* iters;             // [G]
  double* trace;          // [G][T] or null
  const int* xchanged;    // [G] changed flag of the exact kernel's rows
  const double* xobj;     // [G] their objective
  int kmeans;             // K-means baseline update instead of eqs. (7)(8)
  const double* ovf;      // [G][nwin][2d+2] window partials of the sorted sums, or null
  const int* boff;        // [G][K + 1] bucket offsets (with ovf)
  int nwin;
};

// Codebook update from the chunk partials (fixed order): d / E lanes per
// codeword, E elements per lane (E = 2, or 4 for d = 256).  Initial pass (t = 0): eq. (8) gains for
// the seed shapes (a codeword without members keeps its seed row's norm).
// Iteration: eqs. (7) and (8) with the safeguards; thread 0 of block 0
// applies the stop test of its subspace.  The trace entry (zeroed by the
// host) receives the objective by atomic adds.  K-means baseline: centroid
// = (sum w x) / W, held as norm and direction, and the trace is the
// distortion after the update, J_before - sum_k W_k ||m_k - c_k||^2 (the
// weighted mean m_k replacing the old centroid c_k), each block adding its
// codewords' share.
template <int E>
__global__ void __launch_bounds__(256) w_finalize_kernel(WFinArgs a) {
  __shared__ double red[4];
  const int g = blockIdx.y;
  if (a.t > 0 && a.done[g] != 0 && a.done[g] < a.t) return;
  const int d = a.d, K = a.K, S = 2 * d + 2;
  const int L = d / E;                 // lanes per codeword (power of two, <= 64)
  const int tid = threadIdx.x;
  const int k = blockIdx.x * (256 / L) + tid / L;
  const int li = tid % L;
  const bool active = k < K;
  const int kk = active ? k : K - 1;
  double sy[E], sx[E], W = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) sy[e] = sx[e] = 0.0;
  for (int c = 0; c < a.rchunks; ++c) {
    const double* p = a.part + (((size_t)g * a.rchunks + c) * K + kk) * S;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      sy[e] += p[E * li + e];
      sx[e] += p[d + E * li + e];
    }
    W += p[2 * d];
  }
  if (a.ovf) {
    // the codeword's members past its first W_SORT_Q, window by window
    const int* bo = a.boff + (size_t)g * (K + 1);
    const int m0 = bo[kk], m1 = bo[kk + 1];
    if (m1 - m0 > W_SORT_Q)
      for (int i = (m0 + W_SORT_Q) / W_SORT_Q; i <= (m1 - 1) / W_SORT_Q; ++i) {
        const double* p = a.ovf + ((size_t)g * a.nwin + i) * S;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          sy[e] += p[E * li + e];
          sx[e] += p[d + E * li + e];
        }
        W += p[2 * d];
      }
  }
  float* sk = a.shape + ((size_t)g * K + kk) * d;
  float* gk = a.gain + (size_t)g * K + kk;
  double sv[E];
#pragma unroll
  for (int e = 0; e < E; ++e) sv[e] = sk[E * li + e];
  double gnew = (a.t == 0) ? (double)a.seednorm[(size_t)g * K + kk] : (double)*gk;
  if (a.t > 0 && a.kmeans) {
    double drop = 0.0;
    if (W > 0.0) {
      double c[E], ee[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        c[e] = sx[e] / W;
        ee[e] = c[e] - gnew * sv[e];
      }
      double q = ee[E - 1] * ee[E - 1], cn = c[E - 1] * c[E - 1];
#pragma unroll
      for (int e = E - 2; e >= 0; --e) {
        q = fma(ee[e], ee[e], q);
        cn = fma(c[e], c[e], cn);
      }
      drop = W * q;
      for (int off = L / 2; off > 0; off >>= 1) cn += __shfl_xor(cn, off);
      cn = sqrt(cn);
#pragma unroll
      for (int e = 0; e < E; ++e) sv[e] = cn > 0.0 ? c[e] / cn : 0.0;
      gnew = cn;
    }
    if (!active) drop = 0.0;
    if (a.trace) {
      for (int off = 32; off > 0; off >>= 1) drop += __shfl_xor(drop, off);
      if ((tid & 63) == 0) red[tid >> 6] = drop;
      __syncthreads();
      if (tid == 0)
        atomicAdd(a.trace + (size_t)g * a.T + (a.t - 1), -(red[0] + red[1] + red[2] + red[3]));
    }
  } else if (W > 0.0) {
    if (a.t > 0) {
      double mn = sy[E - 1] * sy[E - 1];
#pragma unroll
      for (int e = E - 2; e >= 0; --e) mn = fma(sy[e], sy[e], mn);
      for (int off = L / 2; off > 0; off >>= 1) mn += __shfl_xor(mn, off);
      mn = sqrt(mn);
      if (mn > SHAPE_KEEP_REL * W) {
#pragma unroll
        for (int e = 0; e < E; ++e) sv[e] = sy[e] / mn;
      }
    }
    double pr = sx[E - 1] * sv[E - 1];
#pragma unroll
    for (int e = E - 2; e >= 0; --e) pr = fma(sx[e], sv[e], pr);
    for (int off = L / 2; off > 0; off >>= 1) pr += __shfl_xor(pr, off);
    gnew = fmax(0.0, pr / W);
  }
  if (active) {
#pragma unroll
    for (int e = 0; e < E; ++e) sk[E * li + e] = (float)sv[e];
    if (li == 0) *gk = (float)gnew;
  }
  if (a.t > 0 && blockIdx.x == 0 && tid < 64) {
    // stop test: the scoring workgroups' changed flags and objectives,
    // strided over the first wave and reduced in a fixed order
    int ch = 0;
    double obj = 0.0;
    for (int c = tid; c < a.nwg; c += 64) {
      ch |= a.changed[(size_t)g * a.nwg + c];
      if (a.obj) obj += a.obj[(size_t)g * a.nwg + c];
    }
    const bool any = __ballot(ch != 0) != 0ull;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) obj += __shfl_xor(obj, off);
    if (tid == 0) {
      const bool changed = any || a.force_changed || a.xchanged[g];
      if (a.obj) obj += a.xobj[g];
      if (a.trace) atomicAdd(a.trace + (size_t)g * a.T + (a.t - 1), obj);
      a.iters[g] = a.t;
      if (!changed && !a.no_early_stop) a.done[g] = a.t;
    }
  }
}

// --------------------------------------------------------------- decoders

struct WDecArgs {
  const uint32_t* codes;
  int64_t N, ldo;
  int d, K, G, M_use, b, words;
  const float* gain;
  const float* shape;
  void* out;
  int gpw, gblocks, vec;
  int64_t rows_per_wg;
  int tab_bytes;          // LDS kernel: table bytes (staged code words follow)
  int vshape;             // shape rows 16-byte aligned (vector table fill)
};

__device__ __forceinline__ int w_read_code(const uint32_t* cr, int64_t bit, int b) {
  const int64_t wi = bit >> 5;
  const int off = (int)(bit & 31);
  uint64_t v = cr[wi];
  if (off + b > 32) v |= (uint64_t)cr[wi + 1] << 32;
  return (int)((v >> off) & ((1ull << b) - 1));
}

template <typename TO> __device__ __forceinline__ void w_store8(TO* p, const float* v, bool vec,
                                                                int n);
template <> __device__ __forceinline__ void w_store8<_Float16>(_Float16* p, const float* v,
                                                               bool vec, int n) {
  if (vec) {
    h8 hv;
#pragma unroll
    for (int j = 0; j < 8; ++j) hv[j] = (_Float16)v[j];
    *(u4*)p = __builtin_bit_cast(u4, hv);
  } else {
    for (int j = 0; j < n; ++j) p[j] = (_Float16)v[j];
  }
}
template <> __device__ __forceinline__ void w_store8<float>(float* p, const float* v, bool vec,
                                                            int n) {
  if (vec) {
    ((f4*)p)[0] = (f4){v[0], v[1], v[2], v[3]};
    ((f4*)p)[1] = (f4){v[4], v[5], v[6], v[7]};
  } else {
    for (int j = 0; j < n; ++j) p[j] = v[j];
  }
}

// Code words of subspaces [g0, g0 + ngr) of stage m within a row: the
// word range [lo, lo + n) holding their b-bit fields.
__device__ __forceinline__ void w_stage_words(int m, int G, int g0, int ngr, int b, int& lo,
                                              int& n) {
  const int64_t first = ((int64_t)m * G + g0) * b;
  const int64_t last = first + (int64_t)ngr * b - 1;
  lo = (int)(first >> 5);
  n = (int)(last >> 5) - lo + 1;
}

// Swizzled decode-table entries: EW elements of type TT in NCH 16-byte
// chunks, chunk c of entry e in slot (c + e / (16 / NCH)) mod NCH.
template <typename TT, int EW> struct WTab {
  static constexpr int NCH = EW * (int)sizeof(TT) / 16;   // 16-byte chunks per entry
  static constexpr int PER = 16 / (int)sizeof(TT);        // elements per chunk
  static constexpr int SH = NCH == 4 ? 2 : (NCH == 2 ? 3 : 4);  // log2(16 / NCH)
};
template <typename TT, int EW>
__device__ __forceinline__ void w_tab_put(TT* tab, int e, const float (&v)[EW]) {
  using W = WTab<TT, EW>;
  u4* base = (u4*)tab + (size_t)e * W::NCH;
#pragma unroll
  for (int c = 0; c < W::NCH; ++c) {
    const int slot = (c + (e >> W::SH)) & (W::NCH - 1);
    u4 chunk;
    if (sizeof(TT) == 2) {
      h8 hv;
#pragma unroll
      for (int j = 0; j < 8; ++j) hv[j] = (_Float16)v[c * 8 + j];
      chunk = __builtin_bit_cast(u4, hv);
    } else {
      chunk = (u4){__float_as_uint(v[c * 4]), __float_as_uint(v[c * 4 + 1]),
                   __float_as_uint(v[c * 4 + 2]), __float_as_uint(v[c * 4 + 3])};
    }
    base[slot] = chunk;
  }
}
template <typename TT, int EW>
__device__ __forceinline__ void w_tab_add(const TT* tab, int e, float (&acc)[EW]) {
  using W = WTab<TT, EW>;
  const u4* base = (const u4*)tab + (size_t)e * W::NCH;
#pragma unroll
  for (int c = 0; c < W::NCH; ++c) {
    const u4 chunk = base[(c + (e >> W::SH)) & (W::NCH - 1)];
    if (sizeof(TT) == 2) {
      const h8 hv = __builtin_bit_cast(h8, chunk);
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[c * 8 + j] += (float)hv[j];
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[c * 4 + j] += __uint_as_float(chunk[j]);
    }
  }
}

// Gather-sum decoder with the codeword table (g s, float32 or, for one
// float16 stage, float16) of `gpw` subspaces in LDS; entries of EW = 8 C
// elements.  One thread per (row, subspace), subspace fastest.  The code
// words of the workgroup's rows and subspaces are staged in LDS with the
// table ([rows][words of stage 0, stage 1, ...]), so the output loop issues
// no global loads (a wait for a load would also wait for the stores issued
// before it).
template <typename TO, typename TT, int C>
__global__ void __launch_bounds__(W_DEC_THREADS) w_decode_lds_kernel(WDecArgs a) {
  extern __shared__ __align__(16) unsigned char wdec_smem[];
  constexpr int EW = 8 * C;
  TT* tab = (TT*)wdec_smem;
  uint32_t* cwl = (uint32_t*)(wdec_smem + a.tab_bytes);
  const int gpw = a.gpw;
  const int id = blockIdx.x;
  const int xcd = id % 8, slot = id / 8;
  const int gb = slot % a.gblocks;
  const int rc = (slot / a.gblocks) * 8 + xcd;
  const int64_t r_begin = (int64_t)rc * a.rows_per_wg;
  if (r_begin >= a.N) return;
  const int64_t r_end = min(a.N, r_begin + a.rows_per_wg);
  const int nrows = (int)(r_end - r_begin);
  const int g0 = gb * gpw;
  const int ngr = min(gpw, a.G - g0);
  const int K = a.K, M = a.M_use, d = a.d, G = a.G, b = a.b;
  const int tid = threadIdx.x;
  // staged code words per row (host-checked: nrows * rs <= W_DEC_CODE_PT * W_DEC_THREADS)
  int rs = 0;
  for (int m = 0; m < M; ++m) {
    int lo, n;
    w_stage_words(m, G, g0, ngr, b, lo, n);
    rs += n;
  }
  const int ncw = nrows * rs;
  const uint32_t* crow = a.codes + r_begin * a.words;
  uint32_t cw[W_DEC_CODE_PT];
#pragma unroll
  for (int q = 0; q < W_DEC_CODE_PT; ++q) {
    if (q * W_DEC_THREADS < ncw) {         // uniform per q
      const int e = min(q * W_DEC_THREADS + tid, ncw - 1);
      const int row = e / rs;
      int j = e - row * rs, m = 0, lo, n;
      w_stage_words(0, G, g0, ngr, b, lo, n);
      while (j >= n) {
        j -= n;
        ++m;
        w_stage_words(m, G, g0, ngr, b, lo, n);
      }
      cw[q] = crow[(int64_t)row * a.words + lo + j];
    }
  }
  // table fill: entry e = (gi M + m) K + k holds g s of codeword k, as NCH
  // 16-byte chunks; chunk c sits in slot (c + e / (16 / NCH)) mod NCH, so
  // entries that share LDS banks (e mod 16/NCH) differ in which chunk they
  // keep where, and random lookups spread over all bank groups
  const int entries = ngr * M * K;
  for (int e = tid; e < entries; e += W_DEC_THREADS) {
    const int k = e & (K - 1), q2 = e >> b;
    const int m = q2 % M, gi = q2 / M;
    const size_t cb = (size_t)m * G + g0 + gi;
    const float gk = a.gain[cb * K + k];
    const float* sv = a.shape + (cb * K + k) * d;
    float v[EW];
    if (d == EW && a.vshape) {
#pragma unroll
      for (int j = 0; j < EW; j += 4) {
        const f4 t = *(const f4*)(sv + j);
        v[j] = t[0]; v[j + 1] = t[1]; v[j + 2] = t[2]; v[j + 3] = t[3];
      }
    } else {
#pragma unroll
      for (int j = 0; j < EW; ++j) v[j] = j < d ? sv[j] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < EW; ++j) v[j] *= gk;
    w_tab_put<TT, EW>(tab, e, v);
  }
#pragma unroll
  for (int q = 0; q < W_DEC_CODE_PT; ++q) {
    const int e = q * W_DEC_THREADS + tid;
    if (e < ncw) cwl[e] = cw[q];
  }
  __syncthreads();
  const int gi = tid % gpw;
  if (gi >= ngr) return;
  const int rstep = W_DEC_THREADS / gpw;
  const int g = g0 + gi;
  constexpr int RBATCH = C == 1 ? 4 : 2;    // rows in flight per thread (no spills)
  for (int r0 = tid / gpw; r0 < nrows; r0 += RBATCH * rstep) {
    float acc[RBATCH][EW];
#pragma unroll
    for (int q = 0; q < RBATCH; ++q)
#pragma unroll
      for (int j = 0; j < EW; ++j) acc[q][j] = 0.f;
    int off = 0;                            // staged words of the stages before m
    for (int m = 0; m < M; ++m) {
      int lo, n;
      w_stage_words(m, G, g0, ngr, b, lo, n);
      const int p = (int)(((int64_t)m * G + g) * b - (int64_t)lo * 32);
      const int wi = off + (p >> 5), sh = p & 31;
      const bool two = sh + b > 32;
      int k[RBATCH];
#pragma unroll
      for (int q = 0; q < RBATCH; ++q) {
        int row = r0 + q * rstep;
        row = row < nrows ? row : 0;        // in range; its result is not stored
        const uint32_t* w = cwl + row * rs + wi;
        uint64_t v = w[0];
        if (two) v |= (uint64_t)w[1] << 32;
        k[q] = (int)((v >> sh) & ((1ull << b) - 1));
      }
#pragma unroll
      for (int q = 0; q < RBATCH; ++q)
        w_tab_add<TT, EW>(tab, (gi * M + m) * K + k[q], acc[q]);
      off += n;
    }
#pragma unroll
    for (int q = 0; q < RBATCH; ++q) {
      const int row = r0 + q * rstep;
      if (row >= nrows) break;
      TO* dst = (TO*)a.out + (r_begin + row) * a.ldo + (int64_t)g * d;
#pragma unroll
      for (int c8 = 0; c8 < C; ++c8)
        w_store8<TO>(dst + 8 * c8, acc[q] + 8 * c8, a.vec != 0, min(8, d - 8 * c8));
    }
  }
}

// Gather-sum decoder for codebooks too large for LDS: C lanes per (row,
// subspace), eight elements per lane, codewords read from global memory.
template <typename TO>
__global__ void __launch_bounds__(256) w_decode_gather_kernel(WDecArgs a, int C) {
  const int tid = threadIdx.x;
  const int per_block = 256 / C;
  const int64_t item = (int64_t)blockIdx.x * per_block + tid / C;
  const int q = tid % C;
  if (tid / C >= per_block || item >= a.N * a.G) return;
  const int64_t row = item / a.G;
  const int g = (int)(item % a.G);
  const int d = a.d, K = a.K;
  const uint32_t* cr = a.codes + row * a.words;
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  for (int m = 0; m < a.M_use; ++m) {
    const int k = w_read_code(cr, ((int64_t)m * a.G + g) * a.b, a.b);
    const size_t cb = (size_t)m * a.G + g;
    const float gk = a.gain[cb * K + k];
    const float* sv = a.shape + (cb * K + k) * d + 8 * q;
    {
      // the codeword g s is rounded to float32 before the stage sum (no
      // fused multiply-add), as the decode contract states
#pragma clang fp contract(off)
      if (a.vec) {
        const f4 lo = ((const f4*)sv)[0], hi = ((const f4*)sv)[1];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[j] += gk * lo[j];
          acc[4 + j] += gk * hi[j];
        }
      } else {
        for (int j = 0; j < 8 && 8 * q + j < d; ++j) acc[j] += gk * sv[j];
      }
    }
  }
  TO* dst = (TO*)a.out + row * a.ldo + (int64_t)g * d + 8 * q;
  w_store8<TO>(dst, acc, a.vec != 0, min(8, d - 8 * q));
}

// ------------------------------------------------------------- host side

int w_groups(int d) { return (d + 7) / 8; }

// Template width C (1, 2, 4, 8, 16) that holds d elements.
int w_cwidth(int d) {
  const int c = w_groups(d);
  int C = 1;
  while (C < c) C *= 2;
  return C;
}

struct WLayout {
  int C, QF, tiles, nwg, rounds, tpc, map_xcd, lg;
  size_t frag_bytes;
  bool resident;
  bool sp;              // single-pass scoring (d >= 64), then the hi/lo pass
  int Qu;
  size_t lds;
};

// Subvectors of at least 64 elements are scored in a single float16 pass
// (P + 1 MFMAs per tile), the few rows it cannot decide in the hi/lo pass.
// Narrower ones, and codebooks below 1024 codewords, keep the hi/lo pass
// alone: there the MFMA chain is short (or the launch is bound by the rows'
// traffic) and the single pass's second-best bookkeeping and second pass
// would cost more than the MFMAs it saves.
constexpr int W_SP_MIN_C = 8;
constexpr int W_SP_MIN_TILES = 32;   // K >= 1024: below, scoring is not MFMA-bound
constexpr int W_HP_WGS = 1024;  // workgroups of the hi/lo pass over listed rows
constexpr int W_HP_SLICES = 8;  // codebook slices of that pass
constexpr int W_SP_RESIDENT_BYTES = 78 * 1024;   // single-pass table kept whole in LDS

// Launch geometry of the scoring kernel for one stage input type; hp: the
// hi/lo pass (every fragment staged) even where the single pass applies.
WLayout w_score_layout(const gsrq_shape* s, size_t x_elt, bool f16rows, bool hp = false) {
  WLayout L;
  const int64_t G = s->D / s->d;
  L.C = w_cwidth(s->d);
  L.QF = w_frags(L.C);
  L.tiles = (s->K + CW - 1) / CW;
  L.frag_bytes = (size_t)L.tiles * L.QF * 64 * sizeof(u4);
  L.sp = !hp && L.C >= W_SP_MIN_C && L.tiles >= W_SP_MIN_TILES;
  L.Qu = L.sp ? w_pairs(L.C) + 1 : L.QF;
  (void)f16rows;
  const size_t used = (size_t)L.tiles * L.Qu * 64 * sizeof(u4);
  // single pass: two workgroups per CU share 160 KiB of LDS
  L.resident = used <= (size_t)(L.sp ? W_SP_RESIDENT_BYTES : W_RESIDENT_BYTES);
  // rows per workgroup round: W_ROWS per row block a wave scores at once
  const int64_t rows_round = (int64_t)RB * w_score_waves(L.C, L.resident, L.sp, false) *
                             w_row_blocks(L.C, L.resident, L.sp, false);
  const int64_t row_rounds = (s->N + rows_round - 1) / rows_round;
  if (L.resident) {
    // enough rounds per workgroup to amortise the table load, while
    // keeping about four workgroups per CU in the grid
    int64_t r = (row_rounds * G + (L.sp ? 511 : 1023)) / (L.sp ? 512 : 1024);
    if (r < 1) r = 1;
    L.rounds = (int)r;
    L.tpc = 0;
    L.lds = used;
  } else {
    L.rounds = 1;
    L.tpc = std::max(1, (int)((L.sp ? w_sp_stream_bytes(w_score_waves(L.C, false, true, false))
                                    : W_STREAM_BYTES) /
                              (L.Qu * 64 * sizeof(u4))));
    L.lds = 2 * (size_t)L.tpc * L.Qu * 64 * sizeof(u4);
  }
  L.nwg = (int)((row_rounds + L.rounds - 1) / L.rounds);
  const size_t seg = (size_t)s->d * x_elt;
  L.lg = seg < 128 ? (int)(128 / seg) : 1;
  L.map_xcd = (G % (8 * L.lg) == 0) ? 1 : 0;
  return L;
}

size_t w_stream_need(const WLayout& L) {
  return 2 * (size_t)L.tpc * L.Qu * 64 * sizeof(u4);
}

template <typename T, int C, int MODE, bool SP, bool IND>
gsrq_status w_score_launch_v(const WScoreArgs& a, const WLayout& L, hipStream_t st) {
  const dim3 grid((unsigned)(a.G * a.nwg * (IND ? a.nslice : 1)));
  // a streamed d = 256 tile pair (2 x 33 KiB) exceeds the default 64 KiB of
  // dynamic LDS
  const void* fn = L.resident ? (const void*)w_score_kernel<T, C, MODE, true, SP, IND>
                              : (const void*)w_score_kernel<T, C, MODE, false, SP, IND>;
  if (L.lds > 65536 &&
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)L.lds) !=
          hipSuccess)
    return GSRQ_E_HIP;
  if (L.resident)
    w_score_kernel<T, C, MODE, true, SP, IND>
        <<<grid, w_score_waves(C, true, SP, IND) * 64, L.lds, st>>>(a);
  else
    w_score_kernel<T, C, MODE, false, SP, IND>
        <<<grid, w_score_waves(C, false, SP, IND) * 64, L.lds, st>>>(a);
  return launch_ok();
}

// The scoring launch(es) of one pass: the hi/lo kernel over every row, or
// (d >= 64) the single pass over every row and then the hi/lo kernel over
// the rows it listed.
template <typename T, int C, int MODE>
gsrq_status w_score_launch_c(const WScoreArgs& a, const WLayout& L, hipStream_t st) {
  if constexpr (C >= W_SP_MIN_C) {
    if (L.sp) {
      gsrq_status e = w_score_launch_v<T, C, MODE, true, false>(a, L, st);
      if (e) return e;
      // hi/lo pass over the listed rows: the codebook in W_HP_SLICES
      // slices (streamed through LDS), about W_HP_WGS workgroups in all
      gsrq_shape s1 = {a.N, a.G * a.d, a.d, a.K, 1};
      WLayout H = w_score_layout(&s1, sizeof(T), sizeof(T) == 2, true);
      const int tile_bytes = H.Qu * 64 * (int)sizeof(u4);
      WScoreArgs b = a;
      b.nslice = std::min(W_HP_SLICES, a.tiles);
      b.tps = (a.tiles + b.nslice - 1) / b.nslice;
      b.nslice = (a.tiles + b.tps - 1) / b.tps;
      b.nwg = std::max(1, W_HP_WGS * (W_WAVES / w_score_waves(C, false, false, true)) /
                              (a.G * b.nslice));
      b.map_xcd = 0;
      H.resident = (size_t)b.tps * tile_bytes <= (size_t)W_RESIDENT_BYTES;
      if (H.resident) H.lds = (size_t)b.tps * tile_bytes;
      b.tpc = H.tpc;
      if ((e = w_score_launch_v<T, C, MODE, false, true>(b, H, st))) return e;
      w_listed_finish_kernel<T, MODE><<<dim3(64, a.G), 256, 0, st>>>(a);
      return launch_ok();
    }
  }
  return w_score_launch_v<T, C, MODE, false, false>(a, L, st);
}

template <typename T, int MODE>
gsrq_status w_score_launch(const WScoreArgs& a, const WLayout& L, hipStream_t st) {
  switch (L.C) {
    case 1: return w_score_launch_c<T, 1, MODE>(a, L, st);
    case 2: return w_score_launch_c<T, 2, MODE>(a, L, st);
    case 4: return w_score_launch_c<T, 4, MODE>(a, L, st);
    case 8: return w_score_launch_c<T, 8, MODE>(a, L, st);
    case 16: return w_score_launch_c<T, 16, MODE>(a, L, st);
    case 32: return w_score_launch_c<T, 32, MODE>(a, L, st);
  }
  return GSRQ_E_UNSUPPORTED;
}

// Deferred-row state of the G codebooks a scoring launch uses: smallest
// gains, row lists and what the exact kernel adds to the stop test and the
// objective.
struct WDefer {
  float* gmin;      // [G] smallest gains, then [G] largest
  int* xcount;      // [G]
  int* xrows;       // [G][N]
  int* xchanged;    // [G]
  double* xobj;     // [G]
  int* hcount;      // [G] rows listed by the single pass (null: no single pass)
  int* hrows;       // [G][N]
  unsigned long long* hbest;   // [G][N]
  float* hrr;       // [G][N]
};

// Fragment tables (and sigma, smallest gain, cleared deferred-row state) of
// the `ncb` codebooks starting at cb0.
gsrq_status w_build_frags(const float* gain, const float* shape, int d, int K, int C, int ncb,
                          int cb0, bool unit_gain, const int* done, int G, int* sig, u4* frag,
                          const WDefer& X, hipStream_t st) {
  TimedLaunch tl(GSRQ_KERNEL_FRAGMENTS, st);
  const int tiles = (K + CW - 1) / CW;
  const dim3 fgrid(tiles, ncb);
  const int ug = unit_gain ? 1 : 0;
  const WDeferPtrs xp{X.gmin, X.xcount, X.xchanged, X.xobj, X.hcount};
  auto go = [&](auto kern) {
    kern<<<fgrid, 64, 0, st>>>(gain, shape, d, K, ug, sig, done, G, cb0, frag, xp);
  };
  switch (w_pairs(C)) {
    case 1: go(w_frag_kernel<1>); break;
    case 2: go(w_frag_kernel<2>); break;
    case 4: go(w_frag_kernel<4>); break;
    case 8: go(w_frag_kernel<8>); break;
    case 16: go(w_frag_kernel<16>); break;
    default: return GSRQ_E_UNSUPPORTED;
  }
  return launch_ok();
}

// A scoring launch, then the exact kernel for the rows it deferred (about
// 512 workgroups in all: most subspaces defer few rows or none, and an empty
// workgroup only reads its count).
constexpr int W_XWGS = 512;

template <typename T, int MODE>
gsrq_status w_score_and_exact(const WScoreArgs& a, const WLayout& L, int kind, hipStream_t st) {
  gsrq_status e;
  {
    TimedLaunch tl(kind, st);
    if ((e = w_score_launch<T, MODE>(a, L, st))) return e;
  }
  TimedLaunch tl(GSRQ_KERNEL_EXACT, st);
  const int per_g = std::max(1, std::min(64, W_XWGS / a.G));
  w_exact_kernel<T, MODE><<<dim3(per_g, a.G), W_XTHREADS, 0, st>>>(a);
  return launch_ok();
}

struct WAccLayout {
  int ks, slices, rchunks;
  int64_t rows_per_chunk;
  size_t lds;
  bool bucket;          // rows bucketed by codeword before accumulating
  bool sorted_sums;     // bucketed sums by w_accumulate_sorted_kernel
};

WAccLayout w_acc_layout(const gsrq_shape* s) {
  WAccLayout A;
  const int64_t G = s->D / s->d;
  const size_t per_k = (size_t)(2 * s->d + 2) * sizeof(double);
  int ks = 1;
  while (ks * 2 <= s->K && (size_t)(ks * 2) * per_k <= (size_t)W_ACC_LDS_BYTES) ks *= 2;
  A.ks = ks;
  A.slices = (s->K + ks - 1) / ks;
  int64_t rc = (1024 + A.slices * G - 1) / (A.slices * G);
  const int64_t max_rc = (s->N + 2047) / 2048;
  if (rc > max_rc) rc = max_rc;
  if (rc < 1) rc = 1;
  A.rows_per_chunk = (s->N + rc - 1) / rc;
  A.rchunks = (int)((s->N + A.rows_per_chunk - 1) / A.rows_per_chunk);
  A.lds = (size_t)ks * per_k;
  // several slices: bucket the rows by codeword once per pass instead of
  // every slice scanning every row (the histogram is K ints of LDS)
  A.bucket = A.slices > 1 && s->K <= W_BUCKET_KMAX;
  // bucketed rows with d >= 64: one wave per codeword sums in registers
  // (w_accumulate_sorted_kernel), one partial per subspace
  A.sorted_sums = A.bucket && s->d >= 64 && s->d <= 256;
  if (A.sorted_sums) {
    A.rchunks = 1;
    A.rows_per_chunk = s->N;
  }
  return A;
}

struct WTrainWs {
  size_t frag, gmin, xcount, xrows, xchanged, xobj, hcount, hrows, hbest, hrr, sig, part,
      changed, obj, assign, done, iters, seednorm, seeds, sorted, boff, bcnt, ovf, wk, total;
};

WTrainWs w_train_ws(const gsrq_shape* s, size_t x_elt) {
  WTrainWs W;
  const int64_t G = s->D / s->d;
  // the larger of the two geometries (a later stage may train on float32)
  const WLayout L16 = w_score_layout(s, x_elt, x_elt == 2);
  const WAccLayout A = w_acc_layout(s);
  size_t off = 0;
  W.frag = off; off = align256(off + (size_t)G * L16.frag_bytes);
  W.gmin = off; off = align256(off + 2 * (size_t)G * sizeof(float));
  W.xcount = off; off = align256(off + (size_t)G * sizeof(int));
  W.xrows = off; off = align256(off + (size_t)G * s->N * sizeof(int));
  W.xchanged = off; off = align256(off + (size_t)G * sizeof(int));
  W.xobj = off; off = align256(off + (size_t)G * sizeof(double));
  W.hcount = off; off = align256(off + (L16.sp ? (size_t)G * sizeof(int) : 0));
  W.hrows = off; off = align256(off + (L16.sp ? (size_t)G * s->N * sizeof(int) : 0));
  W.hbest = off; off = align256(off + (L16.sp ? (size_t)G * s->N * 8 : 0));
  W.hrr = off; off = align256(off + (L16.sp ? (size_t)G * s->N * sizeof(float) : 0));
  W.sig = off; off = align256(off + (size_t)G * sizeof(int));
  W.part = off;
  off = align256(off + (size_t)G * A.rchunks * s->K * (2 * s->d + 2) * sizeof(double));
  W.changed = off; off = align256(off + (size_t)G * L16.nwg * sizeof(int));
  W.obj = off; off = align256(off + (size_t)G * L16.nwg * sizeof(double));
  W.assign = off; off = align256(off + (size_t)G * s->N * sizeof(uint16_t));
  W.done = off; off = align256(off + (size_t)G * sizeof(int));
  W.iters = off; off = align256(off + (size_t)G * sizeof(int));
  W.seednorm = off; off = align256(off + (size_t)G * s->K * sizeof(float));
  W.seeds = off; off = align256(off + (size_t)G * s->K * sizeof(int32_t));
  W.sorted = off; off = align256(off + (A.bucket ? (size_t)G * s->N * sizeof(int) : 0));
  W.boff = off; off = align256(off + (A.bucket ? (size_t)G * (s->K + 1) * sizeof(int) : 0));
  W.bcnt = off;
  const int64_t bch = w_bucket_rows(s->N, s->K);
  off = align256(off + (A.bucket ? (size_t)G * ((s->N + bch - 1) / bch) * s->K * sizeof(int) : 0));
  const size_t nwin = A.sorted_sums ? (size_t)w_sort_windows(s->N) : 0;
  W.ovf = off; off = align256(off + (size_t)G * nwin * (2 * s->d + 2) * sizeof(double));
  W.wk = off; off = align256(off + (size_t)G * nwin * sizeof(int));
  W.total = off;
  return W;
}

struct WEncWs {
  size_t frag, gmin, xcount, xrows, xchanged, xobj, hcount, hrows, hbest, hrr, sig, res0, res1,
      total;
};

// Several stages of narrow wide rows (d <= 16) with resident fragment
// tables are encoded by the stage-fused kernel.
bool w_fused(const gsrq_shape* s) {
  if (s->M <= 1 || w_cwidth(s->d) > 2) return false;
  return w_score_layout(s, 4, false).resident;
}

// Several stages at d = 64 or 128 scored by the hi/lo pass (K <= 512) whose
// stage table fits in LDS: one stage-fused launch (w_encode_fused_wide_kernel).
bool w_fused_wide(const gsrq_shape* s) {
  const int C = w_cwidth(s->d);
  if (s->M <= 1 || (C != 8 && C != 16) || s->K > W_FW_KMAX) return false;
  const WLayout L = w_score_layout(s, 4, false);
  return !L.sp && (size_t)L.tiles * L.QF * 64 * sizeof(u4) <= (size_t)W_FW_LDS_MAX;
}

WEncWs w_encode_ws(const gsrq_shape* s) {
  WEncWs W;
  const int64_t G = s->D / s->d;
  const WLayout L = w_score_layout(s, 4, false);
  size_t off = 0;
  if (w_fused(s) || w_fused_wide(s)) {
    // every stage's fragment table, per-codebook sigma state; no residual
    // buffers and no deferred-row lists
    const size_t ncb = (size_t)s->M * G;
    W.frag = off; off = align256(off + ncb * L.frag_bytes);
    W.gmin = off; off = align256(off + 2 * ncb * sizeof(float));
    W.xcount = off; off = align256(off + ncb * sizeof(int));
    W.xrows = off;
    W.xchanged = off; off = align256(off + ncb * sizeof(int));
    W.xobj = off; off = align256(off + ncb * sizeof(double));
    W.hcount = W.hrows = W.hbest = W.hrr = off;
    W.sig = off; off = align256(off + ncb * sizeof(int));
    W.res0 = W.res1 = off;
    W.total = std::max(off, (size_t)256);
    return W;
  }
  W.frag = off; off = align256(off + (size_t)G * L.frag_bytes);
  W.gmin = off; off = align256(off + 2 * (size_t)G * sizeof(float));
  W.xcount = off; off = align256(off + (size_t)G * sizeof(int));
  W.xrows = off; off = align256(off + (size_t)G * s->N * sizeof(int));
  W.xchanged = off; off = align256(off + (size_t)G * sizeof(int));
  W.xobj = off; off = align256(off + (size_t)G * sizeof(double));
  W.hcount = off; off = align256(off + (L.sp ? (size_t)G * sizeof(int) : 0));
  W.hrows = off; off = align256(off + (L.sp ? (size_t)G * s->N * sizeof(int) : 0));
  W.hbest = off; off = align256(off + (L.sp ? (size_t)G * s->N * 8 : 0));
  W.hrr = off; off = align256(off + (L.sp ? (size_t)G * s->N * sizeof(float) : 0));
  W.sig = off; off = align256(off + (size_t)s->M * G * sizeof(int));
  W.res0 = W.res1 = off;
  if (s->M > 1) {
    W.res0 = off; off = align256(off + (size_t)s->N * s->D * sizeof(float));
    W.res1 = off; off = align256(off + (size_t)s->N * s->D * sizeof(float));
  }
  W.total = std::max(off, (size_t)256);
  return W;
}

// One encode stage: input rows (type T) -> code bits of stage m and the
// residual (optional).  The stage's fragment table must be built.
template <typename T>
gsrq_status w_encode_stage(const gsrq_shape* s, int m, const void* x, int64_t ldx,
                           const float* gain, const float* shape, const int* sig, const u4* frag,
                           const WDefer& X, uint32_t* codes, int words, float* res_out,
                           hipStream_t st) {
  const bool f16 = sizeof(T) == 2;
  const WLayout L = w_score_layout(s, sizeof(T), f16);
  WScoreArgs a = {};
  a.x = x; a.ldx = ldx; a.N = s->N; a.d = s->d; a.K = s->K; a.G = s->D / s->d;
  a.tiles = L.tiles; a.QF = L.QF; a.cb0 = m * a.G; a.fcb0 = m * a.G;
  a.frag = frag; a.sig = sig; a.gain = gain; a.shape = shape; a.unit_gain = 0;
  a.gmin = X.gmin; a.xcount = X.xcount; a.xrows = X.xrows; a.xchanged = X.xchanged;
  a.xobj = X.xobj; a.hcount = X.hcount; a.hrows = X.hrows; a.hbest = X.hbest; a.hrr = X.hrr;
  a.codes = codes; a.words = words; a.b = log2i(s->K); a.m = m; a.res_out = res_out;
  a.nwg = L.nwg; a.rounds = L.rounds; a.tpc = L.tpc; a.map_xcd = L.map_xcd; a.lg = L.lg;
  return w_score_and_exact<T, W_ENCODE>(a, L, GSRQ_KERNEL_ENCODE, st);
}

template <typename T>
gsrq_status w_train(const gsrq_shape* s, const void* X, int64_t ldx, const float* w, int T_,
                    const int32_t* seed_rows, uint32_t flags, float* gain, float* shape,
                    float* R_next, uint16_t* assign_io, int32_t* iters_run, double* obj_trace,
                    void* ws, hipStream_t st) {
  const int G = s->D / s->d;
  const int d = s->d, K = s->K;
  const bool f16 = sizeof(T) == 2;
  const WLayout L = w_score_layout(s, sizeof(T), f16);
  const WAccLayout A = w_acc_layout(s);
  const WTrainWs W = w_train_ws(s, sizeof(T));
  char* base = (char*)ws;
  u4* frag = (u4*)(base + W.frag);
  const WDefer XD = {(float*)(base + W.gmin), (int*)(base + W.xcount), (int*)(base + W.xrows),
                     (int*)(base + W.xchanged), (double*)(base + W.xobj),
                     W.hrows > W.hcount ? (int*)(base + W.hcount) : nullptr,
                     W.hrows > W.hcount ? (int*)(base + W.hrows) : nullptr,
                     W.hrows > W.hcount ? (unsigned long long*)(base + W.hbest) : nullptr,
                     W.hrows > W.hcount ? (float*)(base + W.hrr) : nullptr};
  int* sig = (int*)(base + W.sig);
  double* part = (double*)(base + W.part);
  int* changed = (int*)(base + W.changed);
  double* objp = (double*)(base + W.obj);
  uint16_t* assign = assign_io ? assign_io : (uint16_t*)(base + W.assign);
  int* done = (int*)(base + W.done);
  int* iters = iters_run ? (int*)iters_run : (int*)(base + W.iters);
  float* seednorm = (float*)(base + W.seednorm);
  int32_t* seeds = (int32_t*)(base + W.seeds);
  gsrq_status e;
  if ((e = fill_u32(done, G, 0, st))) return e;
  if ((e = fill_u32(iters, G, 0, st))) return e;
  if (obj_trace && T_ > 0 && (e = fill_u32(obj_trace, (size_t)G * T_ * 2, 0, st))) return e;
  const int kmeans = (flags & GSRQ_KMEANS) ? 1 : 0;

  WScoreArgs sa = {};
  sa.x = X; sa.ldx = ldx; sa.N = s->N; sa.d = d; sa.K = K; sa.G = G;
  sa.tiles = L.tiles; sa.QF = L.QF; sa.cb0 = 0; sa.fcb0 = 0; sa.frag = frag; sa.sig = sig;
  sa.gmin = XD.gmin; sa.xcount = XD.xcount; sa.xrows = XD.xrows; sa.xchanged = XD.xchanged;
  sa.xobj = XD.xobj; sa.hcount = XD.hcount; sa.hrows = XD.hrows; sa.hbest = XD.hbest;
  sa.hrr = XD.hrr;
  sa.gain = gain; sa.shape = shape; sa.w = w; sa.done = done; sa.assign = assign;
  sa.changed = changed; sa.obj = nullptr;
  sa.nwg = L.nwg; sa.rounds = L.rounds; sa.tpc = L.tpc; sa.map_xcd = L.map_xcd; sa.lg = L.lg;

  WAccArgs aa;
  aa.x = X; aa.ldx = ldx; aa.N = s->N; aa.d = d; aa.K = K; aa.G = G; aa.w = w;
  aa.assign = assign; aa.done = done; aa.part = part;
  aa.ks = A.ks; aa.slices = A.slices; aa.rchunks = A.rchunks; aa.rows_per_chunk = A.rows_per_chunk;
  aa.sorted = A.bucket ? (const int*)(base + W.sorted) : nullptr;
  aa.boff = A.bucket ? (const int*)(base + W.boff) : nullptr;
  aa.nwin = A.sorted_sums ? w_sort_windows(s->N) : 0;
  aa.wk = A.sorted_sums ? (const int*)(base + W.wk) : nullptr;
  aa.ovf = nullptr;       // set per launch: the sorted-sum kernel only
  const dim3 agrid((unsigned)(A.slices * A.rchunks), (unsigned)G);

  WFinArgs fa;
  fa.d = d; fa.K = K; fa.G = G; fa.rchunks = A.rchunks; fa.T = T_; fa.t = 0;
  fa.no_early_stop = (flags & GSRQ_NO_EARLY_STOP) ? 1 : 0;
  fa.force_changed = 0; fa.nwg = L.nwg; fa.part = part; fa.changed = changed; fa.obj = nullptr;
  fa.seednorm = seednorm; fa.gain = gain; fa.shape = shape; fa.done = done; fa.iters = iters;
  fa.trace = obj_trace; fa.xchanged = XD.xchanged; fa.xobj = XD.xobj; fa.kmeans = kmeans;
  fa.ovf = nullptr; fa.boff = aa.boff; fa.nwin = aa.nwin;
  // elements per lane of the accumulation and the update: lane groups of
  // d / E lanes, at most one wave
  const bool e4 = d > 128;
  const int cpb = 256 / (d / (e4 ? 4 : 2));
  const dim3 fgrid((unsigned)((K + cpb - 1) / cpb), (unsigned)G);

  // the accumulator slice can exceed the default dynamic LDS limit
  if (hipFuncSetAttribute(e4 ? (const void*)w_accumulate_kernel<T, 4>
                             : (const void*)w_accumulate_kernel<T, 2>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)A.lds) != hipSuccess)
    return GSRQ_E_HIP;
  auto accumulate_finalize = [&]() -> gsrq_status {
    gsrq_status e2;
    {
      TimedLaunch tl(GSRQ_KERNEL_ACCUMULATE, st);
      if (A.bucket) {
        const int64_t bch = w_bucket_rows(s->N, K);
        const int bchunks = (int)((s->N + bch - 1) / bch);
        int* bcnt = (int*)(base + W.bcnt);
        w_bucket_count_kernel<<<dim3(bchunks, G), 256, (size_t)K * sizeof(int), st>>>(
            assign, s->N, K, bch, aa.done, bcnt);
        const size_t slds = (size_t)bchunks * K * sizeof(int);   // <= 128 KiB
        if (slds > 65536 &&
            hipFuncSetAttribute((const void*)w_bucket_scan_kernel,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)slds) != hipSuccess)
          return GSRQ_E_HIP;
        w_bucket_scan_kernel<<<G, 1024, slds, st>>>(s->N, K, bchunks, aa.done, bcnt,
                                                    (int*)(base + W.boff), aa.nwin,
                                                    (int*)aa.wk);
        w_bucket_scatter_kernel<<<dim3(bchunks, G), 256, (size_t)K * sizeof(int), st>>>(
            assign, s->N, K, bch, aa.done, bcnt, (int*)(base + W.sorted));
        if ((e2 = launch_ok())) return e2;
      }
      // the register kernel reads E consecutive elements with vector loads:
      // 16-byte aligned rows (else the LDS kernel, with the same single
      // row chunk)
      const bool svec = ((uintptr_t)X % 16 == 0) && ((ldx * (int64_t)sizeof(T)) % 16 == 0);
      aa.ovf = (A.sorted_sums && svec) ? (double*)(base + W.ovf) : nullptr;
      fa.ovf = aa.ovf;
      if (A.sorted_sums && svec) {
        const dim3 sgrid((unsigned)((K + 3) / 4 + (aa.nwin + 3) / 4), (unsigned)G);
        if (d == 64)
          w_accumulate_sorted_kernel<T, 4><<<sgrid, 256, 0, st>>>(aa);
        else if (d == 128)
          w_accumulate_sorted_kernel<T, 8><<<sgrid, 256, 0, st>>>(aa);
        else
          w_accumulate_sorted_kernel<T, 16><<<sgrid, 256, 0, st>>>(aa);
      } else if (e4) {
        w_accumulate_kernel<T, 4><<<agrid, W_THREADS, A.lds, st>>>(aa);
      } else {
        w_accumulate_kernel<T, 2><<<agrid, W_THREADS, A.lds, st>>>(aa);
      }
    }
    if ((e2 = launch_ok())) return e2;
    {
      TimedLaunch tl(GSRQ_KERNEL_FINALIZE, st);
      if (e4)
        w_finalize_kernel<4><<<fgrid, 256, 0, st>>>(fa);
      else
        w_finalize_kernel<2><<<fgrid, 256, 0, st>>>(fa);
    }
    return launch_ok();
  };

  if (!(flags & GSRQ_RESUME)) {
    if (hipMemcpyAsync(seeds, seed_rows, (size_t)G * K * sizeof(int32_t), hipMemcpyHostToDevice,
                       st) != hipSuccess)
      return GSRQ_E_HIP;
    {
      TimedLaunch tl(GSRQ_KERNEL_TRANSPOSE, st);
      w_seed_kernel<T><<<dim3((K + 255) / 256, G), 256, 0, st>>>((const T*)X, ldx, d, K, seeds,
                                                                 shape, seednorm, kmeans, gain);
    }
    if ((e = launch_ok())) return e;
  }
  if (!(flags & GSRQ_RESUME) && kmeans) {
    // K-means starts from the seed centroids; there is no previous assignment
    fa.force_changed = 1;
  } else if (!(flags & GSRQ_RESUME)) {
    // equal-gain assignment, then eq. (8) gains for the seed shapes
    if ((e = w_build_frags(gain, shape, d, K, L.C, G, 0, true, nullptr, G, sig, frag, XD, st)))
      return e;
    sa.unit_gain = 1;
    sa.done = nullptr;
    if ((e = w_score_and_exact<T, W_TRAIN>(sa, L, GSRQ_KERNEL_ASSIGN, st))) return e;
    sa.unit_gain = 0;
    sa.done = done;
    fa.t = 0;
    if ((e = accumulate_finalize())) return e;
    fa.force_changed = 0;
  } else {
    fa.force_changed = (flags & GSRQ_ASSIGN_IN) ? 0 : 1;
  }
  sa.obj = obj_trace ? objp : nullptr;
  fa.obj = sa.obj;
  for (int t = 1; t <= T_; ++t) {
    if ((e = w_build_frags(gain, shape, d, K, L.C, G, 0, false, done, G, sig, frag, XD, st)))
      return e;
    if ((e = w_score_and_exact<T, W_TRAIN>(sa, L, GSRQ_KERNEL_ASSIGN, st))) return e;
    fa.t = t;
    if ((e = accumulate_finalize())) return e;
    fa.force_changed = 0;
  }
  if (R_next) {
    // next stage's input: the rows re-encoded with the final codebook
    if ((e = w_build_frags(gain, shape, d, K, L.C, G, 0, false, nullptr, G, sig, frag, XD, st)))
      return e;
    gsrq_shape s1 = *s;
    s1.M = 1;
    return w_encode_stage<T>(&s1, 0, X, ldx, gain, shape, sig, frag, XD, nullptr, 0, R_next,
                             st);
  }
  return GSRQ_OK;
}

}  // namespace

namespace gsrq_wide {

bool serves(const gsrq_shape* s) {
  // d / 8 a power of two: lane groups of d / 2 lanes share a row
  if (s->d % 8 != 0 || s->d > 8 * W_CMAX || !is_pow2(s->d / 8)) return false;
  return s->d > 8 || s->K > 256;
}

size_t train_workspace_bytes(const gsrq_shape* s, size_t x_elt) {
  if (x_elt == 0)   // either input type
    return std::max(w_train_ws(s, 2).total, w_train_ws(s, 4).total);
  return w_train_ws(s, x_elt).total;
}

size_t encode_workspace_bytes(const gsrq_shape* s) { return w_encode_ws(s).total; }

gsrq_status train_stage(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype, int64_t ldx,
                        const float* w, int32_t T, const int32_t* seed_rows, uint32_t flags,
                        float* gain, float* shape, float* R_next, uint16_t* assign_io,
                        int32_t* iters_run, double* obj_trace, void* workspace, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  if (x_dtype == GSRQ_F16)
    return w_train<_Float16>(s, X, ldx, w, T, seed_rows, flags, gain, shape, R_next, assign_io,
                             iters_run, obj_trace, workspace, st);
  return w_train<float>(s, X, ldx, w, T, seed_rows, flags, gain, shape, R_next, assign_io,
                        iters_run, obj_trace, workspace, st);
}

gsrq_status encode(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype, int64_t ldx,
                   const float* gain, const float* shape, uint32_t* codes, float* residual,
                   void* workspace, void* stream) {
  hipStream_t st = (hipStream_t)stream;
  const int G = s->D / s->d;
  const WEncWs W = w_encode_ws(s);
  char* base = (char*)workspace;
  u4* frag = (u4*)(base + W.frag);
  const WDefer XD = {(float*)(base + W.gmin), (int*)(base + W.xcount), (int*)(base + W.xrows),
                     (int*)(base + W.xchanged), (double*)(base + W.xobj),
                     W.hrows > W.hcount ? (int*)(base + W.hcount) : nullptr,
                     W.hrows > W.hcount ? (int*)(base + W.hrows) : nullptr,
                     W.hrows > W.hcount ? (unsigned long long*)(base + W.hbest) : nullptr,
                     W.hrows > W.hcount ? (float*)(base + W.hrr) : nullptr};
  int* sig = (int*)(base + W.sig);
  float* res[2] = {(float*)(base + W.res0), (float*)(base + W.res1)};
  const int words = (int)((s->M * (int64_t)G * log2i(s->K) + 31) / 32);
  gsrq_status e;
  if (codes && (e = fill_u32(codes, (size_t)s->N * words, 0u, st))) return e;
  const int C = w_cwidth(s->d);
  if (w_fused(s)) {
    // all stages' fragment tables, then one launch for every stage
    if ((e = w_build_frags(gain, shape, s->d, s->K, C, s->M * G, 0, false, nullptr, G, sig, frag,
                           XD, st)))
      return e;
    const WLayout L = w_score_layout(s, 4, false);
    WFusedArgs a;
    a.x = X; a.ldx = ldx; a.N = s->N; a.d = s->d; a.K = s->K; a.G = G; a.M = s->M;
    a.tiles = L.tiles; a.QF = L.QF; a.b = log2i(s->K); a.words = words;
    a.frag = frag; a.sig = sig; a.gain = gain; a.shape = shape; a.codes = codes;
    a.res_out = residual; a.res_vec = ((uintptr_t)residual % 16) == 0;
    a.svec = ((uintptr_t)shape % 16) == 0;
    const int64_t row_rounds = (s->N + W_ROWS - 1) / W_ROWS;
    a.nwg = (int)((row_rounds + W_FUSED_ROUNDS - 1) / W_FUSED_ROUNDS);
    a.map_xcd = L.map_xcd; a.lg = L.lg;
    const dim3 grid((unsigned)(G * a.nwg));
    TimedLaunch tl(GSRQ_KERNEL_ENCODE, st);
    if (x_dtype == GSRQ_F16) {
      if (C == 1) w_encode_fused_kernel<_Float16, 1><<<grid, W_THREADS, L.lds, st>>>(a);
      else w_encode_fused_kernel<_Float16, 2><<<grid, W_THREADS, L.lds, st>>>(a);
    } else {
      if (C == 1) w_encode_fused_kernel<float, 1><<<grid, W_THREADS, L.lds, st>>>(a);
      else w_encode_fused_kernel<float, 2><<<grid, W_THREADS, L.lds, st>>>(a);
    }
    return launch_ok();
  }
  if (w_fused_wide(s)) {
    // all stages' fragment tables, then one launch: one 32-row block per
    // wave, its residual in registers through every stage
    if ((e = w_build_frags(gain, shape, s->d, s->K, C, s->M * G, 0, false, nullptr, G, sig, frag,
                           XD, st)))
      return e;
    const WLayout L = w_score_layout(s, 4, false);
    WFusedArgs a;
    a.x = X; a.ldx = ldx; a.N = s->N; a.d = s->d; a.K = s->K; a.G = G; a.M = s->M;
    a.tiles = L.tiles; a.QF = L.QF; a.b = log2i(s->K); a.words = words;
    a.frag = frag; a.sig = sig; a.gain = gain; a.shape = shape; a.codes = codes;
    a.res_out = residual; a.res_vec = ((uintptr_t)residual % 16) == 0;
    a.svec = ((uintptr_t)shape % 16) == 0;
    a.nwg = (int)((s->N + W_FW_ROWS - 1) / W_FW_ROWS);
    a.map_xcd = L.map_xcd; a.lg = L.lg;
    const dim3 grid((unsigned)(G * a.nwg));
    const size_t lds = (size_t)L.tiles * w_frags(C) * 64 * sizeof(u4);
    auto go = [&](const void* fn, auto kern) -> gsrq_status {
      if (lds > 65536 &&
          hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
              hipSuccess)
        return GSRQ_E_HIP;
      kern<<<grid, W_FW_THREADS, lds, st>>>(a);
      return launch_ok();
    };
    TimedLaunch tl(GSRQ_KERNEL_ENCODE, st);
    if (x_dtype == GSRQ_F16)
      return C == 8 ? go((const void*)w_encode_fused_wide_kernel<_Float16, 8>,
                         w_encode_fused_wide_kernel<_Float16, 8>)
                    : go((const void*)w_encode_fused_wide_kernel<_Float16, 16>,
                         w_encode_fused_wide_kernel<_Float16, 16>);
    return C == 8 ? go((const void*)w_encode_fused_wide_kernel<float, 8>,
                       w_encode_fused_wide_kernel<float, 8>)
                  : go((const void*)w_encode_fused_wide_kernel<float, 16>,
                       w_encode_fused_wide_kernel<float, 16>);
  }
  for (int m = 0; m < s->M; ++m) {
    if ((e = w_build_frags(gain, shape, s->d, s->K, C, G, m * G, false, nullptr, G, sig, frag,
                           XD, st)))
      return e;
    float* out = (m + 1 < s->M) ? res[m & 1] : residual;
    if (m == 0 && x_dtype == GSRQ_F16)
      e = w_encode_stage<_Float16>(s, m, X, ldx, gain, shape, sig, frag, XD, codes, words, out,
                                   st);
    else if (m == 0)
      e = w_encode_stage<float>(s, m, X, ldx, gain, shape, sig, frag, XD, codes, words, out,
                                st);
    else
      e = w_encode_stage<float>(s, m, res[(m - 1) & 1], s->D, gain, shape, sig, frag, XD,
                                codes, words, out, st);
    if (e) return e;
  }
  return GSRQ_OK;
}

gsrq_status decode(const gsrq_shape* s, const uint32_t* codes, int32_t M_use, const float* gain,
                   const float* shape, void* Xhat, gsrq_dtype out_dtype, int64_t ldo,
                   void* stream) {
  hipStream_t st = (hipStream_t)stream;
  WDecArgs a;
  a.codes = codes; a.N = s->N; a.ldo = ldo; a.d = s->d; a.K = s->K; a.G = s->D / s->d;
  a.M_use = M_use; a.b = log2i(s->K);
  a.words = (int)((s->M * (int64_t)a.G * a.b + 31) / 32);
  a.gain = gain; a.shape = shape; a.out = Xhat;
  const size_t esz = out_dtype == GSRQ_F16 ? 2 : 4;
  // vector stores, and (gather kernel) vector codeword loads
  a.vec = ((uintptr_t)Xhat % 16 == 0) && ((ldo * esz) % 16 == 0) && (s->d % 8 == 0) &&
          ((uintptr_t)shape % 16 == 0);
  a.vshape = ((uintptr_t)shape % 16 == 0) && (s->d % 4 == 0);
  const int C = w_cwidth(s->d);
  TimedLaunch tl(GSRQ_KERNEL_DECODE, st);
  const bool half_tab = M_use == 1 && out_dtype == GSRQ_F16;
  const int64_t per_group = (int64_t)M_use * s->K * 8 * C * (half_tab ? 2 : 4);
  if (C <= 2 && per_group <= W_DEC_TABLE_BYTES) {
    int gpw = 1;
    while (gpw * 2 <= 64 && gpw * 2 * per_group <= W_DEC_TABLE_BYTES && gpw < a.G) gpw *= 2;
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
    a.tab_bytes = (int)(gpw * per_group);
    // code words fill the LDS the table leaves, up to W_DEC_CODE_PT per thread
    const int64_t code_words = std::min<int64_t>(
        (int64_t)W_DEC_CODE_PT * W_DEC_THREADS, ((int64_t)W_DEC_LDS_BYTES - a.tab_bytes) / 4);
    const int64_t max_rows = code_words / rs;
    if (max_rows < 1) return GSRQ_E_UNSUPPORTED;
    int64_t rchunks = (256 + a.gblocks - 1) / a.gblocks;
    if (rchunks * 256 > s->N) rchunks = (s->N + 255) / 256;
    if (rchunks < 1) rchunks = 1;
    a.rows_per_wg = (s->N + rchunks - 1) / rchunks;
    if (a.rows_per_wg > max_rows) a.rows_per_wg = max_rows;
    rchunks = (s->N + a.rows_per_wg - 1) / a.rows_per_wg;
    if (8 * a.gblocks * ((rchunks + 7) / 8) > INT32_MAX) return GSRQ_E_UNSUPPORTED;
    const int blocks = (int)(8 * a.gblocks * ((rchunks + 7) / 8));
    const size_t lds = (size_t)a.tab_bytes + (size_t)a.rows_per_wg * rs * sizeof(uint32_t);
    gsrq_status e = GSRQ_OK;
#define W_DEC(TO, TT, CC)                                                                    \
  do {                                                                                       \
    if (lds > 65536 && hipFuncSetAttribute((const void*)w_decode_lds_kernel<TO, TT, CC>,     \
                                           hipFuncAttributeMaxDynamicSharedMemorySize,       \
                                           (int)lds) != hipSuccess)                          \
      e = GSRQ_E_HIP;                                                                        \
    else                                                                                     \
      w_decode_lds_kernel<TO, TT, CC><<<blocks, W_DEC_THREADS, lds, st>>>(a);                \
  } while (0)
    if (C == 1) {
      if (half_tab) W_DEC(_Float16, _Float16, 1);
      else if (out_dtype == GSRQ_F16) W_DEC(_Float16, float, 1);
      else W_DEC(float, float, 1);
    } else {
      if (half_tab) W_DEC(_Float16, _Float16, 2);
      else if (out_dtype == GSRQ_F16) W_DEC(_Float16, float, 2);
      else W_DEC(float, float, 2);
    }
    if (e) return e;
#undef W_DEC
  } else {
    const int cg = w_groups(s->d);
    const int per_block = 256 / cg;
    const int64_t items = s->N * a.G;
    const int blocks = (int)((items + per_block - 1) / per_block);
    if (out_dtype == GSRQ_F16)
      w_decode_gather_kernel<_Float16><<<blocks, 256, 0, st>>>(a, cg);
    else
      w_decode_gather_kernel<float><<<blocks, 256, 0, st>>>(a, cg);
  }
  return launch_ok();
}

}  // namespace gsrq_wide
