// One decoding step of attention over a GSRQ-coded KV cache on AMD MI355X
// (gfx950): the codes are unpacked, the keys dequantised and rotated by
// RoPE, and softmax attention is taken, without an intermediate float16
// K/V tensor (arXiv 2607.01065, Appendix C, decoding latency analysis).
// Shapes: d = 8 subvectors, K = 256 codewords, one stage (the 1-bit cache),
// 128-element heads (16 subspaces per head), grouped-query attention with
// GQ = Hq / Hkv in {1, 2, 4}.
//
// One workgroup owns (sequence, key/value head, chunk of tokens); its four
// waves work through groups of U = 32 / GQ blocks of 32 tokens
// independently (flash-decoding within the chunk):
//  * Scores on the matrix cores.  The A operand of a v_mfma_f32_32x32x16_f16
//    holds 32 tokens' keys (each lane one 8-element codeword gathered from a
//    float16 table of the head's 16 codebooks in LDS, rotated in float32);
//    the B operand's 32 columns are the GQ query heads of the U blocks of a
//    group.  Both sides enter as float16 (rounded after their rotation in
//    float32), with float32 sums: the operand precision of float16
//    attention over a rotated float16 cache.
//    RoPE enters as a relative rotation: score(i) = (R_{pq - 32b} q) .
//    (R_t k_i) for token i = 32 b + t, so the rotation of a key depends only
//    on its row t in the block (fixed per lane) and that of the query on the
//    group (one sine/cosine per lane per group).
//  * Softmax per wave with a running reference maximum per query head
//    (raised by a margin, with the wave's sums rescaled, when a block's
//    scores exceed it).
//  * Values on the matrix cores: the weights leave the score accumulators
//    already in the A-operand layout of the value product (float16),
//    and the B operand gathers each token's float16 value codeword element
//    from a second LDS table, in the transposed layout the product needs,
//    through the block's value codes staged in LDS by subspace.
//  * The waves' partial results are merged at the end of the chunk, and a
//    second kernel merges the chunks of every (sequence, query head) with
//    their reference maxima (the split form of one softmax).
#include <algorithm>
#include <mutex>

#include "gsrq_common.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int AT_HD = 128;            // head dimension
constexpr int AT_SUB = 16;            // d = 8 subspaces per head
constexpr int AT_K = 256;             // codewords per codebook
constexpr int AT_WAVES = 8;            // two waves per SIMD share the tables
constexpr int AT_THREADS = AT_WAVES * 64;
constexpr int AT_BLK = 32;            // tokens per MFMA block
constexpr int AT_PART = AT_HD + 2;    // partial record: o[128], reference max, sum
constexpr int AT_TARGET_WG = 256;     // workgroups aimed for per launch (1 per CU)
constexpr float AT_HEADROOM = 8.f;    // log2 margin of a raised reference maximum
constexpr float AT_PSHIFT = 15.f;     // weights 2^(s - m + 15) <= 2^15: float16 range
constexpr int AT_TAB = AT_SUB * AT_K * 8;   // float16 elements of one codeword table
constexpr int AT_RED = 8 + 4 * AT_HD;       // floats per wave in the final merge
constexpr int AT_TRIG_BLOCKS = 16;          // tables kernel: 2 x 32 x 64 angles, one per thread

template <int GQ> struct AtCfg {
  static constexpr int U = 32 / GQ;                         // blocks per wave group
  static constexpr int ROUND = AT_WAVES * U * AT_BLK;       // tokens of one group per wave
  // LDS layout in bytes
  static constexpr int KTAB = 0;                            // f16 [16][256][8] keys
  static constexpr int VTAB = KTAB + AT_TAB * 2;            // f16 [16][256][8] values
  static constexpr int QT = VTAB + AT_TAB * 2;              // f32 [32][128] queries
  // per wave: the value tile of a quarter head [32 k positions][32 dims]
  // f16; the group's angle table (float2 [64]) shares it at the start of a
  // group.  The final merge (f32 [AT_WAVES][AT_RED]) reuses the key table.
  static constexpr int TILE = QT + 32 * AT_HD * 4;
  static constexpr int TILE_BYTES = 32 * AT_BLK * 2;
  static constexpr int BYTES = TILE + AT_WAVES * TILE_BYTES;
};
static_assert(64 * 8 <= 32 * AT_BLK * 2, "angle table fits the tile");
static_assert(AT_WAVES * AT_RED * 4 <= AT_TAB * 2, "merge records fit the key table");
static_assert(AtCfg<4>::BYTES <= 160 * 1024, "LDS budget");

struct AttnArgs {
  const uint32_t* kc;       // [B][cap][W] key codes
  const uint32_t* vc;       // [B][cap][W] value codes
  const int32_t* seq_len;   // [B]
  const void* q;            // [B][Hq][128]
  int q_f16;
  const float2* t1;         // [32][64] cos/sin of t theta_j
  const float2* t2;         // [32][64] cos/sin of 32 u theta_j
  const double* th;         // [64] theta_j / 2 pi
  const u4* tabk;           // [Hkv][16][256][8] f16 key codewords (16-byte rows)
  const u4* tabv;           // same for values
  float* part;              // [B][Hkv][nch][GQ][AT_PART]
  int cap, W, Hkv, nch, rpc;
  int xmap;                 // XCD-grouped block order (B * nch a multiple of 8)
  float qscale;             // softmax scale * log2(e)
};

// Tag of the tables in a workspace: written by the tables kernel, compared
// by the merge kernel with what the call expects, so that a call that skips
// the table build (GSRQ_ATTN_TABLES_READY) on a workspace that holds no
// tables, or tables of other codebook arrays, head count or RoPE base,
// returns NaN outputs instead of plausible wrong ones.
constexpr uint32_t AT_TAG_MAGIC = 0x47535251u;
constexpr int AT_TAG_WORDS = 16;
struct AttnTag {
  uint32_t w[AT_TAG_WORDS];
};

// Per call: cos/sin tables of the rotations a block needs (float64
// arithmetic; the first AT_TRIG_BLOCKS blocks), and the float16 decode
// fp16(fp32(g * s)) of every key and value codeword (the other blocks, one
// codeword per thread).
__global__ void __launch_bounds__(256) attn_tables_kernel(double base, float2* __restrict__ t1,
                                                          float2* __restrict__ t2,
                                                          double* __restrict__ th,
                                                          const float* __restrict__ kg,
                                                          const float* __restrict__ ks,
                                                          const float* __restrict__ vg,
                                                          const float* __restrict__ vs, int ncw,
                                                          u4* __restrict__ tabk,
                                                          u4* __restrict__ tabv, AttnTag tag,
                                                          uint32_t* __restrict__ tagp) {
  if (blockIdx.x == 0 && threadIdx.x < AT_TAG_WORDS) tagp[threadIdx.x] = tag.w[threadIdx.x];
  if (blockIdx.x < AT_TRIG_BLOCKS) {
    // one angle per thread: the entries of t1 (n = t), then those of t2
    // (n = 32 t), reduced to one turn in float64 before the sine and cosine
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int e = i & 2047, t = e >> 6, j = e & 63;
    const double theta = pow(base, -2.0 * j / AT_HD);
    const double n = i < 2048 ? (double)t : 32.0 * t;
    double rev = n * (theta / (2.0 * M_PI));
    rev -= floor(rev);
    double s, c;
    sincos(rev * (2.0 * M_PI), &s, &c);
    (i < 2048 ? t1 : t2)[e] = make_float2((float)c, (float)s);
    if (i < 64) th[j] = theta / (2.0 * M_PI);
    return;
  }
  const int cw = (blockIdx.x - AT_TRIG_BLOCKS) * 256 + threadIdx.x;
  if (cw >= 2 * ncw) return;
  const bool val = cw >= ncw;
  const int k = val ? cw - ncw : cw;
  const float g = (val ? vg : kg)[k];
  const f4* sp = (const f4*)((val ? vs : ks) + (size_t)k * 8);
  const f4 a = sp[0], b = sp[1];
  _Float16 h[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    h[e] = (_Float16)(g * a[e]);
    h[4 + e] = (_Float16)(g * b[e]);
  }
  (val ? tabv : tabk)[k] = pack_h8(h);
}

// Order a wave's own LDS accesses around this point: the tile is read and
// written through different types, so the compiler must not move accesses
// across it (the LDS itself serves one wave's accesses in order).
__device__ __forceinline__ void wave_lds_order() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// Offset in float16 elements of 16-byte chunk c (dims 8 c .. 8 c + 7) of row
// r in a wave's value tile [32 k positions][32 dims] (64-byte rows, four to
// 256 bytes of banks).  Chunks are permuted per row by c ^ ((r / 4) % 4), so
// that the 16-byte writes of 16 consecutive rows (one chunk each) and the
// 8-byte transposing reads of 4 consecutive rows (4 chunks each) hit
// distinct banks.
__device__ __forceinline__ int tile_off(int r, int c) {
  return r * 32 + ((c ^ ((r >> 2) & 3)) << 3);
}

// ds_read_b64_tr_b16: lane l of each group of 16 lanes receives element
// l % 4 of the 8-byte chunks addressed by lanes 4 r + l / 4 of its group,
// r = 0 .. 3 (the MFMA operand layout of a row-major 16-bit matrix).
__device__ __forceinline__ uint2 tr_load_b64(const _Float16* p) {
  typedef __attribute__((__vector_size__(4 * sizeof(__fp16)))) __fp16 fp16x4;
  typedef __attribute__((address_space(3))) fp16x4* lds_fp16x4;
  const fp16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4f16((lds_fp16x4)(p));
  return __builtin_bit_cast(uint2, v);
}

template <int GQ>
__global__ void __launch_bounds__(AT_THREADS, 1) attn_chunk_kernel(AttnArgs a) {
  using C = AtCfg<GQ>;
  constexpr int U = C::U;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  _Float16* ktab = (_Float16*)(lds + C::KTAB);
  _Float16* vtab = (_Float16*)(lds + C::VTAB);

  // Blocks go round-robin to the 8 XCDs.  With xmap, the Hkv workgroups of
  // one (sequence, chunk), which read the same 128-byte code rows (each its
  // head's 16 bytes), are numbered onto one XCD, so its L2 serves the rows
  // once instead of each XCD fetching them from HBM.
  int chunk, hk, b;
  {
    const int id = blockIdx.x;
    if (a.xmap) {
      const int x = id & 7, slot = id >> 3;
      const int gid = (slot / a.Hkv) * 8 + x;
      hk = slot % a.Hkv;
      b = gid / a.nch;
      chunk = gid % a.nch;
    } else {
      chunk = id % a.nch;
      hk = (id / a.nch) % a.Hkv;
      b = id / (a.nch * a.Hkv);
    }
  }
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int tl = lane & 31, hh = lane >> 5;
  const int ul = tl / GQ, hl = tl % GQ;      // B-operand column: block variant, query head
  _Float16* tile = (_Float16*)(lds + C::TILE + w * C::TILE_BYTES);
  float2* ang = (float2*)tile;
  // k position of the lane's token row in the value product: token t sits
  // where the score accumulators hold it, 16 (t / 16) + 8 ((t / 4) % 2) +
  // 4 ((t / 8) % 2) + t % 4 (bits 2 and 3 of t exchanged)
  const int kpos = (tl & ~12) | ((tl & 4) << 1) | ((tl & 8) >> 1);
  const int len = min(max(a.seq_len[b], 0), a.cap);
  const int tok0 = chunk * a.rpc * C::ROUND;
  float* outp = a.part + (((size_t)b * a.Hkv + hk) * a.nch + chunk) * GQ * AT_PART;
  if (tok0 >= len) {
    if (tid < GQ) {
      outp[tid * AT_PART + AT_HD] = -INFINITY;
      outp[tid * AT_PART + AT_HD + 1] = 0.f;
    }
    return;
  }
  const int tend = min(len, tok0 + a.rpc * C::ROUND);
  const int Hq = a.Hkv * GQ;
  const int g0 = hk * AT_SUB;
  const size_t seq_row0 = (size_t)b * a.cap;

  // this head's float16 codeword tables (16 u4 of keys and 16 of values
  // per thread, every load issued before the first store)
  {
    const u4* sk = a.tabk + (size_t)hk * AT_SUB * AT_K;
    const u4* sv = a.tabv + (size_t)hk * AT_SUB * AT_K;
    constexpr int PER = AT_SUB * AT_K / AT_THREADS;
    u4 rk[PER], rv[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      rk[m] = sk[m * AT_THREADS + tid];
      rv[m] = sv[m * AT_THREADS + tid];
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      ((u4*)ktab)[m * AT_THREADS + tid] = rk[m];
      ((u4*)vtab)[m * AT_THREADS + tid] = rv[m];
    }
  }
  // query of every B-operand column j = (u, h), turned by R_{-32u} and
  // scaled by the softmax scale times log2(e) (scores come out in log2
  // units): qt[j][jd], qt[j][jd + 64] for the pairs jd < 64
  float* qt = (float*)(lds + C::QT);
  {
    constexpr int PER = 32 * 64 / AT_THREADS;
    float x[PER], y[PER];
    float2 cs[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int it = m * AT_THREADS + tid, j = it >> 6, jd = it & 63;
      const size_t qo = ((size_t)b * Hq + hk * GQ + j % GQ) * AT_HD + jd;
      if (a.q_f16) {
        x[m] = (float)((const _Float16*)a.q)[qo];
        y[m] = (float)((const _Float16*)a.q)[qo + 64];
      } else {
        x[m] = ((const float*)a.q)[qo];
        y[m] = ((const float*)a.q)[qo + 64];
      }
      cs[m] = a.t2[(j / GQ) * 64 + jd];
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int it = m * AT_THREADS + tid, j = it >> 6, jd = it & 63;
      qt[j * AT_HD + jd] = (x[m] * cs[m].x + y[m] * cs[m].y) * a.qscale;   // R_{-32u}
      qt[j * AT_HD + jd + 64] = (y[m] * cs[m].x - x[m] * cs[m].y) * a.qscale;
    }
  }

  // lane constant: R_t for the lane's token row as float16 pairs; element
  // m < 32 of a lane is head element jd = 32 hh + m, paired with jd + 64;
  // cp[m / 2] holds the cosines of elements m, m + 1 (m even), sp the sines
  h2 cp[16], sp[16];
  {
    const float4* t1 = (const float4*)(a.t1 + tl * 64 + 32 * hh);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const float4 v = t1[m];
      cp[m] = (h2){(_Float16)v.x, (_Float16)v.z};
      sp[m] = (h2){(_Float16)v.y, (_Float16)v.w};
    }
  }
  const double thl = a.th[lane];
  __syncthreads();

  float mw[GQ];                  // running reference maximum per head (log2 units)
#pragma unroll
  for (int h = 0; h < GQ; ++h) mw[h] = -INFINITY;
  float lsum = 0.f;              // softmax sum of this lane's column (scaled by 2^PSHIFT)
  f16v o[4] = {};                // value sums: rows = columns (variant, head), cols = dims
  const int ngroups = (tend - tok0 + 32 * U - 1) / (32 * U);
  for (int gi = w; gi < ngroups; gi += AT_WAVES) {
    const int gb0 = (tok0 >> 5) + gi * U;
    {
      const int n = (len - 1) - 32 * gb0;           // query-side angle in positions, >= 0
      double rev = (double)n * thl;
      rev -= floor(rev);
      float s, c;
      sincosf((float)(rev * (2.0 * M_PI)), &s, &c);
      ang[lane] = make_float2(c, s);
    }
    wave_lds_order();
    // query of the lane's column turned by R_{pq - 32 gb0} R_{-32u} (its
    // block's relative rotation), rounded to float16
    u4 bq[8];
    {
      const float4* qxp = (const float4*)(qt + tl * AT_HD + 32 * hh);
      const float4* qyp = (const float4*)(qt + tl * AT_HD + 64 + 32 * hh);
      const float4* ap = (const float4*)(ang + 32 * hh);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        _Float16 xh[8], yh[8];
#pragma unroll
        for (int m2 = 0; m2 < 2; ++m2) {
          const float4 qx4 = qxp[2 * i + m2], qy4 = qyp[2 * i + m2];
          const float4 va = ap[4 * i + 2 * m2], vb = ap[4 * i + 2 * m2 + 1];
          const float qxv[4] = {qx4.x, qx4.y, qx4.z, qx4.w};
          const float qyv[4] = {qy4.x, qy4.y, qy4.z, qy4.w};
          const float cv[4] = {va.x, va.z, vb.x, vb.z};
          const float sv[4] = {va.y, va.w, vb.y, vb.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int e = 4 * m2 + r;
            xh[e] = (_Float16)(qxv[r] * cv[r] - qyv[r] * sv[r]);
            yh[e] = (_Float16)(qxv[r] * sv[r] + qyv[r] * cv[r]);
          }
        }
        bq[i] = pack_h8(xh);
        bq[i + 4] = pack_h8(yh);
      }
    }
    wave_lds_order();                               // angle table reads before tile writes
    const int nblk = min(U, (len - 32 * gb0 + 31) >> 5);
    // codes of the next block are loaded while this one is scored; rows
    // past the sequence end read the last row instead (their weights are
    // zero), so that every load is unconditional and the wait for the
    // current block's codes leaves the next block's loads in flight
    const u4* kcp = (const u4*)(a.kc + seq_row0 * a.W + 4 * hk);
    const u4* vcp = (const u4*)(a.vc + seq_row0 * a.W + 4 * hk);
    const int wq = a.W / 4;                          // u4 per row
    u4 kcn, vcn;
    {
      const int row = min(32 * gb0 + tl, len - 1);
      kcn = kcp[(size_t)row * wq];
      vcn = vcp[(size_t)row * wq];
    }
    for (int u = 0; u < nblk; ++u) {
      const u4 kcw = kcn, vcw = vcn;
      {
        const int row = min(32 * (gb0 + min(u + 1, nblk - 1)) + tl, len - 1);
        kcn = kcp[(size_t)row * wq];
        vcn = vcp[(size_t)row * wq];
      }
      const uint32_t kw0 = hh ? kcw[1] : kcw[0], kw1 = hh ? kcw[3] : kcw[2];

      // ---- scores: pair (i, i + 4) of k-steps holds elements jd and jd + 64;
      // R_t in packed float16 arithmetic (x' = x c - y s, y' = x s + y c)
      f16v acc = {};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int cx = (kw0 >> (8 * i)) & 255, cy = (kw1 >> (8 * i)) & 255;
        const u4 x = *(const u4*)(ktab + ((4 * hh + i) * AT_K + cx) * 8);
        const u4 y = *(const u4*)(ktab + ((8 + 4 * hh + i) * AT_K + cy) * 8);
        h2 xr[4], yr[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const uint32_t xw = x[p], yw = y[p];    // scalar copies before the bit casts
          const h2 xp = __builtin_bit_cast(h2, xw), yp = __builtin_bit_cast(h2, yw);
          const h2 c = cp[4 * i + p], sn = sp[4 * i + p];
          xr[p] = __builtin_elementwise_fma(xp, c, -(yp * sn));
          yr[p] = __builtin_elementwise_fma(xp, sn, yp * c);
        }
        const h8 kx = __builtin_shufflevector(__builtin_shufflevector(xr[0], xr[1], 0, 1, 2, 3),
                                              __builtin_shufflevector(xr[2], xr[3], 0, 1, 2, 3),
                                              0, 1, 2, 3, 4, 5, 6, 7);
        const h8 ky = __builtin_shufflevector(__builtin_shufflevector(yr[0], yr[1], 0, 1, 2, 3),
                                              __builtin_shufflevector(yr[2], yr[3], 0, 1, 2, 3),
                                              0, 1, 2, 3, 4, 5, 6, 7);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kx, as_h8(bq[i]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ky, as_h8(bq[i + 4]), acc, 0, 0, 0);
      }

      // ---- softmax weights of this block (only the columns of variant u)
      // register v holds token row t = 8 (v / 4) + 4 hh + v % 4
      const int rowb = 32 * (gb0 + u);
      // (a lane's maximum is read only for columns of variant u; rows past
      // the sequence end, only in its last block, are masked out)
      float sc[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[v] = acc[v];
      if (rowb + 32 > len) {                         // uniform
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int t = 8 * (v >> 2) + 4 * hh + (v & 3);
          if (rowb + t >= len) sc[v] = -INFINITY;
        }
      }
      float ml = sc[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) ml = fmaxf(ml, sc[v]);
      ml = fmaxf(ml, __shfl_xor(ml, 32));
      // raise the references of the heads whose block maximum exceeds
      // them, rescaling this wave's sums once for all heads (rare)
      float mbh[GQ];
      bool raise = false;
#pragma unroll
      for (int h = 0; h < GQ; ++h) {
        mbh[h] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ml), u * GQ + h));
        raise |= mbh[h] > mw[h];
      }
      if (raise) {                                   // uniform
        float fac[GQ];
#pragma unroll
        for (int h = 0; h < GQ; ++h) {
          const float nref = mbh[h] > mw[h] ? mbh[h] + AT_HEADROOM : mw[h];
          fac[h] = exp2f(mw[h] - nref);              // 1 if kept, 0 from -inf
          mw[h] = nref;
        }
        float fl = fac[0];
#pragma unroll
        for (int h = 1; h < GQ; ++h) fl = hl == h ? fac[h] : fl;
        lsum *= fl;
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[c][v] *= fac[(v & 3) % GQ];
      }
      // weights 2^(s - m + PSHIFT) of the lane's column; columns of other
      // variants get 2^-inf = 0
      float mine = mw[0];
#pragma unroll
      for (int h = 1; h < GQ; ++h) mine = hl == h ? mw[h] : mine;
      mine = ul == u ? mine - AT_PSHIFT : INFINITY;
      u4 ph[2];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        _Float16 xh[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sv = sc[8 * s2 + e];
          const float pv = __builtin_amdgcn_exp2f(sv - mine);
          lsum += pv;
          xh[e] = (_Float16)pv;
        }
        ph[s2] = pack_h8(xh);
      }

      // ---- value sums o[c] += P . V over four quarters of the head (tile
      // c = 2 hp + cc: dims 32 c .. 32 c + 31, subspaces 4 c .. 4 c + 3):
      // every lane writes two of its token's value codewords of the quarter
      // into row kpos of the wave's tile ([kpos][32 dims], swizzled 16-byte
      // chunks), then reads its B operands (8 k positions of one dim) with
      // transposing loads
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t vw = vcw[c];                  // codes of subspaces 4 c .. 4 c + 3
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int code = (vw >> (8 * (2 * hh + i))) & 255;
          const u4 v8 = *(const u4*)(vtab + ((4 * c + 2 * hh + i) * AT_K + code) * 8);
          *(u4*)(tile + tile_off(kpos, 2 * hh + i)) = v8;     // dims 16 hh + 8 i ..
        }
        wave_lds_order();
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          // lane j of a 16-lane group supplies k position 16 s2 + 8 hh + 4 ld
          // + (j % 16) / 4, dims 16 ((j / 16) % 2) + 4 (j % 4) .. + 3; lane l
          // then receives dim l % 32 of the quarter at the four k positions
          // 16 s2 + 8 hh + 4 ld + 0..3
          const int cq = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
          const int r0 = 16 * s2 + 8 * hh + ((lane >> 2) & 3);
          const uint2 t0 = tr_load_b64(tile + tile_off(r0, cq) + 4 * (lane & 1));
          const uint2 t1 = tr_load_b64(tile + tile_off(r0 + 4, cq) + 4 * (lane & 1));
          const u4 vb = {t0.x, t0.y, t1.x, t1.y};
          o[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(ph[s2]), as_h8(vb), o[c], 0, 0, 0);
        }
        wave_lds_order();
      }
    }
  }

  // ---- merge the waves: per head the reference, the sum and o (records
  // in the key table, once every wave is done with it)
  __syncthreads();
  float* rw = (float*)(lds + C::KTAB) + w * AT_RED;
  {
    float l = lsum;
#pragma unroll
    for (int off = GQ; off < 64; off <<= 1) l += __shfl_xor(l, off);
    if (lane < GQ) {
      rw[lane] = mw[0];
#pragma unroll
      for (int h = 1; h < GQ; ++h)
        if (lane == h) rw[lane] = mw[h];
      rw[4 + lane] = l;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int h = 0; h < GQ; ++h) {
        float v = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if ((r & 3) % GQ == h) v += o[c][r];
        v += __shfl_xor(v, 32);
        if (hh == 0) rw[8 + h * AT_HD + 32 * c + tl] = v;
      }
  }
  __syncthreads();
  const float* red = (const float*)(lds + C::KTAB);
  constexpr int RS = AT_RED;                         // floats between waves' records
  for (int i = tid; i < GQ * AT_HD; i += AT_THREADS) {
    const int h = i / AT_HD, n = i % AT_HD;
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < AT_WAVES; ++v)
      if (red[v * RS + 4 + h] > 0.f) M = fmaxf(M, red[v * RS + h]);
    double num = 0.0, den = 0.0;
#pragma unroll
    for (int v = 0; v < AT_WAVES; ++v) {
      const float* r = red + v * RS;
      if (!(r[4 + h] > 0.f)) continue;
      const double f = exp2((double)r[h] - (double)M);
      num += f * (double)r[8 + h * AT_HD + n];
      den += f * (double)r[4 + h];
    }
    outp[h * AT_PART + n] = (float)num;
    if (n == 0) {
      outp[h * AT_PART + AT_HD] = M - AT_PSHIFT;
      outp[h * AT_PART + AT_HD + 1] = (float)den;
    }
  }
}

// Merge the chunks of every (sequence, query head): o = sum_c 2^(m_c - M) o_c
// / sum_c 2^(m_c - M) l_c over the chunks holding tokens.  Both passes are
// branch-free and unrolled, so that the loads of several chunks are in
// flight together.
__global__ void __launch_bounds__(AT_HD) attn_merge_kernel(const float* __restrict__ part, int Hq,
                                                          int Hkv, int nch,
                                                          float* __restrict__ out, AttnTag tag,
                                                          const uint32_t* __restrict__ tagp) {
  const int bq = blockIdx.x, b = bq / Hq, hq = bq % Hq;
  bool tag_ok = true;
#pragma unroll
  for (int i = 0; i < AT_TAG_WORDS; ++i) tag_ok &= tagp[i] == tag.w[i];
  if (!tag_ok) {
    out[(size_t)bq * AT_HD + threadIdx.x] = __builtin_nanf("");
    return;
  }
  const int GQ = Hq / Hkv, hk = hq / GQ, h = hq % GQ, n = threadIdx.x;
  const float* p = part + (((size_t)b * Hkv + hk) * nch * GQ + h) * AT_PART;
  const size_t cs = (size_t)GQ * AT_PART;
  float M = -INFINITY;
#pragma unroll 8
  for (int c = 0; c < nch; ++c) {
    const float m = p[c * cs + AT_HD], l = p[c * cs + AT_HD + 1];
    M = l > 0.f ? fmaxf(M, m) : M;
  }
  double num = 0.0, den = 0.0;
#pragma unroll 8
  for (int c = 0; c < nch; ++c) {
    const float m = p[c * cs + AT_HD], l = p[c * cs + AT_HD + 1], o = p[c * cs + n];
    // a chunk without tokens writes only its (m, l) record: its o slots hold
    // whatever the workspace held, which must not reach the sums (0 * NaN)
    const bool has = l > 0.f;
    const double f = has ? exp2((double)m - (double)M) : 0.0;
    num += has ? f * (double)o : 0.0;
    den += has ? f * (double)l : 0.0;
  }
  out[(size_t)bq * AT_HD + n] = den > 0.0 ? (float)(num / den) : 0.f;
}

struct AttnPlan {
  int GQ, rpc, nch;
  size_t off_tag, off_t1, off_t2, off_th, off_tk, off_tv, off_part, bytes;
};

int at_round(int GQ) { return AT_WAVES * (32 / GQ) * AT_BLK; }

gsrq_status attn_plan(const gsrq_attn_shape* a, AttnPlan& p) {
  if (!a) return GSRQ_E_ARG;
  if (a->B < 1 || a->cap < 1 || a->Hkv < 1 || a->Hq < 1 || a->head_dim < 1) return GSRQ_E_ARG;
  if (a->Hq % a->Hkv) return GSRQ_E_ARG;
  if (!(a->rope_base > 0.f) || !(a->rope_base < INFINITY)) return GSRQ_E_ARG;
  if (!(a->scale > 0.f) || !(a->scale < INFINITY)) return GSRQ_E_ARG;
  if (a->flags & ~(uint32_t)GSRQ_ATTN_TABLES_READY) return GSRQ_E_ARG;
  if (a->B > 65535 || a->Hkv > 65535) return GSRQ_E_ARG;
  p.GQ = a->Hq / a->Hkv;
  if (a->head_dim != AT_HD) return GSRQ_E_UNSUPPORTED;
  if (p.GQ != 1 && p.GQ != 2 && p.GQ != 4) return GSRQ_E_UNSUPPORTED;
  const int64_t round = at_round(p.GQ);
  const int64_t rounds = ((int64_t)a->cap + round - 1) / round;
  const int64_t pairs = (int64_t)a->B * a->Hkv;
  int64_t r = (rounds * pairs + AT_TARGET_WG - 1) / AT_TARGET_WG;
  r = std::max<int64_t>(1, std::min<int64_t>(r, rounds));
  p.rpc = (int)r;
  p.nch = (int)((rounds + r - 1) / r);
  if ((int64_t)p.nch * a->Hkv * a->B > INT32_MAX) return GSRQ_E_UNSUPPORTED;
  p.off_tag = 0;
  p.off_t1 = 256;
  p.off_t2 = p.off_t1 + align256(32 * 64 * sizeof(float2));
  p.off_th = p.off_t2 + align256(32 * 64 * sizeof(float2));
  p.off_tk = p.off_th + align256(64 * sizeof(double));
  p.off_tv = p.off_tk + align256((size_t)a->Hkv * AT_SUB * AT_K * 16);
  p.off_part = p.off_tv + align256((size_t)a->Hkv * AT_SUB * AT_K * 16);
  p.bytes = p.off_part + align256((size_t)pairs * p.nch * p.GQ * AT_PART * sizeof(float));
  return GSRQ_OK;
}

template <int GQ> gsrq_status attn_launch(const AttnArgs& args, int B, int Hkv, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute((const void*)attn_chunk_kernel<GQ>,
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            AtCfg<GQ>::BYTES) != hipSuccess)
      return GSRQ_E_HIP;
    attr_set = true;
  }
  TimedLaunch tm(GSRQ_KERNEL_ATTENTION, st);
  const int blocks = args.nch * Hkv * B;
  attn_chunk_kernel<GQ><<<blocks, AT_THREADS, AtCfg<GQ>::BYTES, st>>>(args);
  return launch_ok();
}

// ------------------------------------------------------------------------
// Residual-coded caches at the paper's sub-1-bit rates: one subspace per head
// (d = head_dim = 128), K = 256, M stages (0.75 bit at M = 12, 1 bit at 16,
// 2 bit at 32).  A head's key codebooks (M x 256 x 128 float16, 768 KiB at
// M = 12) do not fit LDS, so the chunk kernel scores in passes over stage
// pairs: per pass the workgroup copies the pair's float16 key table
// (128 KiB) into LDS, and every wave adds, for all the blocks it owns, the
// pair's share of each score (a key is the sum of its stages' codewords, so
// a score is the sum of the stages' shares) into score accumulators it keeps
// across passes.  Per 32-token block the A operand holds the block's partial
// keys (two gathered codeword pieces summed in float16, turned by the lane's
// R_t as in the 1-bit kernel); the B operand is the group's query columns
// with every column of another block zeroed, so one accumulator collects a
// whole group of U blocks, each column its own block's scores.  After the
// last pass the softmax takes one reference maximum per head for the whole
// workgroup and float32 weights, and the value side needs no gathers: with
// v_i = sum_m c_m[code_m(i)], sum_i p_i v_i = sum_m sum_k W_m[k] c_m[k] for
// W_m[k] = sum of the weights of the tokens whose stage-m code is k, so the
// workgroup adds each weight into its M per-stage bins (LDS float atomics)
// and writes the bins; the merge kernel sums the chunks' bins and contracts
// them with the value codewords fl(g s).
constexpr int AQ_MAXM = 16;               // stages supported (0.75 and 1 bit)
constexpr int AQ_NG = 2;                  // groups of U blocks per wave
constexpr int AQ_TAB_U4 = 2 * AT_K * 16;  // u4 of a stage-pair table (128 KiB)

constexpr int AQ_CHUNK = 4096;           // tokens per workgroup
template <int GQ> struct AqCfg {
  static constexpr int U = 32 / GQ;
  static constexpr int CHUNK = AQ_CHUNK;                        // AQ_CHUNK / (32 U) groups
  static constexpr int KTAB = 0;                                // u4 [2][256][16], swizzled
  static constexpr int QT = KTAB + AQ_TAB_U4 * 16;              // f32 [32][128]
  static constexpr int ANG = QT + 32 * AT_HD * 4;               // float2 [AT_WAVES][64]
  static constexpr int RED = ANG + AT_WAVES * 64 * 8;           // f32 [AT_WAVES][2][GQ]
  static constexpr int KC = RED + AT_WAVES * 2 * 4 * 4;         // u8 [CHUNK][2]: the pass's codes
  static constexpr int BYTES = KC + CHUNK * 2;
  // after the last pass the key table's space holds the bins of a group of
  // stages and the chunk's value codes
  static constexpr int BINS = 0;                                // u64 [32 / GQ][256][GQ]
  static constexpr int VC = 32 * AT_K * 8;                      // u8 [CHUNK][16]
};
static_assert(AqCfg<4>::BYTES <= 160 * 1024, "LDS budget");
static_assert(32 * AT_K * 8 + AQ_CHUNK * AQ_MAXM <= AQ_TAB_U4 * 16,
              "bins and value codes fit the key table");
static_assert(AQ_CHUNK % (32 * 32) == 0 && AQ_CHUNK / (32 * 8) <= AQ_NG * AT_WAVES,
              "every group of a chunk has a wave");

struct AqArgs {
  const uint8_t* kc;        // [B][cap][4 W] key code bytes: stage m, head h at m Hkv + h
  const uint8_t* vc;        // same for values
  const int32_t* seq_len;   // [B]
  const void* q;            // [B][Hq][128]
  int q_f16;
  const float2* t1;         // [32][64] cos/sin of t theta_j
  const float2* t2;         // [32][64] cos/sin of 32 u theta_j
  const double* th;         // [64] theta_j / 2 pi
  const u4* tabk;           // [Hkv][M][256][16] f16 key codewords, 16 chunks of 8
  float* part;              // [B][Hkv][nch][GQ][M 256 + 2]
  int cap, rowb, Hkv, M, nch;  // rowb: code bytes per token row (4 W)
  int xmap;
  float qscale;
};

// Float16 key table of a residual-coded head: fp16(fp32(g s)) of every
// codeword, chunk c = elements 8c .. 8c + 7, one chunk per thread.
__global__ void __launch_bounds__(256) attn_rq_keytab_kernel(const float* __restrict__ kg,
                                                             const float* __restrict__ ks,
                                                             int Hkv, int M,
                                                             u4* __restrict__ tabk) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;   // ((h M + m) 256 + k) 16 + c
  if (e >= (int64_t)Hkv * M * AT_K * 16) return;
  const int c = (int)(e & 15);
  const int64_t hmk = e >> 4;
  const int k = (int)(hmk % AT_K);
  const int64_t hm = hmk / AT_K;
  const int m = (int)(hm % M), h = (int)(hm / M);
  const size_t cw = ((size_t)m * Hkv + h) * AT_K + k;          // codebook order [M][G][K]
  const float g = kg[cw];
  const f4* sp = (const f4*)(ks + cw * AT_HD + 8 * c);
  const f4 a = sp[0], b = sp[1];
  _Float16 v[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[j] = (_Float16)(g * a[j]);
    v[4 + j] = (_Float16)(g * b[j]);
  }
  tabk[e] = pack_h8(v);
}

// LDS layout of a stage-pair key table: chunk c of codeword k of stage sl
// sits in u4 slot ((sl K + k) << 4) | (c ^ (k & 15)), so that lanes gathering
// the same chunk of random codewords spread over the banks.  A lane of half
// hh reads chunks 4 hh + i and 8 + 4 hh + i (i < 4); with
// base = ((sl K + k) << 8) | (((4 hh) ^ (k & 15)) << 4) their byte offsets are
// base ^ (i << 4) and base ^ ((8 | i) << 4): one XOR per gather.
__device__ __forceinline__ uint32_t aq_base(int sl, int k, int hh) {
  return ((uint32_t)(sl * AT_K + k) << 8) | ((uint32_t)((4 * hh) ^ (k & 15)) << 4);
}

template <int GQ>
__global__ void __launch_bounds__(AT_THREADS, 1) attn_rq_chunk_kernel(AqArgs a) {
  using C = AqCfg<GQ>;
  constexpr int U = C::U;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  u4* ktab = (u4*)(lds + C::KTAB);
  unsigned long long* bins = (unsigned long long*)(lds + C::BINS);
  float* qt = (float*)(lds + C::QT);
  float* red = (float*)(lds + C::RED);

  int chunk, hk, b;
  {
    const int id = blockIdx.x;
    if (a.xmap) {
      const int x = id & 7, slot = id >> 3;
      const int gid = (slot / a.Hkv) * 8 + x;
      hk = slot % a.Hkv;
      b = gid / a.nch;
      chunk = gid % a.nch;
    } else {
      chunk = id % a.nch;
      hk = (id / a.nch) % a.Hkv;
      b = id / (a.nch * a.Hkv);
    }
  }
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int tl = lane & 31, hh = lane >> 5;
  const int ul = tl / GQ, hl = tl % GQ;
  const int M = a.M, RS = M * AT_K + 2;
  float2* ang = (float2*)(lds + C::ANG) + w * 64;
  const int len = min(max(a.seq_len[b], 0), a.cap);
  const int tok0 = chunk * C::CHUNK;
  float* outp = a.part + (((size_t)b * a.Hkv + hk) * a.nch + chunk) * GQ * RS;
  if (tok0 >= len) {
    if (tid < GQ) {
      outp[tid * RS + M * AT_K] = -INFINITY;
      outp[tid * RS + M * AT_K + 1] = 0.f;
    }
    return;
  }
  const int tend = min(len, tok0 + C::CHUNK);
  const int Hq = a.Hkv * GQ;
  const size_t seq_row0 = (size_t)b * a.cap;

  // queries turned by R_{-32u} and scaled (as the 1-bit kernel)
  {
    constexpr int PER = 32 * 64 / AT_THREADS;
    float x[PER], y[PER];
    float2 cs[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int it = m * AT_THREADS + tid, j = it >> 6, jd = it & 63;
      const size_t qo = ((size_t)b * Hq + hk * GQ + j % GQ) * AT_HD + jd;
      if (a.q_f16) {
        x[m] = (float)((const _Float16*)a.q)[qo];
        y[m] = (float)((const _Float16*)a.q)[qo + 64];
      } else {
        x[m] = ((const float*)a.q)[qo];
        y[m] = ((const float*)a.q)[qo + 64];
      }
      cs[m] = a.t2[(j / GQ) * 64 + jd];
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int it = m * AT_THREADS + tid, j = it >> 6, jd = it & 63;
      qt[j * AT_HD + jd] = (x[m] * cs[m].x + y[m] * cs[m].y) * a.qscale;
      qt[j * AT_HD + jd + 64] = (y[m] * cs[m].x - x[m] * cs[m].y) * a.qscale;
    }
  }
  h2 cp[16], sp[16];
  {
    const float4* t1 = (const float4*)(a.t1 + tl * 64 + 32 * hh);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const float4 v = t1[m];
      cp[m] = (h2){(_Float16)v.x, (_Float16)v.z};
      sp[m] = (h2){(_Float16)v.y, (_Float16)v.w};
    }
  }
  const double thl = a.th[lane];
  __syncthreads();

  // this wave's groups: gi = w + AT_WAVES j, j < AQ_NG.  A group's query
  // operand (its columns turned by R_{pq - 32 gb0}, float16) is rebuilt in
  // every pass: one sine/cosine per lane, cheaper than keeping 32 registers
  // per group live across the passes
  const int ngroups = (tend - tok0 + 32 * U - 1) / (32 * U);
  f16v acc[AQ_NG];
#pragma unroll
  for (int j = 0; j < AQ_NG; ++j) acc[j] = (f16v){};
  auto make_bq = [&](int gb0, u4 (&bq)[8]) {
    {
      const int n = max((len - 1) - 32 * gb0, 0);
      double rev = (double)n * thl;
      rev -= floor(rev);
      float s, c;
      sincosf((float)(rev * (2.0 * M_PI)), &s, &c);
      ang[lane] = make_float2(c, s);
    }
    wave_lds_order();
    const float4* qxp = (const float4*)(qt + tl * AT_HD + 32 * hh);
    const float4* qyp = (const float4*)(qt + tl * AT_HD + 64 + 32 * hh);
    const float4* ap = (const float4*)(ang + 32 * hh);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      _Float16 xh[8], yh[8];
#pragma unroll
      for (int m2 = 0; m2 < 2; ++m2) {
        const float4 qx4 = qxp[2 * i + m2], qy4 = qyp[2 * i + m2];
        const float4 va = ap[4 * i + 2 * m2], vb = ap[4 * i + 2 * m2 + 1];
        const float qxv[4] = {qx4.x, qx4.y, qx4.z, qx4.w};
        const float qyv[4] = {qy4.x, qy4.y, qy4.z, qy4.w};
        const float cv[4] = {va.x, va.z, vb.x, vb.z};
        const float sv[4] = {va.y, va.w, vb.y, vb.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = 4 * m2 + r;
          xh[e] = (_Float16)(qxv[r] * cv[r] - qyv[r] * sv[r]);
          yh[e] = (_Float16)(qxv[r] * sv[r] + qyv[r] * cv[r]);
        }
      }
      bq[i] = pack_h8(xh);
      bq[i + 4] = pack_h8(yh);
    }
    wave_lds_order();                               // angle reads before the next writes
  };

  const uint8_t* kcb = a.kc + seq_row0 * a.rowb + hk;
  uint8_t* kcl = lds + C::KC;
  const int npass = (M + 1) >> 1;
  for (int pass = 0; pass < npass; ++pass) {
    const int s0 = 2 * pass;
    const bool two = s0 + 1 < M;                     // uniform
    __syncthreads();                                 // the previous pair's table is read
    {
      // the pair's table (16 u4 per thread) and the chunk's code bytes of
      // the pair's stages (16 per thread, token t stage sl at 2 t + sl),
      // every load issued before the first store
      // the thread index made opaque per pass, so that the addresses
      // derived from it are recomputed here rather than hoisted out of the
      // pass loop and held (spilled) across it
      int tq = tid;
      asm volatile("" : "+v"(tq));
      const u4* src = a.tabk + ((size_t)hk * M + s0) * AT_K * 16;
      const int n = (two ? 2 : 1) * AT_K * 16;       // a single stage's pass: stage 1 zero
      constexpr int PER = AQ_TAB_U4 / AT_THREADS;
      constexpr int PERC = 2 * AQ_CHUNK / AT_THREADS;
      u4 v[PER];
      uint32_t cb[PERC];
#pragma unroll
      for (int r = 0; r < PER; ++r) {
        const int e = min(r * AT_THREADS + tq, n - 1);
        v[r] = src[e];
      }
      {
        const int sl = tq & 1, s = s0 + (two ? sl : 0);
        const uint8_t* cp0 = kcb + (size_t)s * a.Hkv;
#pragma unroll
        for (int r = 0; r < PERC; ++r) {
          const int row = min(tok0 + r * (AT_THREADS / 2) + (tq >> 1), len - 1);
          cb[r] = cp0[(size_t)row * a.rowb];
        }
      }
      {
        // entry e = r * AT_THREADS + tid is chunk tid % 16 of codeword
        // (tid / 16 + 32 r) % 256 of stage r / 8; 32 r leaves k & 15 and
        // so the chunk's slot c ^ (k & 15) unchanged: base + 512 r
        const int kq = tq >> 4, c = tq & 15;
        u4* dst = ktab + (kq << 4) + (c ^ (kq & 15));
        const u4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int r = 0; r < PER; ++r) dst[512 * r] = r * AT_THREADS + tq < n ? v[r] : z;
      }
#pragma unroll
      for (int r = 0; r < PERC; ++r) kcl[r * AT_THREADS + tq] = (uint8_t)cb[r];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < AQ_NG; ++j) {
      const int gi = w + AT_WAVES * j;
      if (gi >= ngroups) continue;                   // uniform per wave
      const int gb0 = (tok0 >> 5) + gi * U;
      const int nblk = min(U, (len - 32 * gb0 + 31) >> 5);
      u4 bq[8];
      make_bq(gb0, bq);
      for (int u = 0; u < nblk; ++u) {
        // the lane's token (rows past the sequence end read the last row's
        // codes; their scores are masked)
        const int t = min(32 * (gb0 + u) + tl, len - 1) - tok0;
        const int c0 = kcl[2 * t], c1 = kcl[2 * t + 1];
        const uint32_t kb0 = aq_base(0, c0, hh), kb1 = aq_base(1, c1, hh);
        const unsigned char* kt8 = lds + C::KTAB;
        const bool mine = ul == u;
        const u4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i2 = 0; i2 < 4; i2 += 2) {
          // the gathers of two k-step pairs issued together (both stages:
          // a single stage's pass reads zeros from stage 1)
          u4 g[2][4];
#pragma unroll
          for (int ii = 0; ii < 2; ++ii) {
            const uint32_t ox = (uint32_t)(i2 + ii) << 4, oy = (uint32_t)(8 | (i2 + ii)) << 4;
            g[ii][0] = *(const u4*)(kt8 + (kb0 ^ ox));
            g[ii][1] = *(const u4*)(kt8 + (kb0 ^ oy));
            g[ii][2] = *(const u4*)(kt8 + (kb1 ^ ox));
            g[ii][3] = *(const u4*)(kt8 + (kb1 ^ oy));
          }
#pragma unroll
          for (int ii = 0; ii < 2; ++ii) {
            const int i = i2 + ii;
            const u4 xa = g[ii][0], ya = g[ii][1], xb = g[ii][2], yb = g[ii][3];
            h2 xr[4], yr[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) {
              // scalar copies before the bit casts; the pair's two codeword
              // pieces summed in float16, then turned by R_t
              const uint32_t xw0 = xa[p], yw0 = ya[p], xw1 = xb[p], yw1 = yb[p];
              const h2 xp = __builtin_bit_cast(h2, xw0) + __builtin_bit_cast(h2, xw1);
              const h2 yp = __builtin_bit_cast(h2, yw0) + __builtin_bit_cast(h2, yw1);
              const h2 c = cp[4 * i + p], sn = sp[4 * i + p];
              xr[p] = __builtin_elementwise_fma(xp, c, -(yp * sn));
              yr[p] = __builtin_elementwise_fma(xp, sn, yp * c);
            }
            const h8 kx = __builtin_shufflevector(
                __builtin_shufflevector(xr[0], xr[1], 0, 1, 2, 3),
                __builtin_shufflevector(xr[2], xr[3], 0, 1, 2, 3), 0, 1, 2, 3, 4, 5, 6, 7);
            const h8 ky = __builtin_shufflevector(
                __builtin_shufflevector(yr[0], yr[1], 0, 1, 2, 3),
                __builtin_shufflevector(yr[2], yr[3], 0, 1, 2, 3), 0, 1, 2, 3, 4, 5, 6, 7);
            const u4 bx = mine ? bq[i] : z, by = mine ? bq[i + 4] : z;
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kx, as_h8(bx), acc[j], 0, 0, 0);
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ky, as_h8(by), acc[j], 0, 0, 0);
          }
        }
      }
    }
  }

  // ---- softmax: one reference per head for the workgroup.  Register v of
  // a lane holds token row t = 8 (v / 4) + 4 hh + v % 4 of block ul of the
  // group, for query head hl.
  float sc[AQ_NG][16];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < AQ_NG; ++j) {
    const int gi = w + AT_WAVES * j;
    const int rowb = 32 * ((tok0 >> 5) + gi * U + ul);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int t = 8 * (v >> 2) + 4 * hh + (v & 3);
      const bool ok = gi < ngroups && rowb + t < len;
      sc[j][v] = ok ? acc[j][v] : -INFINITY;
      mx = fmaxf(mx, sc[j][v]);
    }
  }
#pragma unroll
  for (int off = GQ; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  __syncthreads();                                   // every wave is done with the table
  if (lane < GQ) red[w * 2 * GQ + lane] = mx;        // lane h (ul = 0, hh = 0) holds head h
  // the chunk's value code bytes, token t stage m at 16 t + m (16 loads in
  // flight per thread)
  uint8_t* vcl = lds + C::VC;
  {
    const uint8_t* vcb = a.vc + seq_row0 * a.rowb + hk;
    const int n = (tend - tok0) * M;
    constexpr int B16 = 16;
    for (int e0 = tid; e0 < n; e0 += B16 * AT_THREADS) {
      uint32_t cv[B16];
#pragma unroll
      for (int r = 0; r < B16; ++r) {
        const int e = min(e0 + r * AT_THREADS, n - 1), t = e / M, m = e - t * M;
        cv[r] = vcb[(size_t)(tok0 + t) * a.rowb + m * a.Hkv];
      }
#pragma unroll
      for (int r = 0; r < B16; ++r) {
        const int e = e0 + r * AT_THREADS, t = e / M, m = e - t * M;
        if (e < n) vcl[16 * t + m] = (uint8_t)cv[r];
      }
    }
  }
  __syncthreads();
  float mref = -INFINITY;
#pragma unroll
  for (int v = 0; v < AT_WAVES; ++v) mref = fmaxf(mref, red[v * 2 * GQ + hl]);
  // mref is finite: the chunk holds at least one token
  // softmax sum of the lane's column (float32)
  float lsum = 0.f;
#pragma unroll
  for (int j = 0; j < AQ_NG; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) lsum += __builtin_amdgcn_exp2f(sc[j][v] - mref);   // 0 if masked
#pragma unroll
  for (int off = GQ; off < 64; off <<= 1) lsum += __shfl_xor(lsum, off);
  if (lane < GQ) red[w * 2 * GQ + GQ + lane] = lsum;
  // value bins, SG stages at a time: every lane adds its own head's weight
  // of each of its 16 tokens into the token's stage bins, as 64-bit fixed
  // point (weight x 2^32, weights <= 1: exact integer sums, the same in any
  // order); a token's codes are one 16-byte LDS read, the next token's
  // issued before the current one's adds.  The bins of each stage group
  // are then written to the chunk's record as float32.
  constexpr int SG = 32 / GQ;                        // SG x 256 x GQ x 8 bytes = 64 KiB
  for (int mg = 0; mg < M; mg += SG) {
    const int ms = min(SG, M - mg);
    __syncthreads();                                 // the previous group's bins are written out
    for (int e = tid; e < ms * AT_K * GQ; e += AT_THREADS) bins[e] = 0ull;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < AQ_NG; ++j) {
      const int gi = w + AT_WAVES * j;
      if (gi >= ngroups) continue;                   // uniform per wave
      const int rowb = 32 * ((tok0 >> 5) + gi * U + ul);
      auto codes_of = [&](int v) {
        const int t = 8 * (v >> 2) + 4 * hh + (v & 3);
        return *(const u4*)(vcl + 16 * (min(rowb + t, len - 1) - tok0));
      };
      u4 cn = codes_of(0);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(sc[j][v] - mref);
        const unsigned long long q = (unsigned long long)(p * 4294967296.0f);
        const u4 cc = cn;
        if (v + 1 < 16) cn = codes_of(v + 1);
        const int t = 8 * (v >> 2) + 4 * hh + (v & 3);
        if (rowb + t < len) {
#pragma unroll
          for (int m2 = 0; m2 < SG; ++m2) {
            if (m2 >= ms) break;
            const int m = mg + m2;
            const int k = (cc[m >> 2] >> (8 * (m & 3))) & 255;
            atomicAdd(&bins[(m2 * AT_K + k) * GQ + hl], q);
          }
        }
      }
    }
    __syncthreads();
    for (int e = tid; e < GQ * ms * AT_K; e += AT_THREADS) {
      const int h = e / (ms * AT_K), r = e - h * (ms * AT_K);
      outp[h * RS + mg * AT_K + r] = (float)((double)bins[r * GQ + h] * 0x1p-32);
    }
  }
  if (tid < GQ) {
    float l = 0.f, mr = -INFINITY;
#pragma unroll
    for (int v = 0; v < AT_WAVES; ++v) {
      l += red[v * 2 * GQ + GQ + tid];
      mr = fmaxf(mr, red[v * 2 * GQ + tid]);
    }
    outp[tid * RS + M * AT_K] = mr;
    outp[tid * RS + M * AT_K + 1] = l;
  }
}

// Value side, one workgroup per (sequence, key/value head, stage m): the
// chunks' bins of stage m merged with their references, W_h[k] =
// sum_c 2^(m_c,h - M_h) W_c,h[k] (float64), then contracted with the
// stage's value codewords fl(g s): o_m,h[n] = sum_k W_h[k] fl(g_k s_kn).
constexpr int AQ_VT = 256;
constexpr int AQ_VCH = 64;      // chunks merged per round (LDS factors [4][AQ_VCH])
__global__ void __launch_bounds__(AQ_VT) attn_rq_values_kernel(const float* __restrict__ part,
                                                               int GQ, int Hkv, int nch, int M,
                                                               const float* __restrict__ vg,
                                                               const float* __restrict__ vs,
                                                               double* __restrict__ om) {
  __shared__ double wb[4][AT_K];
  __shared__ double hs[4][AT_HD];
  __shared__ double fac[4][AQ_VCH];
  __shared__ float mcl[4][AQ_VCH], lcl[4][AQ_VCH];
  __shared__ float mrefs[4];
  __shared__ float gl[AT_K];
  const int m = blockIdx.x % M, hk = (blockIdx.x / M) % Hkv, b = blockIdx.x / (M * Hkv);
  const int tid = threadIdx.x;
  const int RS = M * AT_K + 2;
  const float* p0 = part + ((size_t)b * Hkv + hk) * nch * GQ * RS;
  const size_t cs = (size_t)GQ * RS;
  const size_t cb = ((size_t)m * Hkv + hk) * AT_K;
  // a launch is a chain of dependent loads: each step below issues all of
  // its loads together (the chunk records one per thread, every head's bins
  // of a round, 64 codeword elements per thread)
  gl[tid] = vg[cb + tid];                            // the stage's gains
  // reference per head: the largest record among chunks with tokens
  {
    float mr = -INFINITY;
    for (int c0 = 0; c0 < nch; c0 += AQ_VCH) {
      const int nc = min(AQ_VCH, nch - c0);
      if (tid < GQ * nc) {
        const int h = tid / nc, c = c0 + tid % nc;
        const float* p = p0 + (size_t)h * RS + c * cs;
        mcl[h][tid % nc] = p[M * AT_K];
        lcl[h][tid % nc] = p[M * AT_K + 1];
      }
      __syncthreads();
      if (tid < GQ)
        for (int c = 0; c < nc; ++c) mr = lcl[tid][c] > 0.f ? fmaxf(mr, mcl[tid][c]) : mr;
      __syncthreads();
    }
    if (tid < GQ) mrefs[tid] = mr;
  }
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int c0 = 0; c0 < nch; c0 += AQ_VCH) {
    const int nc = min(AQ_VCH, nch - c0);
    __syncthreads();                                 // mrefs written, previous factors read
    if (tid < GQ * nc) {
      const int h = tid / nc, c = c0 + tid % nc;
      float mc, lc;
      if (nch <= AQ_VCH) {                           // one round: the records are in LDS
        mc = mcl[h][tid % nc];
        lc = lcl[h][tid % nc];
      } else {
        const float* p = p0 + (size_t)h * RS + c * cs;
        mc = p[M * AT_K];
        lc = p[M * AT_K + 1];
      }
      fac[h][tid % nc] = lc > 0.f ? exp2((double)mc - (double)mrefs[h]) : 0.0;
    }
    __syncthreads();
    // thread k: codeword k of stage m, every head, the round's chunks, eight
    // chunks of every head in flight
    constexpr int UN = 8;
    for (int c1 = 0; c1 < nc; c1 += UN) {
      float bv[4][UN];
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float* p = p0 + (size_t)min(h, GQ - 1) * RS + (size_t)m * AT_K + tid;
#pragma unroll
        for (int u = 0; u < UN; ++u) bv[h][u] = p[(size_t)(c0 + min(c1 + u, nc - 1)) * cs];
      }
#pragma unroll
      for (int h = 0; h < 4; ++h)
        if (h < GQ) {
#pragma unroll
          for (int u = 0; u < UN; ++u)
            if (c1 + u < nc) {
              // a chunk without tokens (factor 0) never wrote its bins: the
              // slots hold stale workspace contents, kept out of the sum
              const double f = fac[h][c1 + u];
              acc[h] += f > 0.0 ? f * (double)bv[h][u] : 0.0;
            }
        }
    }
  }
  for (int h = 0; h < GQ; ++h) wb[h][tid] = acc[h];
  __syncthreads();
  // contraction: thread (half, n) takes codewords half * 128 .. + 127,
  // element n of each, 64 loads in flight
  const int n = tid & (AT_HD - 1), half = tid >> 7;
  const float* sp = vs + cb * AT_HD + n;
  double o[4] = {0.0, 0.0, 0.0, 0.0};
  constexpr int UK = 64;
  for (int k0 = half * 128; k0 < half * 128 + 128; k0 += UK) {
    float sv[UK];
#pragma unroll
    for (int u = 0; u < UK; ++u) sv[u] = sp[(size_t)(k0 + u) * AT_HD];
#pragma unroll
    for (int u = 0; u < UK; ++u) {
      const double cw = (double)(gl[k0 + u] * sv[u]);                // fl(g s)
#pragma unroll
      for (int h = 0; h < 4; ++h)
        if (h < GQ) o[h] = fma(wb[h][k0 + u], cw, o[h]);
    }
  }
  if (half) {
#pragma unroll
    for (int h = 0; h < 4; ++h) hs[h][n] = o[h];
  }
  __syncthreads();
  if (!half) {
    for (int h = 0; h < GQ; ++h)
      om[(((size_t)b * Hkv + hk) * GQ + h) * M * AT_HD + (size_t)m * AT_HD + n] = o[h] + hs[h][n];
  }
}

// Output of one (sequence, query head): o = sum_m o_m / sum_c 2^(m_c - M) l_c.
__global__ void __launch_bounds__(AT_HD) attn_rq_out_kernel(const float* __restrict__ part,
                                                            const double* __restrict__ om,
                                                            int Hq, int Hkv, int nch, int M,
                                                            float* __restrict__ out, AttnTag tag,
                                                            const uint32_t* __restrict__ tagp) {
  const int bq = blockIdx.x, b = bq / Hq, hq = bq % Hq, n = threadIdx.x;
  bool tag_ok = true;
#pragma unroll
  for (int i = 0; i < AT_TAG_WORDS; ++i) tag_ok &= tagp[i] == tag.w[i];
  if (!tag_ok) {
    out[(size_t)bq * AT_HD + n] = __builtin_nanf("");
    return;
  }
  const int GQ = Hq / Hkv, hk = hq / GQ, h = hq % GQ;
  const int RS = M * AT_K + 2;
  const float* p = part + (((size_t)b * Hkv + hk) * nch * GQ + h) * RS;
  const size_t cs = (size_t)GQ * RS;
  float mref = -INFINITY;
  for (int c = 0; c < nch; ++c) {
    const float mc = p[c * cs + M * AT_K], lc = p[c * cs + M * AT_K + 1];
    mref = lc > 0.f ? fmaxf(mref, mc) : mref;
  }
  double den = 0.0;
  for (int c = 0; c < nch; ++c) {
    const float mc = p[c * cs + M * AT_K], lc = p[c * cs + M * AT_K + 1];
    den += lc > 0.f ? exp2((double)mc - (double)mref) * (double)lc : 0.0;
  }
  const double* op = om + (((size_t)b * Hkv + hk) * GQ + h) * M * AT_HD + n;
  double v = 0.0;
  for (int m = 0; m < M; ++m) v += op[(size_t)m * AT_HD];
  out[(size_t)bq * AT_HD + n] = den > 0.0 ? (float)(v / den) : 0.f;
}

struct AqPlan {
  int GQ, nch, W;
  size_t off_tag, off_t1, off_t2, off_th, off_tk, off_part, off_om, bytes;
};

gsrq_status aq_plan(const gsrq_attn_shape* a, const gsrq_shape* kv, AqPlan& p) {
  p.GQ = a->Hq / a->Hkv;
  const int M = kv->M;
  const int64_t nch = ((int64_t)a->cap + AQ_CHUNK - 1) / AQ_CHUNK;
  if (nch * a->Hkv * a->B > INT32_MAX || (int64_t)M * a->Hkv * a->B > INT32_MAX)
    return GSRQ_E_UNSUPPORTED;
  p.nch = (int)nch;
  p.W = (int)(((int64_t)M * a->Hkv * 8 + 31) / 32);
  const size_t pairs = (size_t)a->B * a->Hkv;
  p.off_tag = 0;
  p.off_t1 = 256;
  p.off_t2 = p.off_t1 + align256(32 * 64 * sizeof(float2));
  p.off_th = p.off_t2 + align256(32 * 64 * sizeof(float2));
  p.off_tk = p.off_th + align256(64 * sizeof(double));
  p.off_part = p.off_tk + align256((size_t)a->Hkv * M * AT_K * 16 * sizeof(u4));
  p.off_om = p.off_part + align256(pairs * p.nch * p.GQ * ((size_t)M * AT_K + 2) * sizeof(float));
  p.bytes = p.off_om + align256(pairs * p.GQ * (size_t)M * AT_HD * sizeof(double));
  return GSRQ_OK;
}

template <int GQ> gsrq_status aq_launch(const AqArgs& args, int B, int Hkv, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute((const void*)attn_rq_chunk_kernel<GQ>,
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            AqCfg<GQ>::BYTES) != hipSuccess)
      return GSRQ_E_HIP;
    attr_set = true;
  }
  TimedLaunch tm(GSRQ_KERNEL_ATTENTION, st);
  const int blocks = args.nch * Hkv * B;
  attn_rq_chunk_kernel<GQ><<<blocks, AT_THREADS, AqCfg<GQ>::BYTES, st>>>(args);
  return launch_ok();
}

}  // namespace

extern "C" {

gsrq_status gsrq_attn_workspace_bytes(const gsrq_attn_shape* a, size_t* bytes) {
  if (!bytes) return GSRQ_E_ARG;
  AttnPlan p;
  gsrq_status e = attn_plan(a, p);
  if (e) return e;
  *bytes = p.bytes;
  return GSRQ_OK;
}

}  // extern "C"

namespace {
gsrq_status attn_layout(const gsrq_attn_shape* a, const gsrq_shape* kv, AttnPlan& p,
                        AqPlan& qp, bool& rq);
}  // namespace

extern "C" {

gsrq_status gsrq_attn_workspace_bytes_kv(const gsrq_attn_shape* a, const gsrq_shape* kv,
                                         size_t* bytes) {
  if (!bytes) return GSRQ_E_ARG;
  AttnPlan p;
  AqPlan qp;
  bool rq = false;
  gsrq_status e = attn_layout(a, kv, p, qp, rq);
  if (e) return e;
  *bytes = rq ? qp.bytes : p.bytes;
  return GSRQ_OK;
}

}  // extern "C"

namespace {

// Host validation shared by both entry points (no HIP call).
// Code layouts: the 1-bit cache (d = 8, K = 256, one stage) or a residual-
// coded one with one subspace per head (d = head_dim, K = 256, 1 <= M <= 32).
gsrq_status attn_layout(const gsrq_attn_shape* a, const gsrq_shape* kv, AttnPlan& p,
                        AqPlan& qp, bool& rq) {
  gsrq_status e = attn_plan(a, p);
  if (e) return e;
  if (!kv || kv->N < 1 || kv->D < 1 || kv->d < 1 || kv->K < 2 || kv->M < 1) return GSRQ_E_ARG;
  if (kv->D != a->Hkv * a->head_dim) return GSRQ_E_ARG;
  if (kv->D % kv->d || !is_pow2(kv->K)) return GSRQ_E_ARG;
  rq = kv->d == a->head_dim && kv->K == AT_K && kv->M <= AQ_MAXM;
  if (!rq && (kv->d != 8 || kv->K != AT_K || kv->M != 1)) return GSRQ_E_UNSUPPORTED;
  if (rq) return aq_plan(a, kv, qp);
  return GSRQ_OK;
}

gsrq_status attn_validate(const gsrq_attn_shape* a, const gsrq_shape* kv,
                          const uint32_t* k_codes, const uint32_t* v_codes,
                          const int32_t* seq_len, const float* k_gain, const float* k_shape,
                          const float* v_gain, const float* v_shape, const void* q,
                          gsrq_dtype q_dtype, float* out, AttnPlan& p, AqPlan& qp, bool& rq) {
  gsrq_status e = attn_layout(a, kv, p, qp, rq);
  if (e) return e;
  if (kv->N < (int64_t)a->B * a->cap) return GSRQ_E_ARG;
  if (!k_codes || !v_codes || !seq_len || !k_gain || !k_shape || !v_gain || !v_shape || !q ||
      !out)
    return GSRQ_E_ARG;
  if ((uintptr_t)k_codes % 16 || (uintptr_t)v_codes % 16 || (uintptr_t)k_shape % 16 ||
      (uintptr_t)v_shape % 16 || (uintptr_t)q % 16)
    return GSRQ_E_ARG;
  if (q_dtype != GSRQ_F32 && q_dtype != GSRQ_F16) return GSRQ_E_ARG;
  return GSRQ_OK;
}

// The launches of one call on a workspace of p.bytes at ws (256-byte aligned).
gsrq_status attn_run(const gsrq_attn_shape* a, const AttnPlan& p, const uint32_t* k_codes,
                     const uint32_t* v_codes, const int32_t* seq_len, const float* k_gain,
                     const float* k_shape, const float* v_gain, const float* v_shape,
                     const void* q, gsrq_dtype q_dtype, float* out, char* ws, void* stream) {
  gsrq_status e;
  hipStream_t st = (hipStream_t)stream;
  AttnArgs args;
  args.kc = k_codes;
  args.vc = v_codes;
  args.seq_len = seq_len;
  args.q = q;
  args.q_f16 = q_dtype == GSRQ_F16;
  args.t1 = (const float2*)(ws + p.off_t1);
  args.t2 = (const float2*)(ws + p.off_t2);
  args.th = (const double*)(ws + p.off_th);
  args.tabk = (const u4*)(ws + p.off_tk);
  args.tabv = (const u4*)(ws + p.off_tv);
  args.part = (float*)(ws + p.off_part);
  args.cap = a->cap;
  args.W = a->Hkv * 4;
  args.Hkv = a->Hkv;
  args.nch = p.nch;
  args.rpc = p.rpc;
  args.xmap = ((int64_t)a->B * p.nch) % 8 == 0 ? 1 : 0;
  args.qscale = (float)((double)a->scale * 1.4426950408889634);
  const int ncw = a->Hkv * AT_SUB * AT_K;
  AttnTag tag = {};
  {
    const void* ptrs[4] = {k_gain, k_shape, v_gain, v_shape};
    tag.w[0] = AT_TAG_MAGIC;
    tag.w[1] = (uint32_t)a->Hkv;
    tag.w[2] = (uint32_t)a->head_dim;
    memcpy(&tag.w[3], &a->rope_base, sizeof(float));
    for (int i = 0; i < 4; ++i) {
      const uint64_t v = (uint64_t)(uintptr_t)ptrs[i];
      tag.w[4 + 2 * i] = (uint32_t)v;
      tag.w[5 + 2 * i] = (uint32_t)(v >> 32);
    }
    tag.w[12] = ~AT_TAG_MAGIC;
  }
  uint32_t* tagp = (uint32_t*)(ws + p.off_tag);
  if (!(a->flags & GSRQ_ATTN_TABLES_READY)) {
    attn_tables_kernel<<<AT_TRIG_BLOCKS + (2 * ncw + 255) / 256, 256, 0, st>>>(
        (double)a->rope_base, (float2*)(ws + p.off_t1), (float2*)(ws + p.off_t2),
        (double*)(ws + p.off_th), k_gain, k_shape, v_gain, v_shape, ncw, (u4*)(ws + p.off_tk),
        (u4*)(ws + p.off_tv), tag, tagp);
    e = launch_ok();
    if (e) return e;
  }
  if (p.GQ == 1) e = attn_launch<1>(args, a->B, a->Hkv, st);
  else if (p.GQ == 2) e = attn_launch<2>(args, a->B, a->Hkv, st);
  else e = attn_launch<4>(args, a->B, a->Hkv, st);
  if (e) return e;
  attn_merge_kernel<<<a->B * a->Hq, AT_HD, 0, st>>>(args.part, a->Hq, a->Hkv, p.nch, out, tag,
                                                     tagp);
  return launch_ok();
}

// The launches of one call on a residual-coded cache.
gsrq_status aq_run(const gsrq_attn_shape* a, const gsrq_shape* kv, const AqPlan& p,
                   const uint32_t* k_codes, const uint32_t* v_codes, const int32_t* seq_len,
                   const float* k_gain, const float* k_shape, const float* v_gain,
                   const float* v_shape, const void* q, gsrq_dtype q_dtype, float* out,
                   char* ws, void* stream) {
  gsrq_status e;
  hipStream_t st = (hipStream_t)stream;
  const int M = kv->M;
  AqArgs args;
  args.kc = (const uint8_t*)k_codes;
  args.vc = (const uint8_t*)v_codes;
  args.seq_len = seq_len;
  args.q = q;
  args.q_f16 = q_dtype == GSRQ_F16;
  args.t1 = (const float2*)(ws + p.off_t1);
  args.t2 = (const float2*)(ws + p.off_t2);
  args.th = (const double*)(ws + p.off_th);
  args.tabk = (const u4*)(ws + p.off_tk);
  args.part = (float*)(ws + p.off_part);
  args.cap = a->cap;
  args.rowb = 4 * p.W;
  args.Hkv = a->Hkv;
  args.M = M;
  args.nch = p.nch;
  args.xmap = ((int64_t)a->B * p.nch) % 8 == 0 ? 1 : 0;
  args.qscale = (float)((double)a->scale * 1.4426950408889634);
  AttnTag tag = {};
  {
    const void* ptrs[4] = {k_gain, k_shape, v_gain, v_shape};
    tag.w[0] = AT_TAG_MAGIC;
    tag.w[1] = (uint32_t)a->Hkv;
    tag.w[2] = (uint32_t)a->head_dim;
    memcpy(&tag.w[3], &a->rope_base, sizeof(float));
    for (int i = 0; i < 4; ++i) {
      const uint64_t v = (uint64_t)(uintptr_t)ptrs[i];
      tag.w[4 + 2 * i] = (uint32_t)v;
      tag.w[5 + 2 * i] = (uint32_t)(v >> 32);
    }
    tag.w[12] = ~AT_TAG_MAGIC;
    tag.w[13] = 0x52510000u | (uint32_t)M;         // residual-coded tables of M stages
  }
  uint32_t* tagp = (uint32_t*)(ws + p.off_tag);
  if (!(a->flags & GSRQ_ATTN_TABLES_READY)) {
    // RoPE tables and the tag (no 1-bit codeword tables), then the key table
    attn_tables_kernel<<<AT_TRIG_BLOCKS, 256, 0, st>>>(
        (double)a->rope_base, (float2*)(ws + p.off_t1), (float2*)(ws + p.off_t2),
        (double*)(ws + p.off_th), k_gain, k_shape, v_gain, v_shape, 0, nullptr, nullptr, tag,
        tagp);
    if ((e = launch_ok())) return e;
    const int64_t n = (int64_t)a->Hkv * M * AT_K * 16;
    attn_rq_keytab_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(k_gain, k_shape, a->Hkv,
                                                                        M, (u4*)(ws + p.off_tk));
    if ((e = launch_ok())) return e;
  }
  if (p.GQ == 1) e = aq_launch<1>(args, a->B, a->Hkv, st);
  else if (p.GQ == 2) e = aq_launch<2>(args, a->B, a->Hkv, st);
  else e = aq_launch<4>(args, a->B, a->Hkv, st);
  if (e) return e;
  double* om = (double*)(ws + p.off_om);
  attn_rq_values_kernel<<<a->B * a->Hkv * M, AQ_VT, 0, st>>>(args.part, p.GQ, a->Hkv, p.nch, M,
                                                             v_gain, v_shape, om);
  if ((e = launch_ok())) return e;
  attn_rq_out_kernel<<<a->B * a->Hq, AT_HD, 0, st>>>(args.part, om, a->Hq, a->Hkv, p.nch, M, out,
                                                     tag, tagp);
  return launch_ok();
}

// Scratch of gsrq_attn_decode_noalloc: a file-scope device array, one copy
// per GPU, alive until the process ends.  In host code its name only stands
// for the variable; its device address on a GPU comes from
// hipGetSymbolAddress with that GPU current, taken once per device and kept.
constexpr size_t AT_NOALLOC_BYTES = GSRQ_ATTN_NOALLOC_BYTES;
static __device__ __align__(256) unsigned char scratch[AT_NOALLOC_BYTES];

constexpr int AT_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[AT_MAX_DEVICES] = {};

gsrq_status scratch_on_current_device(char** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return GSRQ_E_HIP;
  if (dev >= AT_MAX_DEVICES) return GSRQ_E_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GSRQ_E_HIP;
    g_scratch_ptr[dev] = (char*)p;
  }
  *ptr = g_scratch_ptr[dev];
  return GSRQ_OK;
}

}  // namespace

extern "C" {

gsrq_status gsrq_attn_decode(const gsrq_attn_shape* a, const gsrq_shape* kv,
                             const uint32_t* k_codes, const uint32_t* v_codes,
                             const int32_t* seq_len, const float* k_gain, const float* k_shape,
                             const float* v_gain, const float* v_shape, const void* q,
                             gsrq_dtype q_dtype, float* out, void* workspace, size_t ws_bytes,
                             void* stream) {
  AttnPlan p;
  AqPlan qp;
  bool rq = false;
  gsrq_status e = attn_validate(a, kv, k_codes, v_codes, seq_len, k_gain, k_shape, v_gain,
                                v_shape, q, q_dtype, out, p, qp, rq);
  if (e) return e;
  if (!workspace || (uintptr_t)workspace % 256) return GSRQ_E_ARG;
  if (ws_bytes < (rq ? qp.bytes : p.bytes)) return GSRQ_E_WORKSPACE;
  if (rq)
    return aq_run(a, kv, qp, k_codes, v_codes, seq_len, k_gain, k_shape, v_gain, v_shape, q,
                  q_dtype, out, (char*)workspace, stream);
  return attn_run(a, p, k_codes, v_codes, seq_len, k_gain, k_shape, v_gain, v_shape, q, q_dtype,
                  out, (char*)workspace, stream);
}

gsrq_status gsrq_attn_decode_noalloc(const gsrq_attn_shape* a, const gsrq_shape* kv,
                                     const uint32_t* k_codes, const uint32_t* v_codes,
                                     const int32_t* seq_len, const float* k_gain,
                                     const float* k_shape, const float* v_gain,
                                     const float* v_shape, const void* q, gsrq_dtype q_dtype,
                                     float* out, void* stream) {
  AttnPlan p;
  AqPlan qp;
  bool rq = false;
  gsrq_status e = attn_validate(a, kv, k_codes, v_codes, seq_len, k_gain, k_shape, v_gain,
                                v_shape, q, q_dtype, out, p, qp, rq);
  if (e) return e;
  if ((rq ? qp.bytes : p.bytes) > AT_NOALLOC_BYTES) return GSRQ_E_WORKSPACE;
  char* ws = nullptr;
  if ((e = scratch_on_current_device(&ws))) return e;
  if (rq)
    return aq_run(a, kv, qp, k_codes, v_codes, seq_len, k_gain, k_shape, v_gain, v_shape, q,
                  q_dtype, out, ws, stream);
  return attn_run(a, p, k_codes, v_codes, seq_len, k_gain, k_shape, v_gain, v_shape, q, q_dtype,
                  out, ws, stream);
}

}  // extern "C"
