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
//    group.  Both sides enter as hi + lo float16 pairs (three products per
//    k-step), so scores carry about 22 bits, as a float32 dot product would.
//    RoPE enters as a relative rotation: score(i) = (R_{pq - 32b} q) .
//    (R_t k_i) for token i = 32 b + t, so the rotation of a key depends only
//    on its row t in the block (fixed per lane) and that of the query on the
//    group (one sine/cosine per lane per group).
//  * Softmax per wave with a running reference maximum per query head
//    (raised by a margin, with the wave's sums rescaled, when a block's
//    scores exceed it).
//  * Values on the matrix cores: the weights leave the score accumulators
//    already in the A-operand layout of the value product (hi + lo float16),
//    and the B operand gathers each token's float16 value codeword element
//    from a second LDS table, in the transposed layout the product needs,
//    through the block's value codes staged in LDS by subspace.
//  * The waves' partial results are merged at the end of the chunk, and a
//    second kernel merges the chunks of every (sequence, query head) with
//    their reference maxima (the split form of one softmax).
#include <algorithm>

#include "gsrq_common.h"

namespace {

constexpr int AT_HD = 128;            // head dimension
constexpr int AT_SUB = 16;            // d = 8 subspaces per head
constexpr int AT_K = 256;             // codewords per codebook
constexpr int AT_WAVES = 4;
constexpr int AT_THREADS = AT_WAVES * 64;
constexpr int AT_BLK = 32;            // tokens per MFMA block
constexpr int AT_PART = AT_HD + 2;    // partial record: o[128], reference max, sum
constexpr int AT_TARGET_WG = 512;     // workgroups aimed for per launch (2 per CU)
constexpr float AT_HEADROOM = 8.f;    // log2 margin of a raised reference maximum
constexpr float AT_PSHIFT = 15.f;     // weights 2^(s - m + 15) <= 2^15: float16 range
constexpr int AT_TAB = AT_SUB * AT_K * 8;   // float16 elements of one codeword table
constexpr int AT_RED = 8 + 4 * AT_HD;       // floats per wave in the final merge

template <int GQ> struct AtCfg {
  static constexpr int U = 32 / GQ;                         // blocks per wave group
  static constexpr int ROUND = AT_WAVES * U * AT_BLK;       // tokens of one group per wave
  // LDS layout in bytes
  static constexpr int KTAB = 0;                            // f16 [16][256][8] keys
  static constexpr int VTAB = KTAB + AT_TAB * 2;            // f16 [16][256][8] values
  static constexpr int VCS = VTAB + AT_TAB * 2;             // u8 [WAVES][16][32] value codes
  static constexpr int ANG = VCS + AT_WAVES * AT_SUB * AT_BLK;      // float2 [WAVES][64]
  static constexpr int RED = ANG + AT_WAVES * 64 * 8;               // f32 [WAVES][AT_RED]
  static constexpr int BYTES = RED + AT_WAVES * AT_RED * 4;
};
static_assert(AtCfg<4>::BYTES <= 160 * 1024, "LDS budget");

struct AttnArgs {
  const uint32_t* kc;       // [B][cap][W] key codes
  const uint32_t* vc;       // [B][cap][W] value codes
  const int32_t* seq_len;   // [B]
  const float* kg;          // [G][256] key gains
  const float* ks;          // [G][256][8] key shapes
  const float* vg;
  const float* vs;
  const void* q;            // [B][Hq][128]
  int q_f16;
  const float2* t1;         // [32][64] cos/sin of t theta_j
  const float2* t2;         // [32][64] cos/sin of 32 u theta_j
  const double* th;         // [64] theta_j / 2 pi
  float* part;              // [B][Hkv][nch][GQ][AT_PART]
  int cap, W, Hkv, nch, rpc;
  float qscale;             // softmax scale * log2(e)
};

// cos/sin tables of the rotations a block needs (float64 arithmetic).
__global__ void __launch_bounds__(256) attn_tables_kernel(double base, float2* __restrict__ t1,
                                                          float2* __restrict__ t2,
                                                          double* __restrict__ th) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= 32 * 64) return;
  const int t = i >> 6, j = i & 63;
  const double theta = pow(base, -2.0 * j / AT_HD);
  double s, c;
  sincos((double)t * theta, &s, &c);
  t1[i] = make_float2((float)c, (float)s);
  sincos(32.0 * t * theta, &s, &c);
  t2[i] = make_float2((float)c, (float)s);
  if (t == 0) th[j] = theta / (2.0 * M_PI);
}

// v = hi + lo with hi = fp16(v), lo = fp16(v - hi): about 22 bits of v.
__device__ __forceinline__ void split16(float v, _Float16& hi, _Float16& lo) {
  hi = (_Float16)v;
  lo = (_Float16)(v - (float)hi);
}

template <int GQ>
__global__ void __launch_bounds__(AT_THREADS, 1) attn_chunk_kernel(AttnArgs a) {
  using C = AtCfg<GQ>;
  constexpr int U = C::U;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  _Float16* ktab = (_Float16*)(lds + C::KTAB);
  _Float16* vtab = (_Float16*)(lds + C::VTAB);
  float* red = (float*)(lds + C::RED);

  const int chunk = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int tl = lane & 31, hh = lane >> 5;
  const int ul = tl / GQ, hl = tl % GQ;      // B-operand column: block variant, query head
  unsigned char* vcs = lds + C::VCS + w * AT_SUB * AT_BLK;
  float2* ang = (float2*)(lds + C::ANG) + w * 64;
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

  // codeword tables: fp16(fp32(g * s)), the float16 decode of a codeword
  for (int i = tid; i < AT_SUB * AT_K * 2; i += AT_THREADS) {
    const int cw = i >> 1, half = i & 1;
    const size_t src = ((size_t)g0 * AT_K + cw) * 8 + half * 4;
    const float gk = a.kg[(size_t)g0 * AT_K + cw], gv = a.vg[(size_t)g0 * AT_K + cw];
    const f4 sk = *(const f4*)(a.ks + src), sv = *(const f4*)(a.vs + src);
    *(uint2*)(ktab + cw * 8 + half * 4) =
        make_uint2(pack2((_Float16)(gk * sk[0]), (_Float16)(gk * sk[1])),
                   pack2((_Float16)(gk * sk[2]), (_Float16)(gk * sk[3])));
    *(uint2*)(vtab + cw * 8 + half * 4) =
        make_uint2(pack2((_Float16)(gv * sv[0]), (_Float16)(gv * sv[1])),
                   pack2((_Float16)(gv * sv[2]), (_Float16)(gv * sv[3])));
  }

  // lane constant: R_t for the lane's token row; element m < 32 of a lane
  // is head element jd = 32 hh + m, paired with jd + 64
  float ct[32], st[32];
  {
    const float4* t1 = (const float4*)(a.t1 + tl * 64 + 32 * hh);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const float4 v = t1[m];
      ct[2 * m] = v.x; st[2 * m] = v.y; ct[2 * m + 1] = v.z; st[2 * m + 1] = v.w;
    }
  }
  const size_t qoff = ((size_t)b * Hq + hk * GQ + hl) * AT_HD + 32 * hh;
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
    __builtin_amdgcn_wave_barrier();
    // query of the lane's column turned by R_{pq - 32 gb0} R_{-32u} (its
    // block's relative rotation), split hi + lo into float16 pairs; loaded
    // again for every group so that no float32 copy stays live
    u4 bqh[8], bql[8];
    {
      int zero = 0;
      asm volatile("" : "+s"(zero));
      float qx[32], qy[32];
      if (a.q_f16) {
        const u4* qp = (const u4*)((const _Float16*)a.q + qoff + zero);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const h8 x = as_h8(qp[m]), y = as_h8(qp[m + 8]);
#pragma unroll
          for (int e = 0; e < 8; ++e) { qx[8 * m + e] = (float)x[e]; qy[8 * m + e] = (float)y[e]; }
        }
      } else {
        const f4* qp = (const f4*)((const float*)a.q + qoff + zero);
#pragma unroll
        for (int m = 0; m < 8; ++m) {
          const f4 x = qp[m], y = qp[m + 16];
#pragma unroll
          for (int e = 0; e < 4; ++e) { qx[4 * m + e] = x[e]; qy[4 * m + e] = y[e]; }
        }
      }
      const float4* t2 = (const float4*)(a.t2 + ul * 64 + 32 * hh + zero);
      const float4* ap = (const float4*)(ang + 32 * hh);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        _Float16 xh[8], xl[8], yh[8], yl[8];
#pragma unroll
        for (int m2 = 0; m2 < 4; ++m2) {
          const float4 v2 = t2[4 * i + m2];
          const float4 v = ap[4 * i + m2];
#pragma unroll
          for (int r2 = 0; r2 < 2; ++r2) {
            const int e = 2 * m2 + r2, m = 8 * i + e;
            const float c2 = r2 ? v2.z : v2.x, s2 = r2 ? v2.w : v2.y;
            const float x1 = qx[m] * c2 + qy[m] * s2;     // R_{-32u}
            const float y1 = qy[m] * c2 - qx[m] * s2;
            const float c = r2 ? v.z : v.x, s = r2 ? v.w : v.y;
            split16(x1 * c - y1 * s, xh[e], xl[e]);       // R_{pq - 32 gb0}
            split16(x1 * s + y1 * c, yh[e], yl[e]);
          }
        }
        bqh[i] = pack_h8(xh); bql[i] = pack_h8(xl);
        bqh[i + 4] = pack_h8(yh); bql[i + 4] = pack_h8(yl);
      }
    }
    const int nblk = min(U, (len - 32 * gb0 + 31) >> 5);
    u4 kcn = u4{0, 0, 0, 0}, vcn = u4{0, 0, 0, 0};
    {
      const int row = 32 * gb0 + tl;
      if (row < len) {
        kcn = *(const u4*)(a.kc + (seq_row0 + row) * a.W + 4 * hk);
        vcn = *(const u4*)(a.vc + (seq_row0 + row) * a.W + 4 * hk);
      }
    }
    for (int u = 0; u < nblk; ++u) {
      const u4 kcw = kcn, vcw = vcn;
      {
        const int row = 32 * (gb0 + u + 1) + tl;
        const bool nx = u + 1 < nblk && row < len;
        kcn = nx ? *(const u4*)(a.kc + (seq_row0 + row) * a.W + 4 * hk) : u4{0, 0, 0, 0};
        vcn = nx ? *(const u4*)(a.vc + (seq_row0 + row) * a.W + 4 * hk) : u4{0, 0, 0, 0};
      }
      // value codes of the block, by subspace: vcs[g][t]; lane half hh
      // writes subspaces 8 hh .. 8 hh + 7 of its token
#pragma unroll
      for (int e = 0; e < 8; ++e)
        vcs[(8 * hh + e) * AT_BLK + tl] = (unsigned char)(vcw[2 * hh + (e >> 2)] >> (8 * (e & 3)));

      // ---- scores: pair (i, i + 4) of k-steps holds elements jd and jd + 64;
      // R_t, then hi + lo float16 pairs; scores = khi.qhi + khi.qlo + klo.qhi
      f16v acc = {};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int cx = (kcw[hh] >> (8 * i)) & 255, cy = (kcw[2 + hh] >> (8 * i)) & 255;
        const h8 x = as_h8(*(const u4*)(ktab + ((4 * hh + i) * AT_K + cx) * 8));
        const h8 y = as_h8(*(const u4*)(ktab + ((8 + 4 * hh + i) * AT_K + cy) * 8));
        _Float16 xh[8], xl[8], yh[8], yl[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xf = (float)x[e], yf = (float)y[e];
          const float c = ct[8 * i + e], s = st[8 * i + e];
          split16(xf * c - yf * s, xh[e], xl[e]);
          split16(xf * s + yf * c, yh[e], yl[e]);
        }
        const h8 kxh = as_h8(pack_h8(xh)), kxl = as_h8(pack_h8(xl));
        const h8 kyh = as_h8(pack_h8(yh)), kyl = as_h8(pack_h8(yl));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kxl, as_h8(bqh[i]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kxh, as_h8(bql[i]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kxh, as_h8(bqh[i]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kyl, as_h8(bqh[i + 4]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kyh, as_h8(bql[i + 4]), acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(kyh, as_h8(bqh[i + 4]), acc, 0, 0, 0);
      }

      // ---- softmax weights of this block (only the columns of variant u)
      // register v holds token row t = 8 (v / 4) + 4 hh + v % 4
      const int rowb = 32 * (gb0 + u);
      float sc[16];
      float ml = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int t = 8 * (v >> 2) + 4 * hh + (v & 3);
        sc[v] = (ul == u && rowb + t < len) ? acc[v] * a.qscale : -INFINITY;
        ml = fmaxf(ml, sc[v]);
      }
      ml = fmaxf(ml, __shfl_xor(ml, 32));
#pragma unroll
      for (int h = 0; h < GQ; ++h) {
        const float mb = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ml), u * GQ + h));
        if (mb > mw[h]) {                            // uniform
          const float nref = mb + AT_HEADROOM;
          if (mw[h] > -INFINITY) {
            const float fac = exp2f(mw[h] - nref);
            if (hl == h) lsum *= fac;
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
              for (int v = 0; v < 16; ++v)
                if ((v & 3) % GQ == h) o[c][v] *= fac;
          }
          mw[h] = nref;
        }
      }
      float mine = mw[0];
#pragma unroll
      for (int h = 1; h < GQ; ++h) mine = hl == h ? mw[h] : mine;
      u4 ph[2], pl[2];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        _Float16 xh[8], xl[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sv = sc[8 * s2 + e];
          const float pv = sv == -INFINITY ? 0.f : exp2f(sv - mine + AT_PSHIFT);
          lsum += pv;
          split16(pv, xh[e], xl[e]);
        }
        ph[s2] = pack_h8(xh);
        pl[s2] = pack_h8(xl);
      }

      // ---- value sums: o[c] += P . V, V gathered in the k order of P
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int g = 4 * c + (tl >> 3), e = tl & 7;
        const unsigned char* cp = vcs + g * AT_BLK + 4 * hh;
        const _Float16* vt = vtab + g * AT_K * 8 + e;
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const uint32_t c0 = *(const uint32_t*)(cp + 16 * s2);
          const uint32_t c1 = *(const uint32_t*)(cp + 16 * s2 + 8);
          _Float16 vv[8];
#pragma unroll
          for (int e2 = 0; e2 < 4; ++e2) {
            vv[e2] = vt[((c0 >> (8 * e2)) & 255) * 8];
            vv[4 + e2] = vt[((c1 >> (8 * e2)) & 255) * 8];
          }
          const h8 vb = as_h8(pack_h8(vv));
          o[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(pl[s2]), vb, o[c], 0, 0, 0);
          o[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(ph[s2]), vb, o[c], 0, 0, 0);
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }

  // ---- merge the four waves: per head the reference, the sum and o
  float* rw = red + w * AT_RED;
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
  for (int i = tid; i < GQ * AT_HD; i += AT_THREADS) {
    const int h = i / AT_HD, n = i % AT_HD;
    float M = -INFINITY;
#pragma unroll
    for (int v = 0; v < AT_WAVES; ++v)
      if (red[v * AT_RED + 4 + h] > 0.f) M = fmaxf(M, red[v * AT_RED + h]);
    double num = 0.0, den = 0.0;
#pragma unroll
    for (int v = 0; v < AT_WAVES; ++v) {
      const float* r = red + v * AT_RED;
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
// / sum_c 2^(m_c - M) l_c over the chunks holding tokens.
__global__ void __launch_bounds__(AT_HD) attn_merge_kernel(const float* __restrict__ part, int Hq,
                                                          int Hkv, int nch,
                                                          float* __restrict__ out) {
  const int bq = blockIdx.x, b = bq / Hq, hq = bq % Hq;
  const int GQ = Hq / Hkv, hk = hq / GQ, h = hq % GQ, n = threadIdx.x;
  const float* p = part + (((size_t)b * Hkv + hk) * nch * GQ + h) * AT_PART;
  const size_t cs = (size_t)GQ * AT_PART;
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c)
    if (p[c * cs + AT_HD + 1] > 0.f) M = fmaxf(M, p[c * cs + AT_HD]);
  double num = 0.0, den = 0.0;
  for (int c = 0; c < nch; ++c) {
    const float l = p[c * cs + AT_HD + 1];
    if (!(l > 0.f)) continue;
    const double f = exp2((double)p[c * cs + AT_HD] - (double)M);
    num += f * (double)p[c * cs + n];
    den += f * (double)l;
  }
  out[(size_t)bq * AT_HD + n] = den > 0.0 ? (float)(num / den) : 0.f;
}

struct AttnPlan {
  int GQ, rpc, nch;
  size_t off_t1, off_t2, off_th, off_part, bytes;
};

int at_round(int GQ) { return AT_WAVES * (32 / GQ) * AT_BLK; }

gsrq_status attn_plan(const gsrq_attn_shape* a, AttnPlan& p) {
  if (!a) return GSRQ_E_ARG;
  if (a->B < 1 || a->cap < 1 || a->Hkv < 1 || a->Hq < 1 || a->head_dim < 1) return GSRQ_E_ARG;
  if (a->Hq % a->Hkv) return GSRQ_E_ARG;
  if (!(a->rope_base > 0.f) || !(a->rope_base < INFINITY)) return GSRQ_E_ARG;
  if (!(a->scale > 0.f) || !(a->scale < INFINITY)) return GSRQ_E_ARG;
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
  p.off_t1 = 0;
  p.off_t2 = align256(32 * 64 * sizeof(float2));
  p.off_th = p.off_t2 + align256(32 * 64 * sizeof(float2));
  p.off_part = p.off_th + align256(64 * sizeof(double));
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
  attn_chunk_kernel<GQ><<<dim3(args.nch, Hkv, B), AT_THREADS, AtCfg<GQ>::BYTES, st>>>(args);
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

gsrq_status gsrq_attn_decode(const gsrq_attn_shape* a, const gsrq_shape* kv,
                             const uint32_t* k_codes, const uint32_t* v_codes,
                             const int32_t* seq_len, const float* k_gain, const float* k_shape,
                             const float* v_gain, const float* v_shape, const void* q,
                             gsrq_dtype q_dtype, float* out, void* workspace, size_t ws_bytes,
                             void* stream) {
  AttnPlan p;
  gsrq_status e = attn_plan(a, p);
  if (e) return e;
  if (!kv || kv->N < 1 || kv->D < 1 || kv->d < 1 || kv->K < 2 || kv->M < 1) return GSRQ_E_ARG;
  if (kv->D != a->Hkv * a->head_dim) return GSRQ_E_ARG;
  if (kv->D % kv->d || !is_pow2(kv->K)) return GSRQ_E_ARG;
  if (kv->d != 8 || kv->K != AT_K || kv->M != 1) return GSRQ_E_UNSUPPORTED;
  if (kv->N < (int64_t)a->B * a->cap) return GSRQ_E_ARG;
  if (!k_codes || !v_codes || !seq_len || !k_gain || !k_shape || !v_gain || !v_shape || !q ||
      !out)
    return GSRQ_E_ARG;
  if ((uintptr_t)k_codes % 16 || (uintptr_t)v_codes % 16 || (uintptr_t)k_shape % 16 ||
      (uintptr_t)q % 16)
    return GSRQ_E_ARG;
  if (q_dtype != GSRQ_F32 && q_dtype != GSRQ_F16) return GSRQ_E_ARG;
  if (!workspace || (uintptr_t)workspace % 256) return GSRQ_E_ARG;
  if (ws_bytes < p.bytes) return GSRQ_E_WORKSPACE;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  AttnArgs args;
  args.kc = k_codes;
  args.vc = v_codes;
  args.seq_len = seq_len;
  args.kg = k_gain;
  args.ks = k_shape;
  args.vg = v_gain;
  args.vs = v_shape;
  args.q = q;
  args.q_f16 = q_dtype == GSRQ_F16;
  args.t1 = (const float2*)(ws + p.off_t1);
  args.t2 = (const float2*)(ws + p.off_t2);
  args.th = (const double*)(ws + p.off_th);
  args.part = (float*)(ws + p.off_part);
  args.cap = a->cap;
  args.W = a->Hkv * 4;
  args.Hkv = a->Hkv;
  args.nch = p.nch;
  args.rpc = p.rpc;
  args.qscale = (float)((double)a->scale * 1.4426950408889634);
  attn_tables_kernel<<<8, 256, 0, st>>>((double)a->rope_base, (float2*)(ws + p.off_t1),
                                        (float2*)(ws + p.off_t2), (double*)(ws + p.off_th));
  e = launch_ok();
  if (e) return e;
  if (p.GQ == 1) e = attn_launch<1>(args, a->B, a->Hkv, st);
  else if (p.GQ == 2) e = attn_launch<2>(args, a->B, a->Hkv, st);
  else e = attn_launch<4>(args, a->B, a->Hkv, st);
  if (e) return e;
  attn_merge_kernel<<<a->B * a->Hq, AT_HD, 0, st>>>(args.part, a->Hq, a->Hkv, p.nch, out);
  return launch_ok();
}

}  // extern "C"
