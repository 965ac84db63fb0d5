// One decoding step of attention over a GSRQ-coded KV cache on AMD MI355X
// (gfx950): the codes are unpacked, the keys dequantised and rotated by
// RoPE, and softmax attention is taken, without an intermediate float16
// K/V tensor (arXiv 2607.01065, Appendix C, decoding latency analysis).
// Shapes: d = 8 subvectors, K = 256 codewords, one stage (the 1-bit cache),
// 128-element heads (16 subspaces per head), grouped-query attention with
// GQ = Hq / Hkv in {1, 2, 4}.
//
// One workgroup owns (sequence, key/value head, chunk of tokens) and runs
// rounds of 4096 / GQ tokens:
//  * Scores on the matrix cores.  A wave takes U = 32 / GQ blocks of 32
//    tokens.  The A operand of a v_mfma_f32_32x32x16_f16 holds 32 tokens'
//    keys (each lane one 8-element codeword gathered from a float16 table of
//    the head's 16 codebooks in LDS, rotated in float32); the B operand's 32
//    columns are the GQ query heads of the U blocks.  Both sides enter as
//    hi + lo float16 pairs (three products per k-step), so scores carry
//    about 22 bits, as a float32 dot product would.  RoPE enters as a relative rotation:
//    score(i) = (R_{pq - 32b} q) . (R_t k_i) for token i = 32 b + t, so the
//    rotation of a key depends only on its row t in the block (fixed per
//    lane) and that of the query on the block (one sine/cosine per lane per
//    wave group).
//  * Softmax weights in float32 with a workgroup-wide reference maximum per
//    query head (raised, and the partial sums rescaled, when a round's
//    scores exceed it).
//  * Values without dequantisation.  The softmax weight p of token i is
//    added to a per-head table H[g][k] at the token's value code k of every
//    subspace g (float32 LDS atomics); at the end of the chunk the output
//    is H times the value codebook, o[8g + e] = sum_k H[g][k] c_g,k[e].
//  * A second kernel merges the chunks of every (sequence, query head) with
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
constexpr int AT_HSTRIDE = AT_SUB * AT_K;   // floats of one head's value table

template <int GQ> struct AtCfg {
  static constexpr int U = 32 / GQ;                         // blocks per wave group
  static constexpr int ROUND = AT_WAVES * U * AT_BLK;       // tokens per round
  static constexpr int TOK_PT = ROUND / AT_THREADS;         // tokens per thread when summing
  // LDS layout in bytes
  static constexpr int KTAB = 0;                                      // f16 [16][256][8]
  static constexpr int HIST = KTAB + AT_SUB * AT_K * 8 * 2;           // f32 [GQ][16][256]
  static constexpr int STAGE = HIST + GQ * AT_HSTRIDE * 4;            // f32 [WAVES*U][GQ][32]
  static constexpr int ANG = STAGE + AT_WAVES * U * GQ * AT_BLK * 4;  // float2 [WAVES][64]
  static constexpr int RED = ANG + AT_WAVES * 64 * 8;                 // f32 [2][WAVES][4]
  static constexpr int BYTES = RED + 2 * AT_WAVES * 4 * 4;
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

__device__ __forceinline__ float wave_max_keep(float v, int keep_mask) {
  // max over the lanes that differ from this one only in bits outside keep_mask
#pragma unroll
  for (int off = 1; off < 64; off <<= 1)
    if (!(off & keep_mask)) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

template <int GQ>
__global__ void __launch_bounds__(AT_THREADS, 1) attn_chunk_kernel(AttnArgs a) {
  using C = AtCfg<GQ>;
  constexpr int U = C::U;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  _Float16* ktab = (_Float16*)(lds + C::KTAB);
  float* hist = (float*)(lds + C::HIST);
  float* stage = (float*)(lds + C::STAGE);
  float2* ang = (float2*)(lds + C::ANG);
  float* red = (float*)(lds + C::RED);

  const int chunk = blockIdx.x, hk = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int tl = lane & 31, hh = lane >> 5;
  const int ul = tl / GQ, hl = tl % GQ;      // B-operand column: block variant, query head
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
  const int Hq = a.Hkv * GQ;
  const int g0 = hk * AT_SUB;
  const size_t seq_row0 = (size_t)b * a.cap;

  // key codeword table: fp16(fp32(g * s)), the float16 decode of a codeword
  for (int i = tid; i < AT_SUB * AT_K * 2; i += AT_THREADS) {
    const int cw = i >> 1, half = i & 1;
    const float gk = a.kg[(size_t)g0 * AT_K + cw];
    const f4 s = *(const f4*)(a.ks + ((size_t)g0 * AT_K + cw) * 8 + half * 4);
    uint2 v;
    v.x = pack2((_Float16)(gk * s[0]), (_Float16)(gk * s[1]));
    v.y = pack2((_Float16)(gk * s[2]), (_Float16)(gk * s[3]));
    *(uint2*)(ktab + cw * 8 + half * 4) = v;
  }
  for (int i = tid; i < GQ * AT_HSTRIDE / 4; i += AT_THREADS) ((f4*)hist)[i] = f4{0.f, 0.f, 0.f, 0.f};

  // lane constants: R_t for the lane's token row, and the query of its
  // column turned by R_{-32u}; element m < 32 of a lane is head element
  // jd = 32 hh + m, paired with jd + 64
  float ct[32], st[32], qx[32], qy[32];
  {
    const float4* t1 = (const float4*)(a.t1 + tl * 64 + 32 * hh);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const float4 v = t1[m];
      ct[2 * m] = v.x; st[2 * m] = v.y; ct[2 * m + 1] = v.z; st[2 * m + 1] = v.w;
    }
    const size_t qoff = ((size_t)b * Hq + hk * GQ + hl) * AT_HD + 32 * hh;
    if (a.q_f16) {
      const u4* qp = (const u4*)((const _Float16*)a.q + qoff);
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const h8 x = as_h8(qp[m]), y = as_h8(qp[m + 8]);
#pragma unroll
        for (int e = 0; e < 8; ++e) { qx[8 * m + e] = (float)x[e]; qy[8 * m + e] = (float)y[e]; }
      }
    } else {
      const f4* qp = (const f4*)((const float*)a.q + qoff);
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        const f4 x = qp[m], y = qp[m + 16];
#pragma unroll
        for (int e = 0; e < 4; ++e) { qx[4 * m + e] = x[e]; qy[4 * m + e] = y[e]; }
      }
    }
    const float4* t2 = (const float4*)(a.t2 + ul * 64 + 32 * hh);
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const float4 v = t2[m];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const float c = r ? v.z : v.x, s = r ? v.w : v.y;
        const float x = qx[2 * m + r], y = qy[2 * m + r];
        qx[2 * m + r] = x * c + y * s;       // R_{-32u}: angle -32 u theta
        qy[2 * m + r] = y * c - x * s;
      }
    }
  }
  const double thl = a.th[lane];
  float mref[GQ], lsum[GQ];
#pragma unroll
  for (int h = 0; h < GQ; ++h) { mref[h] = -INFINITY; lsum[h] = 0.f; }
  __syncthreads();

  for (int r = 0; r < a.rpc; ++r) {
    const int rt0 = tok0 + r * C::ROUND;
    if (rt0 >= len) break;
    // value codes of the tokens this thread sums, fetched before the scores
    u4 vcode[C::TOK_PT];
#pragma unroll
    for (int k = 0; k < C::TOK_PT; ++k) {
      const int tok = rt0 + tid + k * AT_THREADS;
      vcode[k] = tok < len ? *(const u4*)(a.vc + (seq_row0 + tok) * a.W + 4 * hk) : u4{0, 0, 0, 0};
    }

    // ---- scores of this wave's U blocks
    const int gb0 = (rt0 >> 5) + w * U;
    if (32 * gb0 < len) {
      {
        const int n = (len - 1) - 32 * gb0;           // query-side angle in positions, >= 0
        double rev = (double)n * thl;
        rev -= floor(rev);
        float s, c;
        sincosf((float)(rev * (2.0 * M_PI)), &s, &c);
        ang[w * 64 + lane] = make_float2(c, s);
      }
      __builtin_amdgcn_wave_barrier();
      // rotated query of every column, split hi + lo into float16 pairs
      u4 bqh[8], bql[8];
      {
        const float4* ap = (const float4*)(ang + w * 64 + 32 * hh);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          _Float16 xh[8], xl[8], yh[8], yl[8];
#pragma unroll
          for (int m2 = 0; m2 < 4; ++m2) {
            const float4 v = ap[4 * i + m2];
#pragma unroll
            for (int r2 = 0; r2 < 2; ++r2) {
              const int e = 2 * m2 + r2, m = 8 * i + e;
              const float c = r2 ? v.z : v.x, s = r2 ? v.w : v.y;
              split16(qx[m] * c - qy[m] * s, xh[e], xl[e]);
              split16(qx[m] * s + qy[m] * c, yh[e], yl[e]);
            }
          }
          bqh[i] = pack_h8(xh); bql[i] = pack_h8(xl);
          bqh[i + 4] = pack_h8(yh); bql[i + 4] = pack_h8(yl);
        }
      }
      const int nblk = min(U, (len - 32 * gb0 + 31) >> 5);
      u4 kcn = u4{0, 0, 0, 0};
      {
        const int row = 32 * gb0 + tl;
        if (row < len) kcn = *(const u4*)(a.kc + (seq_row0 + row) * a.W + 4 * hk);
      }
      for (int u = 0; u < nblk; ++u) {
        const u4 kcw = kcn;
        {
          const int row = 32 * (gb0 + u + 1) + tl;
          kcn = (u + 1 < nblk && row < len) ? *(const u4*)(a.kc + (seq_row0 + row) * a.W + 4 * hk)
                                             : u4{0, 0, 0, 0};
        }
        u4 ak[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t word = i < 4 ? kcw[hh] : kcw[2 + hh];
          const int code = (word >> (8 * (i & 3))) & 255;
          const int sub = i < 4 ? 4 * hh + i : 8 + 4 * hh + (i - 4);
          ak[i] = *(const u4*)(ktab + (sub * AT_K + code) * 8);
        }
        // R_t, then hi + lo float16 pairs; scores = khi.qhi + khi.qlo + klo.qhi
        u4 akl[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const h8 x = as_h8(ak[i]), y = as_h8(ak[i + 4]);
          _Float16 xh[8], xl[8], yh[8], yl[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float xf = (float)x[e], yf = (float)y[e];
            const float c = ct[8 * i + e], s = st[8 * i + e];
            split16(xf * c - yf * s, xh[e], xl[e]);
            split16(xf * s + yf * c, yh[e], yl[e]);
          }
          ak[i] = pack_h8(xh); akl[i] = pack_h8(xl);
          ak[i + 4] = pack_h8(yh); akl[i + 4] = pack_h8(yl);
        }
        f16v acc = {};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(akl[i]), as_h8(bqh[i]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(ak[i]), as_h8(bql[i]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_h8(ak[i]), as_h8(bqh[i]), acc, 0, 0, 0);
        }
        if (ul == u) {
          float* sp = stage + ((w * U + u) * GQ + hl) * AT_BLK + 4 * hh;
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4)
            *(f4*)(sp + 8 * q4) = f4{acc[4 * q4] * a.qscale, acc[4 * q4 + 1] * a.qscale,
                                     acc[4 * q4 + 2] * a.qscale, acc[4 * q4 + 3] * a.qscale};
        }
      }
    }
    __syncthreads();

    // ---- round maximum per query head; raise the reference if exceeded
    {
      const int run = tid >> 1, h = run % GQ, blk = run / GQ;
      const int qi0 = blk * AT_BLK + (tid & 1) * 16;
      const f4* sp = (const f4*)(stage + run * AT_BLK + (tid & 1) * 16);
      float m = -INFINITY;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const f4 x = sp[v];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (rt0 + qi0 + 4 * v + e < len) m = fmaxf(m, x[e]);
      }
      m = wave_max_keep(m, 2 * (GQ - 1));
      if (lane < 2 * GQ && !(lane & 1)) red[w * 4 + (lane >> 1)] = m;
      (void)h;
    }
    __syncthreads();
    bool rescale = false;
    float fac[GQ];
#pragma unroll
    for (int h = 0; h < GQ; ++h) {
      float m = red[h];
#pragma unroll
      for (int v = 1; v < AT_WAVES; ++v) m = fmaxf(m, red[v * 4 + h]);
      fac[h] = 1.f;
      if (m > mref[h]) {
        const float nref = m + AT_HEADROOM;
        if (mref[h] > -INFINITY) {
          fac[h] = exp2f(mref[h] - nref);
          rescale = true;
        }
        mref[h] = nref;
      }
    }
    if (rescale) {
#pragma unroll
      for (int h = 0; h < GQ; ++h) {
        if (fac[h] == 1.f) continue;
        lsum[h] *= fac[h];
        f4* hp = (f4*)(hist + h * AT_HSTRIDE) + tid * (AT_HSTRIDE / 4 / AT_THREADS);
#pragma unroll
        for (int v = 0; v < AT_HSTRIDE / 4 / AT_THREADS; ++v) hp[v] = hp[v] * fac[h];
      }
      __syncthreads();
    }

    // ---- softmax weights into the value tables
#pragma unroll
    for (int k = 0; k < C::TOK_PT; ++k) {
      const int qi = tid + k * AT_THREADS;
      if (rt0 + qi >= len) continue;
      const float* sp = stage + (qi >> 5) * GQ * AT_BLK + (qi & 31);
      float p[GQ];
#pragma unroll
      for (int h = 0; h < GQ; ++h) {
        p[h] = exp2f(sp[h * AT_BLK] - mref[h]);
        lsum[h] += p[h];
      }
#pragma unroll
      for (int g = 0; g < AT_SUB; ++g) {
        const int code = (vcode[k][g >> 2] >> (8 * (g & 3))) & 255;
        float* hp = hist + g * AT_K + code;
#pragma unroll
        for (int h = 0; h < GQ; ++h)
          __hip_atomic_fetch_add(hp + h * AT_HSTRIDE, p[h], __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
    __syncthreads();
  }

  // ---- chunk result: softmax sums and o = H x value codebook
  float* lred = red + AT_WAVES * 4;
#pragma unroll
  for (int h = 0; h < GQ; ++h) {
    float v = lsum[h];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) lred[w * 4 + h] = v;
  }
  __syncthreads();
  for (int o = tid; o < GQ * AT_HD; o += AT_THREADS) {
    const int h = o / AT_HD, n = o % AT_HD, g = n >> 3, e = n & 7;
    const float* gp = a.vg + (size_t)(g0 + g) * AT_K;
    const float* sp = a.vs + (size_t)(g0 + g) * AT_K * 8 + e;
    const float* hp = hist + h * AT_HSTRIDE + g * AT_K;
    double acc = 0.0;
#pragma unroll 8
    for (int k = 0; k < AT_K; ++k) acc += (double)hp[k] * (double)(gp[k] * sp[8 * k]);
    outp[h * AT_PART + n] = (float)acc;
  }
  if (tid < GQ) {
    float l = 0.f;
#pragma unroll
    for (int v = 0; v < AT_WAVES; ++v) l += lred[v * 4 + tid];
    outp[tid * AT_PART + AT_HD] = mref[tid];
    outp[tid * AT_PART + AT_HD + 1] = l;
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
