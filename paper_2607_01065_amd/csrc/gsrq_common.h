// Private header shared by the translation units of libgsrq (subvectors of
// d <= 8 in gsrq.hip, wider subvectors in gsrq_wide.hip, per-token weights in
// gsrq_weights.hip): operand types, the
// scaling constants of the MFMA distance contraction, small device helpers
// and host-side launch plumbing.  Everything here has internal linkage except
// the launch-timing state, which every translation unit shares.
#ifndef GSRQ_COMMON_H
#define GSRQ_COMMON_H

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "gsrq.h"

// Opt-in launch timing: HIP events bracket instrumented launches on their
// own streams (gsrq_timing_enable / gsrq_timing_read).
struct GsrqTimingState {
  bool on = false;
  uint32_t kinds = 0;     // bit k: launches of kind k are recorded
  struct Rec { hipEvent_t a, b; int kind; };
  Rec* recs = nullptr;
  int n = 0, cap = 0;
};
extern GsrqTimingState g_gsrq_timing;

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int CW = 32;                    // codewords per MFMA tile (M dimension)
constexpr int RB = 32;                    // rows per block (MFMA N dimension)
constexpr float Y_EPS = 1e-8f;            // y = x / (||x|| + eps)
constexpr double SHAPE_KEEP_REL = 1e-6;   // keep s when ||sum w y|| <= 1e-6 W
constexpr float PAD_BIAS = 65504.f;       // g^2 slot of a padding codeword
constexpr int SA = 12;                    // codeword operand scale 2^SA (no subnormals)
constexpr int SB = 8;                     // float32-row operand scale 2^SB

// ------------------------------------------------------------ device helpers

__device__ __forceinline__ uint32_t pack2(_Float16 lo, _Float16 hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

__device__ __forceinline__ h8 as_h8(u4 v) { return __builtin_bit_cast(h8, v); }

__device__ __forceinline__ u4 pack_h8(const _Float16 (&v)[8]) {
  u4 r;
  r[0] = pack2(v[0], v[1]); r[1] = pack2(v[2], v[3]);
  r[2] = pack2(v[4], v[5]); r[3] = pack2(v[6], v[7]);
  return r;
}

template <typename T> __device__ __forceinline__ float to_f(T v) { return (float)v; }

__device__ __forceinline__ int wave_lane() { return threadIdx.x & 63; }

// Exponent e with 2^e >= maxg (sigma = 2^e scales a codebook's operands).
__device__ __forceinline__ int sigma_exp(float maxg) {
  if (!(maxg > 0.f)) return 0;
  int e;
  frexpf(maxg, &e);   // maxg = m 2^e, m in [0.5, 1)
  return e;
}

// Wait until this wave's LDS (and scalar memory) operations have completed:
// s_waitcnt lgkmcnt(0), leaving the vector-memory and export counters alone.
__device__ __forceinline__ void lgkm_wait_all() { __builtin_amdgcn_s_waitcnt(0xc07f); }

__device__ __forceinline__ int min3i(int a, int b, int c) {
  int r;
  asm volatile("v_min3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Bias terms of the distance contraction.  The codeword side supplies
//   [gg_h gg_l 2^SA 2^SA | gg'_h gg'_l 0 0]
// and the row side
//   [c c rr_h rr_l | c 2^-16  c 2^-16  0 0],
// whose dot product is gg c + 2^SA rr.  A gg of at least 1/8 goes to the
// plain hi/lo pair; a smaller one, scaled by 2^16, to the primed pair, so
// near-zero gains keep a hi/lo pair of normal float16 numbers (about 22
// bits) instead of float16 subnormals: their g^2 decides between codewords
// for rows far below the codebook's scale.  rr is the same for every
// codeword of a row, so its rounding cannot change the row's argmin.
constexpr float BIAS_SPLIT = 0.125f;
constexpr int BIAS_SHIFT = 16;

__device__ __forceinline__ void split_bias(float v, _Float16& h, _Float16& l, _Float16& hs,
                                           _Float16& ls) {
  const bool big = v >= BIAS_SPLIT;
  const float vb = big ? v : 0.f;
  const float vs = big ? 0.f : ldexpf(v, BIAS_SHIFT);
  h = (_Float16)vb;
  l = (_Float16)(vb - (float)h);
  hs = (_Float16)vs;
  ls = (_Float16)(vs - (float)hs);
}

// Codeword-side bias entries for gg = (g / sigma)^2 2^SA; a padding
// codeword (real = false) gets a float16-max g^2 slot.
__device__ __forceinline__ void bias_codeword_h(bool real, float gg, _Float16 (&b)[8]) {
  _Float16 h, l, hs, ls;
  split_bias(gg, h, l, hs, ls);
  b[0] = real ? h : (_Float16)PAD_BIAS;
  b[1] = real ? l : (_Float16)0.f;
  b[2] = b[3] = (_Float16)(float)(1 << SA);
  b[4] = real ? hs : (_Float16)0.f;
  b[5] = real ? ls : (_Float16)0.f;
  b[6] = b[7] = (_Float16)0.f;
}

__device__ __forceinline__ u4 bias_codeword(bool real, float gg) {
  _Float16 b[8];
  bias_codeword_h(real, gg, b);
  return pack_h8(b);
}

// Row-side bias entries for the bias scale c = 2^sr (sr in [-14, 15]) and
// the row term rr.
__device__ __forceinline__ u4 bias_row(int sr, float rr) {
  const _Float16 c = (_Float16)ldexpf(1.f, sr);
  const _Float16 cs = (_Float16)ldexpf(1.f, sr - BIAS_SHIFT);
  const _Float16 h = (_Float16)rr;
  const _Float16 l = (_Float16)(rr - (float)h);
  return (u4){pack2(c, c), pack2(h, l), pack2(cs, cs), 0u};
}

__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// --------------------------------------------------------------- host side

struct TimedLaunch {
  GsrqTimingState::Rec* rec = nullptr;
  hipStream_t st;
  TimedLaunch(int kind, hipStream_t s) : st(s) {
    GsrqTimingState& T = g_gsrq_timing;
    if (!T.on || !((T.kinds >> kind) & 1u)) return;
    if (T.n == T.cap) {
      const int nc = T.cap ? 2 * T.cap : 1024;
      auto* nr = new GsrqTimingState::Rec[nc];
      for (int i = 0; i < T.n; ++i) nr[i] = T.recs[i];
      // timing-only events: no system-scope cache writeback per record
      // (results are read after a full device synchronisation)
      for (int i = T.n; i < nc; ++i) {
        hipEventCreateWithFlags(&nr[i].a, hipEventDisableSystemFence);
        hipEventCreateWithFlags(&nr[i].b, hipEventDisableSystemFence);
      }
      delete[] T.recs;
      T.recs = nr;
      T.cap = nc;
    }
    rec = &T.recs[T.n++];
    rec->kind = kind;
    hipEventRecord(rec->a, st);
  }
  ~TimedLaunch() {
    if (rec) hipEventRecord(rec->b, st);
  }
};

inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

inline bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

inline int log2i(int64_t v) {
  int b = 0;
  while ((1ll << b) < v) ++b;
  return b;
}

inline int grid_for(int64_t work, int block) {
  int64_t b = (work + block - 1) / block;
  if (b > 65536) b = 65536;
  if (b < 1) b = 1;
  return (int)b;
}

inline gsrq_status launch_ok() {
  return hipGetLastError() == hipSuccess ? GSRQ_OK : GSRQ_E_HIP;
}

inline gsrq_status fill_u32(void* p, size_t n, uint32_t v, hipStream_t st) {
  if (n == 0) return GSRQ_OK;
  fill_u32_kernel<<<grid_for((int64_t)n, 256), 256, 0, st>>>((uint32_t*)p, n, v);
  return launch_ok();
}

}  // namespace

#endif  // GSRQ_COMMON_H
