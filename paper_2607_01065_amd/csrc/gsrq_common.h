// Private header shared by the two kernel families of libgsrq (subvectors of
// d <= 8 in gsrq.hip, wider subvectors in gsrq_wide.hip): operand types, the
// scaling constants of the MFMA distance contraction, small device helpers
// and host-side launch plumbing.  Everything here has internal linkage except
// the launch-timing state, which both translation units share.
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

__device__ __forceinline__ int min3i(int a, int b, int c) {
  int r;
  asm volatile("v_min3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
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
    if (!T.on) return;
    if (T.n == T.cap) {
      const int nc = T.cap ? 2 * T.cap : 1024;
      auto* nr = new GsrqTimingState::Rec[nc];
      for (int i = 0; i < T.n; ++i) nr[i] = T.recs[i];
      for (int i = T.n; i < nc; ++i) {
        hipEventCreate(&nr[i].a);
        hipEventCreate(&nr[i].b);
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
