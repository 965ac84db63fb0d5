// Private interface of the wide-subspace kernel family (gsrq_wide.hip): the
// C ABI in gsrq.hip validates arguments and hands shapes this family serves
// to the functions below.  Argument meanings are those of include/gsrq.h.
#ifndef GSRQ_WIDE_H
#define GSRQ_WIDE_H

#include <stddef.h>
#include <stdint.h>

#include "gsrq.h"

namespace gsrq_wide {

// d = 8 C with C a power of two, 8 <= d <= 256, and d > 8 or K > 256.
bool serves(const gsrq_shape* s);

size_t train_workspace_bytes(const gsrq_shape* s, size_t x_elt);
size_t encode_workspace_bytes(const gsrq_shape* s);

gsrq_status train_stage(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype, int64_t ldx,
                        const float* w, int32_t T, const int32_t* seed_rows, uint32_t flags,
                        float* gain, float* shape, float* R_next, uint16_t* assign_io,
                        int32_t* iters_run, double* obj_trace, void* workspace, void* stream);

gsrq_status encode(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype, int64_t ldx,
                   const float* gain, const float* shape, uint32_t* codes, float* residual,
                   void* workspace, void* stream);

gsrq_status decode(const gsrq_shape* s, const uint32_t* codes, int32_t M_use, const float* gain,
                   const float* shape, void* Xhat, gsrq_dtype out_dtype, int64_t ldo,
                   void* stream);

}  // namespace gsrq_wide

#endif  // GSRQ_WIDE_H
