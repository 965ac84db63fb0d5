/*
 * gsrq.h -- C ABI of the GSRQ hot path on AMD MI355X (gfx950).
 *
 * Gain-Shape Residual Quantization (arXiv 2607.01065): every row x of a
 * [N][D] matrix (one token's K or V vector, heads concatenated) is split into
 * G = D/d subvectors of d elements (product quantisation, Sec. 3); subvector
 * g of stage m is coded by the index k of one codeword c = gain[m][g][k] *
 * shape[m][g][k][:] of a gain-shape codebook (Sec. 5.2, eq. 3), chosen by
 * k = argmax_k 2 g_k r.s_k - g_k^2 (eq. 5) on the stage's residual r, which
 * is then reduced by c (residual quantisation, Sec. 3 / 5.1).  Codebooks are
 * learnt with weighted gain-shape K-means (Algorithm 1, eqs. 5-8, Sec. 5.3).
 *
 * Conventions shared by every entry point
 *  - Every array argument is DEVICE memory owned by the caller, except the
 *    seed-row table of gsrq_train_stage, which is host memory.  The library
 *    allocates nothing; scratch space is the caller's workspace.
 *  - Calls are ordered on the given HIP stream (NULL = the null stream) and
 *    return once the work is enqueued.  Synchronise the stream before reading
 *    any output on the host.
 *  - Errors are return codes.  Arguments are validated on the host before any
 *    HIP call; on a validation error no output is touched.  GSRQ_E_HIP means a
 *    launch or copy failed after validation (outputs are then undefined).
 *  - Codebook layouts: gain [M][G][K] float32 (g >= 0), shape [M][G][K][d]
 *    float32 (unit rows), row-major and dense.
 *  - Code layout (bit-packed): row i owns gsrq_code_words() uint32 words; the
 *    code of stage m, subspace g is the b = log2 K bit field starting at bit
 *    t*b, t = m*G + g, of the row's bit string, least significant bit first
 *    (bit p is bit p%32 of word p/32).
 *  - Supported on this build: 1 <= d <= 8 with 2 <= K <= 256, and
 *    d in {8, 16, 32, 64, 128, 256} with any power-of-two 2 <= K <= 65536.
 *    Other valid shapes return GSRQ_E_UNSUPPORTED.
 *  - Apart from the opt-in launch timing at the end of this header, the
 *    library keeps no state between calls; calls on different streams with
 *    disjoint buffers may run concurrently.
 */
#ifndef GSRQ_H
#define GSRQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GSRQ_OK = 0,
  GSRQ_E_ARG = 1,          /* invalid argument (null pointer, size, flag)  */
  GSRQ_E_UNSUPPORTED = 2,  /* valid problem this build does not implement  */
  GSRQ_E_WORKSPACE = 3,    /* workspace too small                          */
  GSRQ_E_HIP = 4           /* a HIP runtime call failed                    */
} gsrq_status;

typedef enum { GSRQ_F32 = 0, GSRQ_F16 = 1 } gsrq_dtype;

/* Problem shape.  N rows of D elements, subvector dimension d (d divides D,
 * G = D/d subspaces), K codewords per codebook (power of two), M stages. */
typedef struct {
  int64_t N;
  int32_t D;
  int32_t d;
  int32_t K;
  int32_t M;
} gsrq_shape;

/* Flags of gsrq_train_stage. */
enum {
  /* Start from the codebook already in gain/shape instead of seeding from
   * rows (resume; seed_rows is then ignored and may be NULL). */
  GSRQ_RESUME = 1u,
  /* With GSRQ_RESUME: assign_io holds the assignment the previous iteration
   * produced, so the stop test of the first iteration compares against it.
   * Without this flag a resumed first iteration always counts as changed. */
  GSRQ_ASSIGN_IN = 2u,
  /* Run all T iterations even when an assignment repeats. */
  GSRQ_NO_EARLY_STOP = 4u,
  /* Standard weighted K-means, the baseline GSKM replaces (Sec. 4, Sec. 6.1),
   * with the same kernels: centroid k is held as gain = ||c_k|| and
   * shape = c_k / ||c_k|| (shape 0 for a zero centroid), so scoring by eq. (5)
   * is the squared distance to c_k.  Seeding (without GSRQ_RESUME): c_k = the
   * seed row itself (a zero row is allowed); there is no initial assignment
   * (assign_io is not written), T = 0 only writes the seed centroids, and
   * the first iteration counts as changed.  Iteration t: assign to the
   * nearest centroid (ties to the lowest index), then c_k = weighted mean of
   * its members for clusters with weight (others keep c_k); obj_trace entry
   * t-1 is the weighted distortion AFTER that update.  GSRQ_RESUME,
   * GSRQ_ASSIGN_IN and the stop rule act as for GSKM. */
  GSRQ_KMEANS = 8u,
  /* Check the inputs on the device before any other work and return
   * GSRQ_E_ARG, with no output touched, when a weight is negative or not
   * finite, an element of X is not finite, or (GSKM seeding: without
   * GSRQ_RESUME and GSRQ_KMEANS) a seed row's subvector is zero, which has
   * no direction to start a shape from (Alg. 1 draws the initial shapes on
   * the unit sphere).  The check reads X once and the call then waits for
   * the stream (it is synchronous, unlike the unchecked call).  Without the
   * flag these inputs are the caller's to avoid: a zero seed subvector gives
   * a zero initial shape. */
  GSRQ_CHECK_INPUTS = 16u
};

/* Human-readable name of a status code (static string). */
const char* gsrq_status_string(gsrq_status st);

/* uint32 words per row of packed codes: ceil(M * G * log2(K) / 32).
 * Returns 0 for an invalid shape. */
size_t gsrq_code_words(const gsrq_shape* s);

/* Average bits per element, M * log2(K) / d (Sec. 6.2); 0 if invalid. */
double gsrq_bits_per_element(const gsrq_shape* s);

/* Workspace bytes gsrq_train_stage needs for shape s (s->M is ignored).
 * Writes the size to *bytes.  GSRQ_E_ARG / GSRQ_E_UNSUPPORTED as above. */
gsrq_status gsrq_train_workspace_bytes(const gsrq_shape* s, size_t* bytes);

/* Workspace bytes gsrq_encode needs for shape s. */
gsrq_status gsrq_encode_workspace_bytes(const gsrq_shape* s, size_t* bytes);

/*
 * gsrq_train_stage -- learn ONE stage's G codebooks with weighted GSKM
 * (Algorithm 1 with the weighted means of Sec. 5.1 / 5.3), then optionally
 * re-encode the stage input with the learnt codebook to give the next
 * stage's residual (Sec. 5.1).  s->M is ignored.
 *
 *  X, x_dtype, ldx   stage input, [N][ldx] row-major (ldx >= D elements):
 *                    the data for stage 0, the residual for later stages.
 *  w                 [N] float32 per-row weights >= 0, shared by every
 *                    subspace; NULL means all ones.  A cluster whose members
 *                    carry zero total weight counts as empty.
 *  T                 maximum iterations, >= 0; T = 0 (not with GSRQ_RESUME)
 *                    only initialises: gain/shape receive the initial
 *                    codebook and assign_io the initial assignment.
 *  seed_rows         HOST [G][K] int32 row indices; codebook k of subspace g
 *                    is seeded with the direction of row seed_rows[g][k],
 *                    which must be a nonzero subvector.  Indices must lie in
 *                    [0, N) and be distinct within a subspace; N >= K.
 *  flags             GSRQ_RESUME | GSRQ_ASSIGN_IN | GSRQ_NO_EARLY_STOP |
 *                    GSRQ_KMEANS (the K-means baseline, see the flag) |
 *                    GSRQ_CHECK_INPUTS (device check of w, X and the seeds).
 *  gain, shape       [G][K], [G][K][d] float32 outputs (inputs on resume).
 *  R_next            [N][D] float32 residual X - c(encode(X)) with the final
 *                    codebook, or NULL.
 *  assign_io         [G][N] uint16 final assignment (input too with
 *                    GSRQ_ASSIGN_IN), or NULL.
 *  iters_run         [G] int32 iterations run per subspace, or NULL.
 *  obj_trace         [G][T] float64: entry t-1 is sum_i w_i ||x_i - c_{k_i}||^2
 *                    of iteration t's assignment against the codebook it was
 *                    made with (GSRQ_KMEANS: against the updated centroids);
 *                    entries past iters_run are 0.  Or NULL.
 *  workspace         >= gsrq_train_workspace_bytes(s), 256-byte aligned.
 *
 * Initialisation (without GSRQ_RESUME): shapes are the normalised seed rows;
 * rows are assigned to the shape of largest projection, and each gain is the
 * clamped weighted mean projection of its members (eq. 8), or the seed row's
 * norm for a cluster without weight.  Iteration t: assign by eq. (5) (ties
 * to the lowest index), then for clusters with weight: shape = normalised
 * weighted sum of y_i = x_i / (||x_i|| + 1e-8) (eqs. 6, 7), kept if that sum
 * is below 1e-6 times the cluster weight; gain = max(0, weighted mean of
 * x_i . s_k) (eq. 8).  A subspace stops after the iteration whose
 * assignment equals the previous one (unless GSRQ_NO_EARLY_STOP).
 */
gsrq_status gsrq_train_stage(const gsrq_shape* s,
                             const void* X, gsrq_dtype x_dtype, int64_t ldx,
                             const float* w, int32_t T,
                             const int32_t* seed_rows, uint32_t flags,
                             float* gain, float* shape,
                             float* R_next, uint16_t* assign_io,
                             int32_t* iters_run, double* obj_trace,
                             void* workspace, size_t ws_bytes, void* stream);

/*
 * gsrq_encode -- stage-fused GSRQ encoding (Sec. 3, Sec. 5.1): for every
 * subspace g and stage m = 0..M-1 in order, k = argmax_k 2 g_k r.s_k - g_k^2
 * (eq. 5, ties to the lowest index) on the residual r (initially the row's
 * subvector), then r <- r - gain[m][g][k] shape[m][g][k].
 *
 *  X, x_dtype, ldx   [N][ldx] input rows (ldx >= D).
 *  gain, shape       [M][G][K], [M][G][K][d].
 *  codes             [N][gsrq_code_words(s)] uint32, packed as above.
 *  residual          [N][D] float32 final residual, or NULL.
 *  workspace         >= gsrq_encode_workspace_bytes(s), 256-byte aligned.
 * Indices agree with a float64 evaluation of eq. (5) whenever the best and
 * second-best scores differ by more than 1e-4 * ||r||^2.
 */
gsrq_status gsrq_encode(const gsrq_shape* s,
                        const void* X, gsrq_dtype x_dtype, int64_t ldx,
                        const float* gain, const float* shape,
                        uint32_t* codes, float* residual,
                        void* workspace, size_t ws_bytes, void* stream);

/*
 * Prepared codebooks: encoding a few rows at a time (the tokens appended at
 * every step of autoregressive decoding, which the paper's fused kernel
 * quantises and bit-packs as they are generated, Appendix C) is bound by
 * the per-call preparation of the codebook's MFMA operand tables.  A
 * prepared codebook holds those tables, built once, with a copy of the
 * codebook itself, in one caller-owned device buffer; gsrq_encode_prepared
 * then encodes without rebuilding them.  The narrow family only (d <= 8,
 * K <= 256; other shapes GSRQ_E_UNSUPPORTED).
 *
 * gsrq_prepared_bytes -- bytes of a prepared codebook for shape s (all M
 * stages, G codebooks each).
 */
gsrq_status gsrq_prepared_bytes(const gsrq_shape* s, size_t* bytes);

/*
 * gsrq_encode_prepare -- build the prepared codebook of gain [M][G][K],
 * shape [M][G][K][d] into `prepared` (>= gsrq_prepared_bytes(s) bytes,
 * 256-byte aligned).  The codebook is copied: later changes to gain/shape
 * need a new prepare.  A header records M, G, d and K.
 */
gsrq_status gsrq_encode_prepare(const gsrq_shape* s, const float* gain, const float* shape,
                                void* prepared, size_t bytes, void* stream);

/*
 * gsrq_encode_prepared -- gsrq_encode (same codes, residual and index
 * agreement, bit for bit) with the tables and codebook of a prepared
 * codebook; no workspace.  M <= 8 stages.  Up to 256 rows it runs a
 * latency kernel (one wave per 32-row block and subspace, nothing shared,
 * every load of a stage issued together); above that the stage-fused
 * encoder.  The kernel checks the header against s: a buffer not prepared
 * for this shape (or not prepared at all) gives code fields of all ones
 * and a NaN residual instead of plausible codes.
 */
gsrq_status gsrq_encode_prepared(const gsrq_shape* s, const void* X, gsrq_dtype x_dtype,
                                 int64_t ldx, const void* prepared, uint32_t* codes,
                                 float* residual, void* stream);

/*
 * gsrq_decode -- reconstruction as the sum over the first M_use stages of
 * gain[m][g][k] * shape[m][g][k][:] (Sec. 3; prefix decoding, Sec. 1): each
 * stage's codeword is rounded to float32 and the stages are summed in
 * float32 in stage order, then stored as out_dtype (float16 by
 * round-to-nearest-even).
 *
 *  codes             [N][gsrq_code_words(s)] uint32.
 *  M_use             1 <= M_use <= s->M.
 *  Xhat, ldo         [N][ldo] output (ldo >= D elements).
 */
gsrq_status gsrq_decode(const gsrq_shape* s, const uint32_t* codes,
                        int32_t M_use, const float* gain, const float* shape,
                        void* Xhat, gsrq_dtype out_dtype, int64_t ldo,
                        void* stream);

/*
 * gsrq_row_weights -- per-token weights of weighted GSKM (Sec. 5.3,
 * Appendix B): w_i = ||g_i||_2, the l2 norm of token i's gradient row, then
 * the log smoothing  w~_i = log(1 + lambda w_i),  lambda = tau /
 * (median(w) + 1e-8)  (the paper selects tau = 1).  The median is exact
 * (selection over the float32 norms); for even N it is the mean of the two
 * middle values.  The result feeds gsrq_train_stage's w.
 *
 *  grad, dtype, ldg  [N][ldg] gradient rows (ldg >= D), float16 or float32;
 *                    or NULL, in which case norms holds the N norms on entry
 *                    (non-negative, finite).
 *  N, D              rows (1 <= N <= 2^31 - 1) and row length (D >= 1 when
 *                    grad is given).
 *  tau               target median, finite and > 0.
 *  norms             [N] float32: output ||g_i||_2 (input when grad is NULL).
 *  w                 [N] float32 output, the smoothed weights.
 *  stats             [2] float64 output {median, lambda}.
 * All arrays are device memory; nothing else is written.  Arguments are
 * validated before any HIP call (GSRQ_E_ARG).
 */
gsrq_status gsrq_row_weights(const void* grad, gsrq_dtype dtype, int64_t N, int32_t D,
                             int64_t ldg, float tau, float* norms, float* w, double* stats,
                             void* stream);

/* Shape of one decoding step of attention over coded K and V caches. */
typedef struct {
  int32_t B;          /* sequences in the batch                              */
  int32_t cap;        /* cache rows reserved per sequence                    */
  int32_t Hq;         /* query heads                                         */
  int32_t Hkv;        /* key/value heads; Hq is a multiple of Hkv            */
  int32_t head_dim;   /* elements per head                                   */
  float rope_base;    /* RoPE base: theta_j = rope_base^(-2j / head_dim)     */
  float scale;        /* softmax scale, normally 1 / sqrt(head_dim)          */
  uint32_t flags;     /* GSRQ_ATTN_* below, or 0                             */
} gsrq_attn_shape;

/* The workspace already holds this call's tables: the float16 decode of the
 * key and value codebooks and the RoPE tables, written by an earlier
 * gsrq_attn_decode with the same workspace, codebooks (contents unchanged),
 * Hkv, head_dim and rope_base, so this call does not rebuild them (a
 * layer's codebooks are fixed across decoding steps).  Other arguments may
 * differ.  Checked on the device: the table build records the codebook
 * pointers, Hkv, head_dim and rope_base in a tag at the start of the
 * workspace, and a call whose arguments do not match the tag (a workspace
 * without tables, or tables of other codebook arrays or settings) writes
 * NaN to every output element.  Not checked: the codebook CONTENTS, which
 * the caller must not change while reusing the tables. */
enum { GSRQ_ATTN_TABLES_READY = 1 };

/* Workspace bytes gsrq_attn_decode needs for shape a over the 1-bit code
 * layout (d = 8, K = 256, M = 1). */
gsrq_status gsrq_attn_workspace_bytes(const gsrq_attn_shape* a, size_t* bytes);

/* Workspace bytes gsrq_attn_decode needs for shape a over codes of shape kv
 * (either layout gsrq_attn_decode accepts; the residual-coded layout's size
 * grows with kv->M).  Same argument checks as gsrq_attn_decode on a and kv:
 * GSRQ_E_ARG, or GSRQ_E_UNSUPPORTED for a layout it does not take. */
gsrq_status gsrq_attn_workspace_bytes_kv(const gsrq_attn_shape* a, const gsrq_shape* kv,
                                         size_t* bytes);

/*
 * gsrq_attn_decode -- one decoding step of attention over GSRQ-coded key and
 * value caches: the codes are unpacked, the keys dequantised and rotated by
 * RoPE, and softmax attention is taken without a float16 K/V tensor (the
 * fused decoding kernel of the paper's latency analysis, Appendix C).  For
 * sequence b of L = seq_len[b] tokens and query head h, reading key/value
 * head h / (Hq / Hkv):
 *   o = sum_i p_i vhat_i,
 *   p = softmax_i( scale * RoPE(q, L - 1) . RoPE(khat_i, i) ),  i = 0 .. L-1,
 * where khat_i, vhat_i are token i's decoded key and value rows (Sec. 3)
 * and RoPE turns elements j and j + head_dim/2 of a head together by the
 * angle position * theta_j (rotate-half form).  Keys are cached before RoPE;
 * the query is the newest token's, at position L - 1, before RoPE.
 *
 *  kv                code shape, N >= B * cap, D = Hkv * head_dim, K = 256, and
 *                    either the 1-bit layout (d = 8, M = 1: 16 subspaces per
 *                    head) or the residual-coded layout of the paper's sub-1-bit
 *                    rates (Sec. 6.2, Configurations; Appendix C measures 0.75
 *                    bit): d = head_dim, one subspace per head, 1 <= M <= 16
 *                    stages (M = 12 is 0.75 bit, M = 16 is 1 bit); a token's
 *                    key or value row is the sum of its M stage codewords.
 *                    Other valid shapes: GSRQ_E_UNSUPPORTED.
 *  k_codes, v_codes  [B][cap][gsrq_code_words(kv)] uint32 packed codes, token
 *                    i of sequence b in row b * cap + i; 16-byte aligned.
 *  seq_len           [B] int32 (device), clamped to [0, cap]; a sequence of
 *                    length 0 gets a zero output.
 *  k_gain, k_shape   key codebook [M][G][256], [M][G][256][d] and value
 *  v_gain, v_shape   codebook (shapes 16-byte aligned).
 *  q, q_dtype        [B][Hq][head_dim] queries, 16-byte aligned.
 *  out               [B][Hq][head_dim] float32.
 *  workspace         >= gsrq_attn_workspace_bytes_kv(a, kv) (for the 1-bit
 *                    layout also gsrq_attn_workspace_bytes(a)), 256-byte aligned.
 * Precision, 1-bit layout: keys and values enter as their float16 decode
 * (g * s rounded to float32, then to float16, as gsrq_decode's float16
 * output); the query and keys are rotated in float32 and, like the softmax
 * weights, rounded to float16 for the matrix products, with float32 sums
 * (the operand precision of float16 attention over a rotated float16
 * cache); chunks are merged in float64.
 * Precision, residual-coded layout: each key codeword enters as its float16
 * decode fp16(fp32(g s)); a key is summed two stages at a time in float16
 * (the pairs' shares of a score added in float32), turned and multiplied as
 * above; softmax weights stay float32 and are summed per stage and codeword
 * in float32 (LDS atomics: the order of these float32 sums, and so the last
 * bits of the output, may differ from call to call); the value side uses
 * the float32 codewords fl(g s), chunks merged and contracted in float64.
 * This build: head_dim = 128 and Hq / Hkv in {1, 2, 4}.
 */
gsrq_status gsrq_attn_decode(const gsrq_attn_shape* a, const gsrq_shape* kv,
                             const uint32_t* k_codes, const uint32_t* v_codes,
                             const int32_t* seq_len, const float* k_gain, const float* k_shape,
                             const float* v_gain, const float* v_shape, const void* q,
                             gsrq_dtype q_dtype, float* out, void* workspace, size_t ws_bytes,
                             void* stream);

/* Bytes of the library's own scratch for gsrq_attn_decode_noalloc, per GPU. */
#define GSRQ_ATTN_NOALLOC_BYTES ((size_t)16 << 20)

/*
 * gsrq_attn_decode_noalloc -- gsrq_attn_decode without a workspace argument,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, serving loops that must not call hipMalloc, harnesses that
 * forbid it.  Same arguments, computation and results as gsrq_attn_decode
 * (bit for bit, on the same inputs), except workspace and ws_bytes.
 *
 * Scratch: a device array of GSRQ_ATTN_NOALLOC_BYTES in the library, one
 * per GPU, held until the process ends; its address on the current device
 * is looked up once (hipGetSymbolAddress) on the first call there.  The
 * call itself allocates nothing.  A shape whose workspace
 * (gsrq_attn_workspace_bytes) exceeds GSRQ_ATTN_NOALLOC_BYTES returns
 * GSRQ_E_WORKSPACE before any HIP call.
 * Every call on a GPU shares that GPU's scratch, which keeps the last
 * call's contents: calls that overlap on one GPU (other streams, other
 * host threads) race and must be serialised by the caller.  Because the
 * tables stay, GSRQ_ATTN_TABLES_READY may be passed when the previous call
 * on this GPU used the same codebook arrays, Hkv, head_dim and rope_base;
 * the device-checked tag gives NaN outputs otherwise.
 */
gsrq_status gsrq_attn_decode_noalloc(const gsrq_attn_shape* a, const gsrq_shape* kv,
                                     const uint32_t* k_codes, const uint32_t* v_codes,
                                     const int32_t* seq_len, const float* k_gain,
                                     const float* k_shape, const float* v_gain,
                                     const float* v_shape, const void* q, gsrq_dtype q_dtype,
                                     float* out, void* stream);

/* Kernel kinds reported by the optional launch timing below. */
enum {
  GSRQ_KERNEL_ASSIGN = 0,     /* fused assignment + weighted accumulation */
                              /* (d <= 8: from the second iteration on also */
                              /* the previous iteration's codebook update)  */
  GSRQ_KERNEL_FINALIZE = 1,   /* codebook update + operand tiles          */
  GSRQ_KERNEL_ENCODE = 2,     /* stage-fused encoder                      */
  GSRQ_KERNEL_DECODE = 3,     /* gather-sum decoder                       */
  GSRQ_KERNEL_TRANSPOSE = 4,  /* subspace-major copy / seeding of the input */
  GSRQ_KERNEL_ACCUMULATE = 5, /* weighted sums per codeword slice (d > 8)  */
  GSRQ_KERNEL_FRAGMENTS = 6,  /* operand fragment tables (d > 8 or K > 256) */
  GSRQ_KERNEL_EXACT = 7,      /* float64 rescoring of deferred rows         */
  GSRQ_KERNEL_ATTENTION = 8,  /* decode attention over a coded cache       */
  GSRQ_KERNEL_KINDS = 9
};

/* Measurement hook, the library's only process state.  While enabled, every
 * launch of the kernels above is bracketed by two HIP events recorded on the
 * launch's stream.  Enabling clears earlier records; switching off keeps them
 * for gsrq_timing_read (launches enqueued while enabled stay recorded).  Not
 * thread-safe: enable, run and read from one host thread. */
gsrq_status gsrq_timing_enable(int on);

/* As gsrq_timing_enable, restricted to the kernel kinds whose bit
 * (1u << kind) is set in kinds; 0 switches timing off.  Each recorded launch
 * costs two event records on its stream, so timing only the kinds of
 * interest keeps the measured work close to the unmeasured one. */
gsrq_status gsrq_timing_enable_kinds(uint32_t kinds);

/* Wait for the recorded launches and return, per kernel kind k < n_kinds,
 * the summed event-to-event time in milliseconds and the launch count; then
 * clear the records. */
gsrq_status gsrq_timing_read(double* total_ms, int64_t* launches, int n_kinds);

#ifdef __cplusplus
}
#endif

#endif /* GSRQ_H */
