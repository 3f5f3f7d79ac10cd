/*
 * sdq.h -- C ABI of libsdq: Sigma-Delta quantized linear layers (SDQ-LLM,
 * arXiv 2510.03275) on AMD Instinct MI355X (gfx950).
 *
 * The library encodes fp32 weight matrices into binary or ternary
 * Sigma-Delta codes (Algorithm 1 without block compensation: block Hadamard
 * smoothing (Sylvester, sign-randomised or none), Resample up to OSR x the
 * block length, per-row scale,
 * first-order Sigma-Delta scan) and evaluates y = x W_hat^T directly on the
 * codes (Fig. 5: the activations are expanded to the oversampled length and
 * contracted against the codes, additions only in the decode kernel).
 *
 * Conventions for every entry point:
 *  - Pointers named *_dev are device (HBM) pointers, *_host are host pointers.
 *    All memory is owned by the caller; the library never frees or retains a
 *    caller pointer.  The library owns only its cached coefficient tables
 *    (one set per device and (block, M, Had) choice, allocated on first use,
 *    released by sdq_release_tables).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  GPU
 *    work is enqueued asynchronously on it; host-side argument errors are
 *    returned before anything is enqueued.
 *  - Matrices are row-major and densely packed unless stated otherwise.
 *  - The weights, activations, packed codes and workspaces passed to
 *    sdq_quantize, sdq_quantize_compensated, sdq_linear,
 *    sdq_expand_activations and sdq_linear_expanded are read and written in
 *    16-byte vectors and must be 16-byte aligned (every hipMalloc or PyTorch
 *    allocation is); a misaligned one is rejected with SDQ_ERR_ARG.
 *  - Functions return SDQ_OK or a negative sdq_status; sdq_last_error()
 *    gives a message for the last failure on the calling thread.
 */
#ifndef SDQ_H
#define SDQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SDQ_OK = 0,
  SDQ_ERR_ARG = -1,        /* null pointer, negative size, bad enum value        */
  SDQ_ERR_SHAPE = -2,      /* K not a multiple of the block, unsupported block   */
  SDQ_ERR_OSR = -3,        /* OSR < 1 or M = round(OSR*B) not a multiple of 32   */
  SDQ_ERR_LEVELS = -4,     /* levels not 2 or 3                                  */
  SDQ_ERR_NONFINITE = -5,  /* a weight (or an upsampled sample) is NaN or Inf    */
  SDQ_ERR_WORKSPACE = -6,  /* workspace pointer missing or too small             */
  SDQ_ERR_HIP = -7,        /* a HIP runtime call failed                          */
  SDQ_ERR_NOMEM = -8,      /* the coefficient-table cache could not allocate     */
  SDQ_ERR_UNSUPPORTED = -9, /* a valid request the library does not implement   */
  SDQ_ERR_NOT_SPD = -10    /* a Hessian (plus damping) is not positive definite  */
} sdq_status;

typedef enum { SDQ_F16 = 0, SDQ_BF16 = 1, SDQ_F32 = 2 } sdq_dtype;

/*
 * The smoothing matrix Had of Algorithm 1 (one B x B orthogonal matrix shared
 * by every block; the weights are encoded as w_b Had and reconstructed with
 * Had^T, Section 3.3):
 *   SDQ_HAD_SYLVESTER  Had = H_B / sqrt(B), the Sylvester matrix of Eq. 13
 *                      (the default of sdq_layout_init);
 *   SDQ_HAD_SIGNED     Had = diag(s) H_B / sqrt(B) for B caller-drawn signs
 *                      s_t in {-1, +1}: Algorithm 1 asks for a random
 *                      Hadamard matrix without fixing how it is drawn; this
 *                      sign flip keeps Had orthogonal;
 *   SDQ_HAD_NONE       Had = I (the ablation without Hadamard, Table 2).
 */
typedef enum { SDQ_HAD_NONE = 0, SDQ_HAD_SYLVESTER = 1, SDQ_HAD_SIGNED = 2 } sdq_hadamard;

/*
 * Storage of the codes: SDQ_PACK_FIELDS (1-bit binary or 2-bit ternary
 * fields, the default) or, for ternary codes, SDQ_PACK_BASE3 -- five codes per
 * byte, 1.6 bits each (Eq. 14 counts a ternary code as log2(3) = 1.58 bits).
 */
typedef enum { SDQ_PACK_FIELDS = 0, SDQ_PACK_BASE3 = 1 } sdq_packing;

/*
 * Geometry of one encoded linear layer (filled by sdq_layout_init; treat as
 * read-only).  Notation of the paper: the weight W has d_row = n rows and
 * d_col = k columns; Algorithm 1 splits the columns into blocks of B and
 * upsamples each block to M = round(OSR * B) samples (Algorithm 1, SDQuant).
 */
typedef struct sdq_layout {
  int64_t n;               /* rows of W (output features)                        */
  int64_t k;               /* columns of W (input features), multiple of block   */
  int32_t block;           /* B: 64, 128 or 256                                  */
  int32_t m_up;            /* M = round(osr * B), a multiple of 32, M >= B       */
  int32_t levels;          /* 2: codes in {-1,+1} (Eq. 4); 3: {-1,0,+1} (Eq. 6)  */
  int32_t bits;            /* bits per stored code: 1 (levels 2), 2 (levels 3)   */
  int64_t nb;              /* k / block                                          */
  int64_t k_up;            /* nb * M codes per row (Algorithm 1: osr * d_col)    */
  int64_t n_pad;           /* n rounded up to a multiple of 64                   */
  int64_t n_chunks;        /* 16-byte chunks per row = ceil(k_up / codes_per_chunk) */
  int32_t codes_per_chunk; /* 128 (binary) or 64 (ternary)                       */
  int32_t hadamard;        /* sdq_hadamard: the smoothing matrix Had             */
  uint32_t had_signs[8];   /* SDQ_HAD_SIGNED: bit t (word t/32, bit t%32) set    */
                           /* <=> s_t = -1, t < block; all zero otherwise        */
  int32_t packing;         /* sdq_packing                                        */
  int32_t reserved;
} sdq_layout;

/*
 * Packed code format (output of sdq_quantize, input of sdq_linear):
 *  - code j of row r is the Sigma-Delta output for sample j % M of block
 *    j / M (block-major, as Algorithm 1 places block i at columns
 *    i*osr ... (i+B)*osr of Q_out);
 *  - 16-byte chunk c of row r (codes c*CPC ... c*CPC+CPC-1, CPC =
 *    codes_per_chunk) starts at byte 16 * (((r/64) * n_chunks + c) * 64 + r%64):
 *    the 64 rows of a panel store their chunk c side by side;
 *  - inside a chunk, position q = j % CPC is in little-endian 32-bit word
 *    q / (32/bits), field of `bits` bits starting at bit bits*(q % (32/bits));
 *  - binary field: 1 = +1, 0 = -1.  Ternary field: 00 = 0, 01 = +1, 11 = -1
 *    (10 is never written and reads as 0);
 *  - padding codes (j >= k_up) and padding rows (r >= n) are zero bits.
 * SDQ_PACK_BASE3 (ternary only): codes_per_chunk = 80; byte p of a chunk
 * holds positions 5p .. 5p+4 with digits d_i = code + 1 as
 * v = 81 d0 + 27 d1 + 9 d2 + 3 d3 + d4 (the first position most significant),
 * stored as q = ceil(256 v / 243): v / 243 as an 8-bit fraction rounded up,
 * so that v = floor(243 q / 256) and the digits come out most significant
 * first as the integer parts of repeated multiplications by 3.  Padding codes
 * of real rows are code 0, padding rows zero bytes.  The chunk and panel
 * layout is the same.
 * Total size: sdq_codes_bytes() = n_pad * n_chunks * 16 bytes.
 */

/* Fill *out for an n x k weight at oversampling ratio osr (Section 3.2) with
 * `levels` code values and block size `block` (0 selects 256).
 * Errors: SDQ_ERR_ARG (out NULL, n < 0, k <= 0), SDQ_ERR_SHAPE (block not
 * 64/128/256 or k % block != 0), SDQ_ERR_OSR, SDQ_ERR_LEVELS. */
sdq_status sdq_layout_init(sdq_layout* out, int64_t n, int64_t k, double osr,
                           int32_t levels, int32_t block);

/* Select the smoothing matrix Had of a layout (Algorithm 1; sdq_hadamard).
 *   mode         SDQ_HAD_NONE, SDQ_HAD_SYLVESTER or SDQ_HAD_SIGNED.
 *   signs_host   SDQ_HAD_SIGNED: `block` int8 values, each -1 or +1 (host
 *                memory, read during the call only); otherwise ignored (may
 *                be NULL).
 * Codes encoded under one choice must be evaluated with the same layout.
 * Errors: SDQ_ERR_ARG (layout NULL, bad mode, signs missing or not +-1). */
sdq_status sdq_layout_set_hadamard(sdq_layout* layout, int32_t mode, const int8_t* signs_host);

/* Select the code storage of a ternary layout (sdq_packing); recomputes
 * codes_per_chunk (80 for SDQ_PACK_BASE3, 64 otherwise) and n_chunks.
 * Decode (m <= 16 activation rows) reads base-3 codes directly; prefill
 * (m > 16) first unpacks them to 2-bit fields in the workspace (one extra
 * pass over the codes per call, see sdq_linear_workspace_bytes).
 * Errors: SDQ_ERR_ARG (layout NULL or not from sdq_layout_init, bad value),
 * SDQ_ERR_LEVELS (base-3 for binary codes). */
sdq_status sdq_layout_set_packing(sdq_layout* layout, int32_t packing);

/* Bytes of the packed code buffer: n_pad * n_chunks * 16 (0 for a NULL layout). */
size_t sdq_codes_bytes(const sdq_layout* layout);

/* Compression ratio of Eq. 14, eta = bits * OSR / 16, using the stored bits
 * per code (1, 2, or 1.6 for base-3 packing) and OSR = M / B. */
double sdq_compression_ratio(const sdq_layout* layout);

/* Device workspace (bytes) sdq_quantize needs for this layout: the rotated
 * weights, the upsampled rows, per-row maxima and a status word (about
 * 4 * n_pad * (k + k_up) + 4 * n_pad + 256 bytes). */
size_t sdq_quantize_workspace_bytes(const sdq_layout* layout);

/*
 * Encode W into Sigma-Delta codes (Algorithm 1 with Had and SDQuant, no
 * block compensation; Eq. 7-8 for the scan, Eq. 4 / Eq. 6 for the
 * quantizer, per-row scale s_r = max |upsampled row|, threshold s_r / 2).
 *   w_dev        fp32 [n x k] row-major weights (device).
 *   codes_dev    device buffer of sdq_codes_bytes(layout) bytes, written in
 *                the packed format above (all bytes, padding included).
 *   scales_dev   fp32 [n] per-row scales (device).
 *   workspace    device buffer of at least sdq_quantize_workspace_bytes bytes;
 *                its contents need no initialisation.
 * Arithmetic is fp32 with every product and sum rounded separately, in the
 * order the paper's definitions give, so the codes are bit-exact and
 * deterministic.  Non-finite weights do not fail the call itself: they set a
 * flag in the workspace that sdq_quantize_check() reports.
 * Errors (host-side, nothing enqueued): SDQ_ERR_ARG, SDQ_ERR_WORKSPACE,
 * SDQ_ERR_NOMEM, SDQ_ERR_HIP. */
sdq_status sdq_quantize(const float* w_dev, const sdq_layout* layout, void* codes_dev,
                        float* scales_dev, void* workspace_dev, size_t workspace_bytes,
                        void* stream);

/* Synchronise `stream` and report the status flag of the last sdq_quantize
 * that used this workspace: SDQ_OK, or SDQ_ERR_NONFINITE when a weight or an
 * upsampled sample was NaN / Inf (the codes of such rows are meaningless). */
sdq_status sdq_quantize_check(const void* workspace_dev, void* stream);

/*
 * Block compensation of Algorithm 1 (its GPTQ-style block loop).  All in fp64.
 *
 * sdq_hessian_accumulate: H += 2 X^T X (the Hessian of Algorithm 1's caption
 * without its damping), for calibration activations x_dev (fp32 [m x k],
 * row-major) and h_dev (fp64 [k x k], row-major, both triangles written;
 * zero it before the first call).  Errors: SDQ_ERR_ARG.
 *
 * sdq_hessian_factor: Algorithm 1's factor step, u_dev = Cholesky((H + lambda I)^-1)^T,
 * the upper factor U with U^T U = (H + lambda I)^-1 (fp64 [k x k], lower part
 * zero), computed without forming the inverse (a blocked Cholesky of the
 * index-reversed matrix and a recursive blocked triangular inverse).  h_dev: symmetric
 * fp64 [k x k]; k a multiple of 64; lambda >= 0 absolute (GPTQ takes 1 % of the
 * mean diagonal).  workspace: sdq_hessian_factor_workspace_bytes(k) bytes
 * (about 18 k^2).  A non-positive pivot does not fail the call; it is reported
 * by sdq_hessian_check(workspace) as SDQ_ERR_NOT_SPD.
 * Errors: SDQ_ERR_SHAPE, SDQ_ERR_ARG, SDQ_ERR_WORKSPACE.
 *
 * sdq_quantize_compensated: as sdq_quantize, with the block compensation:
 * the row scales are those of the plain encoding of W; W is then walked in
 * blocks of B columns in fp64, each block rounded to fp32 and encoded with
 * those scales, and the columns after it corrected from the block's error
 * E = W_Q - Q_hat against its reconstruction (Resample back to B, Had^T),
 * with U_QQ, U_QF the blocks of u_dev on the block's rows:
 *   update = SDQ_COMP_GPTQ   W_F -= E diag(U_QQ)^-1 U_QF: GPTQ's block-wise
 *                            compensation, which Section 3.5 keeps, with its
 *                            column-wise part removed (each column's error
 *                            divided by its pivot; the printed listing writes
 *                            W_F -= E U_QF without the division);
 *   update = SDQ_COMP_JOINT  W_F -= E U_QQ^-1 U_QF: the optimal-brain-surgeon
 *                            correction of the jointly quantized block.
 * u_dev: fp64 [k x k] upper factor as from sdq_hessian_factor.  workspace:
 * sdq_quantize_compensated_workspace_bytes (the plain encoder's plus about
 * 8 n (k + 2B + M) + 24 nb B^2 bytes).  Codes and scales as sdq_quantize; the
 * non-finite flag is reported by sdq_quantize_check on the same workspace.
 * Errors as sdq_quantize, and SDQ_ERR_ARG for an unknown update.
 */
typedef enum { SDQ_COMP_GPTQ = 0, SDQ_COMP_JOINT = 1 } sdq_comp_update;
sdq_status sdq_hessian_accumulate(const float* x_dev, int64_t m, int64_t k, double* h_dev, void* stream);
size_t sdq_hessian_factor_workspace_bytes(int64_t k);
sdq_status sdq_hessian_factor(const double* h_dev, int64_t k, double lambda, double* u_dev,
                              void* workspace_dev, size_t workspace_bytes, void* stream);
sdq_status sdq_hessian_check(const void* workspace_dev, void* stream);
size_t sdq_quantize_compensated_workspace_bytes(const sdq_layout* layout);
sdq_status sdq_quantize_compensated(const float* w_dev, const sdq_layout* layout, const double* u_dev,
                                    int32_t update, void* codes_dev, float* scales_dev,
                                    void* workspace_dev, size_t workspace_bytes, void* stream);

/* Device workspace (bytes) sdq_linear needs for m activation rows: the
 * expanded activations, at offset 0 --
 *   m = 1:        fp32 x_tilde, k_up rounded up to whole chunks (binary,
 *                 base-3, or k_up < 16384); else the planes below in a
 *                 compact form (192 bytes per 64-code step) and the plane
 *                 scale of every block;
 *   2 <= m <= 16: x_tilde as 24-bit fixed point (three signed-byte planes,
 *                 rows in groups of four, per block in chunk slots; for
 *                 base-3 codes in the order of their digits: per group of
 *                 four 80-code chunks, five 64-code steps), then the fp32
 *                 plane scale of every (row, block);
 *   m > 16:       fp16 x_tilde, m x k_up rounded up to whole chunks (twice,
 *                 an fp16 pair hi + lo, for layouts with SDQ_HAD_NONE), each
 *                 row scaled by a power of two p_i that keeps it inside
 *                 fp16's normal range, then p_i and 1 / p_i (fp32 [m] each);
 * for a base-3 layout and m > 16 the chunks are those of 2-bit fields, and the
 * 2-bit copy of the codes follows (n_pad x ceil(k_up / 64) x 16 bytes). */
size_t sdq_linear_workspace_bytes(const sdq_layout* layout, int64_t m);

/*
 * y = x W_hat^T for the encoded layer (Fig. 5 and Algorithm 1's reconstruction: W_hat is
 * the decimated, Hadamard-restored reconstruction of the codes).  Computed as
 * x_tilde = per-block (x_b Had) D^T (D: Resample back to B), then
 * y[i, r] = s_r * sum_j C[r, j] x_tilde[i, j].  Equivalent to
 * sdq_expand_activations followed by sdq_linear_expanded on the same workspace.
 *   x_dev        [m x k] activations of type xt (F16, BF16 or F32), row-major.
 *   m            activation rows, >= 0 (m = 0 is a no-op).  m = 1 with
 *                binary or base-3 codes or k_up < 16384: fp32 expansion and
 *                a GEMV with additions only over the codes; 2 <= m <= 16, and
 *                one row of ternary 2-bit fields with k_up >= 16384: the
 *                expansion (for fp16 and bf16 x and m >= 2 on the matrix
 *                cores against E as an fp16 pair hi + lo, ~22 bits; else
 *                fp32) quantised to 24-bit fixed point and an exact int8 x
 *                int8 -> int32 matrix-core contraction against the codes
 *                (each code a +-1 or 0 weight: the products select, negate
 *                or drop the activations); larger m: the prefill path (fp16
 *                expansion, fp16 matrix cores).
 *   codes_dev, scales_dev  as written by sdq_quantize for `layout`.
 *   y_dev        fp32 [m x n] output, row-major.
 *   accumulate   0: y = x W_hat^T (y fully overwritten);  nonzero: y += x W_hat^T
 *                (e.g. a residual add fused into the projection).
 *   workspace    >= sdq_linear_workspace_bytes(layout, m) bytes, no
 *                initialisation needed.
 * Accuracy: max_r |y - y*| / max_r |y*| <= 1e-3 per activation row against the
 * fp64 definition.  The decode path splits K across workgroups for large
 * layers and then adds the partial sums into y with fp32 atomics, so results
 * may differ between calls in the last bits (relative ~1e-6); the prefill path
 * and unsplit decodes are bitwise deterministic.  Calls that share a
 * workspace must be ordered (same stream).
 * Errors: SDQ_ERR_ARG, SDQ_ERR_SHAPE, SDQ_ERR_WORKSPACE, SDQ_ERR_NOMEM, SDQ_ERR_HIP. */
sdq_status sdq_linear(const void* x_dev, sdq_dtype xt, int64_t m, const void* codes_dev,
                      const float* scales_dev, const sdq_layout* layout, float* y_dev,
                      int32_t accumulate, void* workspace_dev, size_t workspace_bytes,
                      void* stream);

/*
 * y_j = x W_hat_j^T for up to four encoded linears that read the same input
 * (e.g. the q, k and v projections of one hidden state, or gate and up), in
 * one expansion and one contraction launch: Fig. 5 brings the activations to
 * the oversampled length once, and the contraction's workgroups cover the
 * panels of every linear (launches and their ramp-up and tail are shared).
 *   count          1 .. 4 linears.
 *   codes_dev, scales_dev, y_dev   host arrays of `count` device pointers,
 *                  one per linear, as in sdq_linear (y_dev[j]: fp32 [m x n_j]).
 *   layouts        host array of `count` layouts, equal in k, block, m_up,
 *                  levels, Had and packing (they may differ in n; a linear with
 *                  n = 0 is skipped).
 *   workspace      >= sdq_linear_group_workspace_bytes(layouts, count, m).
 * Results, accuracy and accumulate as sdq_linear for each linear.
 * Errors: as sdq_linear; SDQ_ERR_ARG also for a count outside 1 .. 4 or
 * layouts that differ in more than n (sdq_linear_group_workspace_bytes
 * returns 0 for those). */
size_t sdq_linear_group_workspace_bytes(const sdq_layout* layouts, int32_t count, int64_t m);
sdq_status sdq_linear_group(const void* x_dev, sdq_dtype xt, int64_t m, int32_t count,
                            const void* const* codes_dev, const float* const* scales_dev,
                            const sdq_layout* layouts, float* const* y_dev, int32_t accumulate,
                            void* workspace_dev, size_t workspace_bytes, void* stream);

/* The contraction of sdq_linear_group alone, from the x_tilde that
 * sdq_expand_activations left in the workspace (same m and a layout of the
 * group's family), as sdq_linear_expanded does for one linear.  Arguments and
 * errors as sdq_linear_group without x. */
sdq_status sdq_linear_group_expanded(int64_t m, int32_t count, const void* const* codes_dev,
                                     const float* const* scales_dev, const sdq_layout* layouts,
                                     float* const* y_dev, int32_t accumulate, void* workspace_dev,
                                     size_t workspace_bytes, void* stream);

/*
 * sdq_linear without a workspace argument and without any device allocation,
 * for callers that cannot allocate: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Arguments, results and
 * errors as sdq_linear; the workspace is a fixed device array of
 * SDQ_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held until the
 * process ends (its address is looked up on the first call on each device).
 *  - Calls needing more workspace than that (sdq_linear_workspace_bytes)
 *    return SDQ_ERR_WORKSPACE; they fit for every one-to-sixteen-row call on
 *    2-bit fields up to k = 28672 at OSR 8, and prefill while
 *    m * k_up * 2 bytes (twice that without Had) plus 8 m bytes of row
 *    factors stay within the limit.
 *  - The coefficient tables are not built here: call sdq_prepare_layout for
 *    the layout on the current device first, else SDQ_ERR_UNSUPPORTED.
 *  - All calls on one GPU share its array; nothing in it needs to start at
 *    zero, but calls that overlap on one GPU (different streams, or threads
 *    without ordering) race on it and must not be issued.
 */
#define SDQ_NOALLOC_SCRATCH_BYTES (((size_t)32) << 20)
sdq_status sdq_linear_noalloc(const void* x_dev, sdq_dtype xt, int64_t m, const void* codes_dev,
                              const float* scales_dev, const sdq_layout* layout, float* y_dev,
                              int32_t accumulate, void* stream);

/* First step of sdq_linear: write x_tilde (the activation expansion of Fig. 5:
 * per block x_b Had D^T) for m activation rows into the workspace.  The
 * expansion depends only on (k, block, m_up, levels) of the layout, so one
 * call can serve several linears that share the input and those four values
 * (e.g. projections of one hidden state); the workspace must then be large
 * enough for each of them.  Errors as sdq_linear. */
sdq_status sdq_expand_activations(const void* x_dev, sdq_dtype xt, int64_t m,
                                  const sdq_layout* layout, void* workspace_dev,
                                  size_t workspace_bytes, void* stream);

/* Second step of sdq_linear: y[i, r] = s_r * sum_j C[r, j] x_tilde[i, j] from
 * the x_tilde that sdq_expand_activations left in the workspace (same m and a
 * layout with the same k, block, m_up, levels and packing).  m = 1 (binary,
 * base-3 or k_up < 16384): addition-only lookup-table GEMV; 2 <= m <= 16 and
 * one row of ternary 2-bit fields with k_up >= 16384: exact int8 matrix-core
 * contraction against the fixed-point expansion; larger m: fp16 MFMA GEMM.
 * accumulate as in sdq_linear.  Errors as sdq_linear. */
sdq_status sdq_linear_expanded(int64_t m, const void* codes_dev, const float* scales_dev,
                               const sdq_layout* layout, float* y_dev, int32_t accumulate,
                               void* workspace_dev, size_t workspace_bytes, void* stream);

/*
 * MultiOSR (Section 3.4): per-linear OSR from weight variance and size, host
 * only.  Reading of the prose rule: layer OSR proportional to the inverse of
 * the layer's parameter-weighted variance, linear OSR inside a layer
 * proportional to n_params / variance, both clipped to [lo, hi] with scale
 * factors found by fp64 bisection so the parameter-weighted means hit the
 * target; then floor to the grid and add one grid step in order of largest
 * remainder while the model's weighted mean stays <= target.
 *   var_host[count]       per-linear weight variance (<= 0 maps to hi).
 *   nparams_host[count]   parameter count of each linear (> 0).
 *   layer_host[count]     layer index of each linear.
 *   osr_out_host[count]   result, multiples of `grid` in [lo, hi].
 * Errors: SDQ_ERR_ARG (null pointers with count > 0, count < 0, a
 * non-positive parameter count, not 0 < lo <= target <= hi, grid <= 0). */
sdq_status sdq_multiosr(const double* var_host, const int64_t* nparams_host,
                        const int32_t* layer_host, int64_t count, double target, double lo,
                        double hi, double grid, double* osr_out_host);

/* Mean and population variance (two-pass, fp64 accumulation) of `count` fp32
 * values on the device: the variance input of MultiOSR (Section 3.4).
 *   out_dev   double[2] = {mean, variance} (device).
 *   workspace >= sdq_moments_workspace_bytes(count) bytes.
 * Errors: SDQ_ERR_ARG, SDQ_ERR_WORKSPACE, SDQ_ERR_HIP. */
size_t sdq_moments_workspace_bytes(int64_t count);
sdq_status sdq_weight_moments(const float* w_dev, int64_t count, double* out_dev,
                              void* workspace_dev, size_t workspace_bytes, void* stream);

/* Unpack a packed code buffer (host copy) into int8 codes [n x k_up] in
 * {-1, 0, +1} (host).  Errors: SDQ_ERR_ARG. */
sdq_status sdq_unpack_codes(const sdq_layout* layout, const void* codes_host, int8_t* out_host);

/* The fp32 interpolation coefficients the encoder uses: out_host[p] =
 * fp32(g(p)) for p in [0, block*m_up), with g the periodic-sinc kernel of
 * the upsampling Resample (1 at p = 0, 0 at other multiples of M,
 * sin(pi tau) / (B tan(pi tau / B)) at tau = p / M).  Errors: SDQ_ERR_ARG,
 * SDQ_ERR_SHAPE, SDQ_ERR_OSR. */
sdq_status sdq_upsample_table(int32_t block, int32_t m_up, float* out_host);

/* Upload the coefficient tables for (block, m_up) with the Sylvester Had on
 * the current device ahead of time, so that later calls allocate nothing.
 * Errors: SDQ_ERR_SHAPE, SDQ_ERR_OSR, SDQ_ERR_NOMEM, SDQ_ERR_HIP. */
sdq_status sdq_prepare(int32_t block, int32_t m_up);

/* As sdq_prepare, for the (block, M, Had) choice of a layout.
 * Errors: SDQ_ERR_ARG (layout not from sdq_layout_init), SDQ_ERR_NOMEM, SDQ_ERR_HIP. */
sdq_status sdq_prepare_layout(const sdq_layout* layout);

/* Free every cached coefficient table (all devices).  No call may be in flight. */
void sdq_release_tables(void);

/* Static description of a status code, and the message of the last failure
 * on the calling thread. */
const char* sdq_status_string(sdq_status status);
const char* sdq_last_error(void);

/* Library version: major * 10000 + minor * 100 + patch. */
int32_t sdq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SDQ_H */
