/*
 * galore.h -- C ABI of the MI355X (gfx950) GaLore 2 gradient-subspace library.
 *
 * Paper: "GaLore 2: Large-Scale LLM Pre-Training by Gradient Low-Rank
 * Projection" (Su, Gu, Xu, Tian, Zhao, 2025).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All matrix pointers are DEVICE pointers, row-major, owned by the caller.
 *    The library never allocates or frees device memory, creates no stream
 *    and never synchronises the device: work is enqueued on the caller's
 *    `stream` (and, where an entry point takes one, on the caller's optional
 *    second stream `aux_stream`, forked from and joined back into `stream`),
 *    and every entry point returns as soon as it is enqueued.
 *  - G is the m x n gradient as produced by autograd (+grad). s = min(m, n) is
 *    the projected side, l = max(m, n). A denotes G when m <= n and G^T when
 *    m > n, so A is always s x l (paper §3: left singular vectors when m <= n,
 *    right ones otherwise).
 *  - Batching: `batch` matrices of identical shape sit at fixed element strides
 *    (`stride_*`); matrix b of a batch is at base + b * stride.
 *  - ld* is the leading dimension (row pitch, in elements) of a row-major
 *    matrix and must be >= its row length.
 *  - Status: every call validates its arguments on the host before enqueuing
 *    anything and returns a galore_status_t (< 0 on error, nothing enqueued).
 *    A launch failure reported by the HIP runtime returns GALORE_ERR_HIP.
 *    NaN/Inf inputs are not checked on the host: they propagate to the
 *    outputs, and the subspace update also reports them in `info` (see
 *    galore_rsvd_update). Signed zeros and subnormal inputs are ordinary
 *    values; a gradient whose entries all lie in the subnormal range keeps
 *    only the precision fp32 arithmetic has there.
 */
#ifndef GALORE_H_
#define GALORE_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#if defined(__GNUC__) || defined(__clang__)
#define GALORE_API __attribute__((visibility("default")))
#else
#define GALORE_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GALORE_F32 = 0,   /* IEEE binary32                                  */
    GALORE_BF16 = 1   /* bfloat16 storage, widened exactly to fp32       */
} galore_dtype_t;

typedef enum {
    GALORE_OK = 0,
    GALORE_ERR_INVALID_ARG = -1,  /* null pointer, bad scalar, bad dtype     */
    GALORE_ERR_SHAPE = -2,        /* sizes, ranks or leading dims invalid    */
    GALORE_ERR_WORKSPACE = -3,    /* workspace missing or too small          */
    GALORE_ERR_HIP = -4           /* the HIP runtime reported a failure      */
} galore_status_t;

/* Human-readable name of a status code (static storage). */
GALORE_API const char* galore_status_string(int status);

/* Library version: major * 10000 + minor * 100 + patch. */
GALORE_API int galore_version(void);

/*
 * Gaussian sketch (randomized range finder of Halko, Martinsson & Tropp 2011,
 * adopted by paper §4.1.2): writes the l x k fp32 matrix Omega (row-major,
 * ld = k). Entries (4 i4 + t, j), t = 0..3, share one Philox4x64-10 block
 * (Salmon et al. 2011) with key (seed, 0) and counter (j * ceil(l/4) + i4,
 * sketch_index, 0, 0); the top 53 bits of output words 0 and 1 give u1 in
 * (0,1] and u2 in [0,1) for rows 4 i4 (sqrt(-2 ln u1) cos(2 pi u2)) and 4 i4 + 1
 * (the sin member of the same Box-Muller pair), words 2 and 3 likewise for rows
 * 4 i4 + 2 and 4 i4 + 3; each normal is computed in fp64 and rounded once to
 * the nearest bfloat16 (ties to even), stored as fp32.
 * Exposed so that callers and tests can inspect the sketch the subspace
 * update uses. Errors: omega NULL -> INVALID_ARG; l < 1 or k < 1 -> SHAPE.
 */
GALORE_API int galore_sketch(float* omega, int64_t l, int64_t k, uint64_t seed, uint64_t sketch_index,
                  hipStream_t stream);

/*
 * Bytes of workspace galore_rsvd_update needs for `batch` m x n matrices with
 * rank r, oversampling p and gradient storage g_dtype (a bf16 gradient also
 * holds its transposed copy and the bf16 split of the fp32 sketch operands).
 * Returns 0 for invalid sizes or dtype.
 */
GALORE_API size_t galore_rsvd_workspace_size(int64_t m, int64_t n, int32_t r, int32_t p, int32_t batch,
                                             int32_t g_dtype);

/*
 * Subspace update (paper §3 and Alg. 1: P = top-r singular vectors of G on
 * its shorter side; paper §4.1.2: computed by the randomized SVD of Halko et
 * al. 2011 -- randomized subspace iteration followed by the direct SVD of the
 * small projected matrix).
 *
 *   k = min(r + p, s); Omega (l x k) from (seed, sketch_index0 + b)
 *   Y = A Omega; Q = orth(Y)
 *   q times: Z = A^T Q; Z = orth(Z); Y = A Z; Q = orth(Y)
 *   B = Q^T A (k x l); B = U_B Sigma V^T
 *   P = Q U_B[:, :r] (s x r) with each column's largest-magnitude entry made
 *   positive (sign convention, paper §4.1.3); sigma = Sigma[:r], descending.
 *
 * Inputs:  G (g_dtype, m x n, ld ldg, batch stride stride_g elements).
 * Outputs: P (fp32, s x r, ld ldp >= r, stride stride_p);
 *          sigma (fp32, r values per matrix at stride stride_sigma; may be NULL);
 *          info (device int32[batch]; may be NULL): 0 = converged; 24 = the
 *          small SVD did not converge within its sweep limit (16 sweeps for
 *          k = min(r + p, s) <= 2048, 24 above);
 *          25 = a column of the small SVD has a NaN or Inf norm (NaN or Inf
 *          in G): sigma and P then hold NaN or Inf and must not be used.
 *          Every non-zero value means failure. The work enqueued is bounded
 *          either way: the sweep count is fixed on the host, every device loop
 *          is bounded by the sizes, and no address depends on a computed value.
 * Workspace: device buffer of at least galore_rsvd_workspace_size(...) bytes,
 *          256-byte aligned; contents are scratch and may be reused afterwards.
 * Streams: everything is enqueued on `stream` when aux_stream is NULL (or
 *          equal to `stream`, or batch < 2). Otherwise aux_stream, a second
 *          stream of the caller on the same device, takes the Cholesky
 *          factorisations and the small SVD's sweeps of the second half of the
 *          batch: it is forked from `stream` and joined back into it with two
 *          events the library creates once per device, so all completion is
 *          still ordered on `stream` and the results are bit-identical either
 *          way (the halves' latency-bound launch chains then overlap). Calls
 *          from several host threads are safe; they serialise only while
 *          enqueuing the fork and join.
 * Errors:  NULL G/P/workspace -> INVALID_ARG; m,n,r < 1, r > s, p < 0, q < 0,
 *          r + p > 4096 (largest supported sketch width), ldg < n, ldp < r,
 *          batch < 1, or 3 * (k rounded up to 128) * (l rounded up to 128) above
 *          2^31 - 1 (the exact Gram's digit planes of one matrix, addressed with
 *          32-bit offsets; e.g. l up to about 600000 at k = 1056) -> SHAPE;
 *          workspace_bytes too small -> WORKSPACE.
 */
GALORE_API int galore_rsvd_update(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg,
                       int64_t stride_g, int32_t r, int32_t p, int32_t q, uint64_t seed,
                       uint64_t sketch_index0, float* P, int64_t ldp, int64_t stride_p,
                       float* sigma, int64_t stride_sigma, int32_t* info, int32_t batch,
                       void* workspace, size_t workspace_bytes, hipStream_t stream,
                       hipStream_t aux_stream);

/*
 * Exact SVD projector (the full SVD that paper §4.1.2 replaces by the
 * randomized one): galore_rsvd_update with the sketch as wide as the short
 * side (k = s, p = s - r) and no power iteration. The sketch then spans the
 * whole short side, Q is an orthonormal basis of it and the SVD of B = Q^T A
 * is the SVD of A, so P and sigma are the exact top-r singular vectors and
 * values up to rounding. Arguments as galore_rsvd_update (no seed: the result
 * does not depend on the sketch). s <= 4096.
 * Errors: as galore_rsvd_update; s > 4096 -> SHAPE.
 */
GALORE_API size_t galore_svd_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch, int32_t g_dtype);
GALORE_API int galore_svd_update(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg,
                                 int64_t stride_g, int32_t r, float* P, int64_t ldp, int64_t stride_p, float* sigma,
                                 int64_t stride_sigma, int32_t* info, int32_t batch, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream, hipStream_t aux_stream);

/*
 * Stages of the subspace update reported by galore_rsvd_update_traced.
 */
typedef enum {
    GALORE_STAGE_SKETCH = 0,      /* Omega from the counter-based generator (1 launch)         */
    GALORE_STAGE_PRODUCT_A = 1,   /* Y = A X, matrix cores (bf16 planes for a bf16 G; 1 launch) */
    GALORE_STAGE_PRODUCT_AT = 2,  /* Z = A^T Q, as PRODUCT_A (1 launch)                         */
    GALORE_STAGE_GRAM = 3,        /* exact Gram X^T X of a tall-skinny block (4 launches)       */
    GALORE_STAGE_CHOLESKY = 4,    /* blocked Cholesky of the Gram (+ inverse of the factor)     */
    GALORE_STAGE_TRIANGULAR = 5,  /* Q = Y R^-1, fp32 matrix cores (1 launch)                   */
    GALORE_STAGE_JACOBI = 6,      /* small SVD: all Jacobi sweeps and the sort                  */
    GALORE_STAGE_PROJECTOR = 7,   /* P = Q U_B[:, :r], fp32 matrix cores (1 launch)             */
    GALORE_STAGE_OTHER = 8,       /* small kernels: dependent-column fill, sign convention      */
    GALORE_STAGE_OPERAND = 9,     /* bf16 G only: transposed copy of G, bf16 split of an fp32    */
                                  /* operand (1 launch each)                                    */
    GALORE_STAGE_REFINE = 10      /* fp64 refinement of the small SVD's vectors                 */
} galore_stage_t;

/*
 * galore_rsvd_update with stage timing: the same work on the same stream;
 * in addition, for the i-th stage instance enqueued (i < capacity), events[2i]
 * is recorded on `stream` just before it and events[2i+1] just after it, and
 * stages[i] receives its galore_stage_t. *count receives the number of
 * instances recorded (stages past `capacity` run untimed). `events` (2 *
 * capacity handles created by the caller, e.g. with timing enabled) and
 * `stages`/`count` are host arrays; read the events after the stream has
 * reached them. For profiling callers: a run of the subspace update broken
 * down by stage, and the per-launch duration of its single-launch stages.
 * Errors: those of galore_rsvd_update; capacity < 0, count NULL, or
 * capacity > 0 with NULL events/stages or a NULL handle -> INVALID_ARG.
 */
GALORE_API int galore_rsvd_update_traced(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg,
                              int64_t stride_g, int32_t r, int32_t p, int32_t q, uint64_t seed,
                              uint64_t sketch_index0, float* P, int64_t ldp, int64_t stride_p,
                              float* sigma, int64_t stride_sigma, int32_t* info, int32_t batch,
                              void* workspace, size_t workspace_bytes, hipStream_t stream,
                              hipStream_t aux_stream, hipEvent_t* events, int32_t* stages, int32_t capacity,
                              int32_t* count);

/*
 * Bytes of workspace galore_project uses for `batch` m x n matrices with rank
 * r and gradient storage g_dtype: for a bf16 gradient, the three bf16 planes
 * of P^T that feed the bf16 matrix cores; 0 for an fp32 gradient (which needs
 * none) and for invalid sizes or dtype.
 */
GALORE_API size_t galore_project_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch, int32_t g_dtype);

/*
 * Projection R = P^T A (paper §3, R_t = P_t^T G_t; paper Alg. 1).
 * P: fp32 s x r (ld ldp); G: g_dtype m x n (ld ldg); R: fp32 r x l (ld ldr).
 * For m > n this is R = (G P)^T.
 * Workspace (optional, device, 256-byte aligned, scratch): with a bf16
 * gradient and at least galore_project_workspace_size(...) bytes, P is split
 * there into three bf16 planes (P = P1 + P2 + P3 exactly to fp32 rounding)
 * and the product runs on the bf16 matrix cores with fp32 accumulation
 * (16-byte aligned rows of G and s a multiple of 32; otherwise, and with
 * workspace NULL, it runs on the fp32 matrix cores). The result is the
 * fp32-accurate product either way.
 * Errors: NULL P/G/R -> INVALID_ARG; sizes/ld invalid, r > s -> SHAPE;
 * misaligned workspace, or bf16 G with a non-NULL workspace shorter than
 * galore_project_workspace_size(...) -> WORKSPACE.
 */
GALORE_API int galore_project(const float* P, int64_t ldp, int64_t stride_p, const void* G, int32_t g_dtype,
                   int64_t m, int64_t n, int64_t ldg, int64_t stride_g, int32_t r, float* R,
                   int64_t ldr, int64_t stride_r, int32_t batch, void* workspace, size_t workspace_bytes,
                   hipStream_t stream);

/*
 * galore_project without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving or training loops,
 * harnesses that forbid allocation): the same projection, kernels and results
 * as galore_project with a workspace of galore_project_workspace_size(...)
 * bytes, with that scratch held instead in a fixed-size device array inside
 * the library (galore_project_noalloc_max_bytes() bytes, 64 MiB; one copy on
 * each device the library runs on, kept until the process ends). The caller
 * passes inputs and outputs as for galore_project; the call allocates nothing
 * (no hipMalloc, no allocating library routine). The first call on a device
 * looks up that device's copy of the array (under a lock).
 * Every call on a device shares that device's array: calls that overlap on one
 * device (concurrent streams or host threads) race and must be serialised by
 * the caller. The array needs no initial contents (each call writes every byte
 * it reads).
 * Errors: as galore_project; a bf16 gradient whose workspace size
 * (galore_project_workspace_size) exceeds galore_project_noalloc_max_bytes()
 * -> WORKSPACE, checked before any device call; the lookup of the array failing
 * -> HIP. An fp32 gradient needs no scratch (fp32 matrix cores).
 */
GALORE_API size_t galore_project_noalloc_max_bytes(void);
GALORE_API int galore_project_noalloc(const float* P, int64_t ldp, int64_t stride_p, const void* G, int32_t g_dtype,
                                      int64_t m, int64_t n, int64_t ldg, int64_t stride_g, int32_t r, float* R,
                                      int64_t ldr, int64_t stride_r, int32_t batch, hipStream_t stream);

/*
 * Low-rank Adam on the rows x cols projected state (paper §3 moment equations;
 * paper Alg. 1 with its bias correction applied to temporaries, the stored
 * moments staying uncorrected):
 *   M <- beta1 M + (1 - beta1) R;  V <- beta2 V + (1 - beta2) R^2
 *   N  = (M / (1 - beta1^t)) / (sqrt(V / (1 - beta2^t)) + eps)
 * R, M, V, N: fp32, same shape, ld and batch stride. M and V are updated in
 * place; N may alias R. t >= 1 is the step number (the bias terms are formed
 * on the host in fp64 from the fp32 betas).
 * Errors: NULL pointers -> INVALID_ARG; beta outside [0,1), eps <= 0, non-finite
 * scalars, t < 1 -> INVALID_ARG; rows/cols < 1, ld < cols -> SHAPE.
 */
GALORE_API int galore_lowrank_adam_step(const float* R, float* M, float* V, float* N, int64_t rows,
                             int64_t cols, int64_t ld, int64_t stride, int32_t batch, float beta1,
                             float beta2, float eps, int64_t t, hipStream_t stream);

/*
 * Bytes of workspace galore_project_back uses for `batch` m x n matrices with
 * rank r: three bf16 planes of P and of N^T per matrix. 0 for invalid sizes.
 */
GALORE_API size_t galore_project_back_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch);

/*
 * Back-projection and weight update (paper §3: G~ = alpha P N, W <- W + eta G~;
 * paper Alg. 1). The library works with the autograd gradient, so it applies
 *   W <- W - (lr * alpha) * P N         (m <= n)
 *   W <- W - (lr * alpha) * (P N)^T     (m > n)
 * P: fp32 s x r (ld ldp); N: fp32 r x l (ld ldn); W: fp32 m x n (ld ldw),
 * updated in place.
 * Workspace (optional, device, 256-byte aligned, scratch): with at least
 * galore_project_back_workspace_size(...) bytes, P and N are split there into
 * three bf16 planes each (exact to fp32 rounding) and P N runs on the bf16
 * matrix cores as the six plane products whose size reaches fp32 rounding,
 * accumulated in fp32 (r a multiple of 32; otherwise, and with workspace NULL,
 * on the fp32 matrix cores).
 * Errors: NULL pointers -> INVALID_ARG; non-finite lr/alpha -> INVALID_ARG;
 * sizes/ld invalid, r > s -> SHAPE; misaligned or short non-NULL workspace ->
 * WORKSPACE.
 */
GALORE_API int galore_project_back(const float* P, int64_t ldp, int64_t stride_p, const float* N,
                        int64_t ldn, int64_t stride_n, float* W, int64_t m, int64_t n,
                        int64_t ldw, int64_t stride_w, int32_t r, float lr, float alpha,
                        int32_t batch, void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Bytes of workspace galore_align_projector needs to re-express the first
 * moment for `batch` projectors of rank r (one r x r overlap matrix each).
 * 0 for invalid sizes.
 */
GALORE_API size_t galore_align_workspace_size(int32_t r, int32_t batch);

/*
 * Subspace switch (paper §4.1.3: singular vectors are defined only up to sign
 * and the randomized SVD adds randomness, so a new projector can disagree in
 * sign with the one it replaces; paper Alg. 1 replaces P every T steps).
 * Column j of P_new is negated in place when its overlap with column j of
 * P_old, <p_old_j, p_new_j> (summed in fp64 from the exact fp32 products), is
 * negative; an overlap of zero (or NaN) keeps the sign. Optionally the first
 * moment is re-expressed in the new basis: M_out = (P_new^T P_old) M_in with
 * the aligned P_new, on the fp32 matrix cores.
 * P_old, P_new: fp32 s x r (ld ld_old / ld_new >= r, batch strides stride_old /
 *          stride_new); flips: device int32[batch * r] or NULL, 1 where a column
 *          was negated.
 * M_in, M_out: fp32 r x l (ld ldm >= l, batch stride stride_m), both NULL (no
 *          re-expression) or both set and not overlapping.
 * Workspace: with M_in, at least galore_align_workspace_size(r, batch) bytes,
 *          device, 256-byte aligned, scratch; unused otherwise (may be NULL).
 * Errors: NULL P_old/P_new, only one of M_in/M_out, or M_out overlapping M_in ->
 *          INVALID_ARG; s, r < 1, r > s, ld/stride too small, l < 1 -> SHAPE;
 *          missing, misaligned or short workspace when re-expressing -> WORKSPACE.
 */
GALORE_API int galore_align_projector(const float* P_old, int64_t ld_old, int64_t stride_old, float* P_new,
                                      int64_t ld_new, int64_t stride_new, int64_t s, int32_t r, int32_t* flips,
                                      const float* M_in, float* M_out, int64_t ldm, int64_t stride_m, int64_t l,
                                      int32_t batch, void* workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/*
 * Number of fp32 block scales galore_lowrank_adam8_step keeps per moment and
 * matrix for a rows x cols state: ceil(rows * cols / 2048). 0 for invalid sizes.
 */
GALORE_API int64_t galore_adam8_scale_count(int64_t rows, int64_t cols);

/*
 * 8-bit block-wise low-rank Adam (paper §4.2: GaLore 2 uses the 8-bit Adam
 * optimizer of bitsandbytes, after Dettmers et al.; the paper fixes no data
 * type). The moments of each matrix are stored in blocks of 2048 consecutive
 * elements of the packed row-major rows x cols state:
 *   M8: OCP FP8 E4M3 codes of M / Ms[block]
 *   V8: OCP FP8 E5M2 codes of V / Vs[block]
 * where a block's scale is the smallest power of two 2^k with block max
 * |value| <= 2^k * 448 (E4M3) or 2^k * 57344 (E5M2), the formats' largest
 * finite values (round half to even, saturating, subnormals kept; an all-zero
 * block has scale 0 and codes 0, so zero-filled codes and scales are the zero
 * state).
 * One call decodes the moments, applies galore_lowrank_adam_step's update in
 * fp32 (N from the new moments, bias exponent t; N is formed with the hardware
 * reciprocal and square root, within a few ulps of the correctly rounded
 * operations), and re-encodes the new moments with new block scales.
 * R, N: fp32 rows x cols (ld ld, batch stride stride); N may alias R.
 * M8, V8: device bytes, rows * cols per matrix, packed, matrix b at b * rows * cols.
 * Ms, Vs: device fp32, galore_adam8_scale_count(rows, cols) per matrix, packed.
 * All state is updated in place.
 * Errors: NULL pointers, betas outside [0, 1), eps <= 0, non-finite scalars,
 * t < 1 -> INVALID_ARG; rows/cols < 1, ld < cols, batch < 1, stride too small -> SHAPE.
 */
GALORE_API int galore_lowrank_adam8_step(const float* R, float* N, int64_t ld, int64_t stride, uint8_t* M8,
                                         float* Ms, uint8_t* V8, float* Vs, int64_t rows, int64_t cols,
                                         int32_t batch, float beta1, float beta2, float eps, int64_t t,
                                         hipStream_t stream);

/*
 * Low-bit projector (paper §4.2: GaLore 2 supports low-bit projection
 * matrices, after Q-GaLore; the paper fixes no scheme). Each column j of the
 * fp32 s x r projector P is quantised symmetrically:
 *   qmax = 2^(bits-1) - 1 (127 for bits = 8, 7 for bits = 4)
 *   scale_j = max_i |P_ij| / qmax            (binary32 division)
 *   code_ij = P_ij / scale_j rounded half to even, clamped to [-qmax, qmax]
 * and a zero column gets scale 0 and codes 0; the dequantised projector is
 * code_ij * scale_j. Codes are row-major: bits = 8 one two's-complement byte
 * each (ldq >= r bytes); bits = 4 two per byte, column 2c in the low nibble
 * and 2c + 1 in the high nibble, 4-bit two's complement (ldq >= ceil(r / 2)).
 * P: fp32 s x r (ld ldp, stride stride_p); Q: device bytes (ld ldq, stride
 * stride_q); scales: fp32, r per matrix (stride stride_scales). Non-finite
 * entries of P give unspecified codes.
 * Errors: NULL pointers, bits not 4 or 8 -> INVALID_ARG; s, r < 1, r > s,
 * ldp < r, ldq too small, strides too small -> SHAPE.
 */
GALORE_API int galore_quantize_projector(const float* P, int64_t ldp, int64_t stride_p, int64_t s, int32_t r,
                                         int32_t bits, uint8_t* Q, int64_t ldq, int64_t stride_q, float* scales,
                                         int64_t stride_scales, int32_t batch, hipStream_t stream);

/* Bytes of workspace galore_project_quantized needs (0 for invalid sizes). */
GALORE_API size_t galore_project_quantized_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch);

/*
 * Projection with the low-bit projector: R = Pq^T A with Pq = code * scale
 * (galore_quantize_projector's codes and scales; paper §3 projection). With a
 * bf16 gradient (16-byte aligned rows, s a multiple of 32 for m <= n) the
 * codes form one exact bf16 plane, the product runs once on the bf16 matrix
 * cores with fp32 accumulation and each row of R is multiplied by its scale;
 * otherwise Pq is rounded to fp32 and the product runs on the fp32 matrix
 * cores. Shapes and errors as galore_project, plus those of the codes;
 * the workspace (galore_project_quantized_workspace_size bytes, device,
 * 256-byte aligned, scratch) is required.
 */
GALORE_API int galore_project_quantized(const uint8_t* Q, int64_t ldq, int64_t stride_q, const float* scales,
                                        int64_t stride_scales, int32_t bits, const void* G, int32_t g_dtype,
                                        int64_t m, int64_t n, int64_t ldg, int64_t stride_g, int32_t r, float* R,
                                        int64_t ldr, int64_t stride_r, int32_t batch, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace galore_project_back_quantized needs (0 for invalid sizes). */
GALORE_API size_t galore_project_back_quantized_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch);

/*
 * Back-projection with the low-bit projector: W <- W - (lr * alpha) Pq N (or
 * its transpose for m > n), Pq = code * scale (paper §3 back-projection). With
 * r a multiple of 32 and 16-byte aligned planes the scales are folded into the
 * rows of N (one fp32 rounding), N^T is split into three bf16 planes and the
 * exact code plane multiplies them on the bf16 matrix cores (three products
 * instead of six for an fp32 P); otherwise Pq is rounded to fp32 and the fp32
 * matrix cores run it. Shapes and errors as galore_project_back, plus those of
 * the codes; the workspace (galore_project_back_quantized_workspace_size bytes,
 * device, 256-byte aligned, scratch) is required.
 */
GALORE_API int galore_project_back_quantized(const uint8_t* Q, int64_t ldq, int64_t stride_q, const float* scales,
                                             int64_t stride_scales, int32_t bits, const float* N, int64_t ldn,
                                             int64_t stride_n, float* W, int64_t m, int64_t n, int64_t ldw,
                                             int64_t stride_w, int32_t r, float lr, float alpha, int32_t batch,
                                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Measurement helper (not part of the method): launches `blocks` workgroups of
 * four waves, each wave running `iterations` x 4 independent bf16 matrix-core
 * products (v_mfma_f32_32x32x16_bf16) on register operands, and writes one
 * float per thread to `sink` (device, blocks * 256 floats). *flops (host)
 * receives the matrix-core work of the launch; divided by the launch time
 * (timed by the caller on `stream`) it is the sustained bf16 MFMA rate of the
 * chip under load, the measured counterpart of the dense peak.
 * Errors: NULL sink/flops -> INVALID_ARG; iterations or blocks < 1 -> SHAPE.
 */
GALORE_API int galore_probe_mfma_bf16(int64_t iterations, int32_t blocks, float* sink, double* flops,
                                      hipStream_t stream);

/*
 * Measurement helper (not part of the method): copies `bytes` from src to dst
 * (device, 16-byte aligned, not overlapping; bytes a multiple of 16) with one
 * 16-byte non-temporal load and store per thread, the access pattern of the
 * element-wise kernels. 2 * bytes divided by the launch time is the measured
 * streaming bandwidth, the counterpart of the HBM peak.
 * Errors: NULL, misaligned or overlapping buffers -> INVALID_ARG; bytes 0 or
 * not a multiple of 16 -> SHAPE.
 */
GALORE_API int galore_probe_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

/* Options of galore_step (bit flags). */
typedef enum {
    GALORE_STEP_ALIGN = 1,      /* after each update but the first, match the new projector's column
                                   signs to the previous projector's (galore_align_projector)        */
    GALORE_STEP_REEXPRESS = 2   /* with ALIGN: also re-express M in the new basis, (P_new^T P_old) M  */
} galore_step_flags_t;

/*
 * Bytes of workspace galore_step needs for `batch` m x n matrices with rank r,
 * oversampling p, gradient storage g_dtype and the given flags. 0 for invalid
 * sizes, dtype or flags.
 */
GALORE_API size_t galore_step_workspace_size(int64_t m, int64_t n, int32_t r, int32_t p, int32_t batch,
                                             int32_t g_dtype, int32_t flags);

/*
 * One GaLore optimizer step on a batch of weight matrices (paper Alg. 1, with
 * the readings of the moment and step-index questions that galore_lowrank_adam_step
 * and galore_align_projector state):
 *   if tau mod T == 0: P <- subspace update of G (galore_rsvd_update with
 *                      seed, sketch_index0, r, p, q); with GALORE_STEP_ALIGN and
 *                      tau > 0 the new P's column signs are matched to the
 *                      previous P, and with GALORE_STEP_REEXPRESS M is replaced
 *                      by (P_new^T P_old) M (V is kept)
 *   R = P^T A; Adam on (M, V) with bias exponent t = tau + 1 gives N;
 *   W <- W - lr * alpha * P N (transposed for m > n)
 * tau >= 0 is the 0-based step index and T >= 1 the update interval; at tau = 0
 * the step must be an update step (tau mod T == 0 always holds there), so P
 * needs no initial value. The kernels and their results are those of the
 * separate entry points called in this order.
 * G: g_dtype m x n (ld ldg, stride stride_g); W: fp32 m x n (ld ldw, stride
 * stride_w), updated in place; P: fp32 s x r (ld ldp, stride stride_p), the
 * projector state, rewritten at update steps; M, V: fp32 r x l (ld ldm >= l,
 * stride stride_m), the moments, updated in place; info: device int32[batch]
 * or NULL, written at update steps (as galore_rsvd_update).
 * Workspace: at least galore_step_workspace_size(...) bytes, device, 256-byte
 * aligned, scratch (holds the projected gradient, the update's workspace and,
 * with the flags, copies of the previous P and M).
 * Streams: as galore_rsvd_update (aux_stream may be NULL).
 * Errors: NULL G/W/P/M/V, bad dtype, tau < 0, T < 1, unknown flags or
 *         REEXPRESS without ALIGN, betas/eps/lr/alpha as galore_lowrank_adam_step
 *         and galore_project_back -> INVALID_ARG; sizes, ld or strides invalid,
 *         r > s, r + p > 4096 -> SHAPE; missing, misaligned or short workspace
 *         -> WORKSPACE.
 */
GALORE_API int galore_step(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg, int64_t stride_g,
                           float* W, int64_t ldw, int64_t stride_w, float* P, int64_t ldp, int64_t stride_p,
                           float* M, float* V, int64_t ldm, int64_t stride_m, int32_t r, int32_t p, int32_t q,
                           uint64_t seed, uint64_t sketch_index0, int64_t tau, int32_t T, float beta1,
                           float beta2, float eps, float lr, float alpha, int32_t flags, int32_t* info,
                           int32_t batch, void* workspace, size_t workspace_bytes, hipStream_t stream,
                           hipStream_t aux_stream);

#ifdef __cplusplus
}
#endif

#endif /* GALORE_H_ */
