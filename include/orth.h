/*
 * orth.h — C ABI of liborth, the MI355X (gfx950) library that turns free
 * parameters into orthogonal matrices and explicit orthogonal convolution
 * kernels, as used by the orthogonal layers of "Orthogonium" (arXiv 2601.13776).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Matrices are row-major with a leading dimension in ELEMENTS.
 * - Data pointers (matrices, kernels, conv inputs, outputs, workspace,
 *   status arrays) are DEVICE pointers owned by the caller.  Descriptor
 *   arrays (orth_mat, orth_conv_desc, orth_check_args) are HOST memory,
 *   read only during the call.
 * - The library never allocates device memory: each entry point that needs
 *   scratch space has a *_workspace_size query; pass at least that many
 *   bytes, 256-byte aligned.  The workspace must not be used by anything
 *   else until the work enqueued by the call has finished.
 * - Every argument is validated on the host before anything is enqueued;
 *   a non-zero return means nothing was launched.  ORTH_EHIP reports a HIP
 *   runtime error at launch time.  Errors inside kernels on well-formed
 *   input cannot occur; degenerate matrices are reported per matrix (see
 *   orth_orthogonalize_batched).
 * - Work is asynchronous on `stream` (a hipStream_t, NULL = the legacy
 *   default stream).  A call's descriptor tables are copied into its
 *   workspace (hipMemcpyAsync on `stream`) from pinned host staging
 *   buffers that the library keeps for the life of the process: a buffer
 *   is reused only once its last copy has completed, and a new one is
 *   allocated (pinned host memory, never device memory) when none is
 *   idle.  The host blocks in one case only: when 64 calls' copies are
 *   still in flight, a call waits for the oldest of them.  Because the
 *   staging buffers are reused, a captured copy would read whatever later
 *   calls left there: every call that copies tables returns
 *   ORTH_EUNSUPPORTED on a capturing stream (HIP graph capture), before
 *   anything is enqueued.  The Björck
 *   entry points may run the small matrices of a batch on side streams
 *   that fork from `stream` and join back into it within the call (event
 *   record and wait; default priority; per calling thread and device,
 *   created on first use and kept until the process ends), so the caller
 *   still sees all of a call's work ordered on `stream`.
 * - bfloat16 is the raw 16-bit pattern (same layout as torch.bfloat16);
 *   conversions to bfloat16 round to nearest, ties to even.
 * - orth_last_error() returns a thread-local message for the last failing
 *   call of the calling thread.
 * - Several host threads may call at once (the plan cache and the staging
 *   pool are shared under locks); calls whose work may overlap on the GPU
 *   need workspaces and outputs of their own.
 */
#ifndef ORTH_H_
#define ORTH_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ORTH_OK = 0,
  ORTH_EINVAL = 1,        /* malformed argument */
  ORTH_EUNSUPPORTED = 2,  /* well-formed but impossible or not implemented */
  ORTH_EWORKSPACE = 3,    /* workspace missing, too small or misaligned */
  ORTH_EHIP = 4           /* HIP runtime error */
} orth_status;

typedef enum { ORTH_F32 = 0, ORTH_BF16 = 1 } orth_dtype;

/* Arithmetic of the Björck products: fp32 operands on fp32 MFMA, or
 * bfloat16 operands with fp32 accumulation (the iterate itself is always
 * kept in fp32). */
typedef enum { ORTH_COMPUTE_F32 = 0, ORTH_COMPUTE_BF16 = 1 } orth_compute;

/* Pre-scaling of W before the iteration: none, W / ||W||_F, or W / sigma
 * with sigma from power iteration on a caller-owned cached vector (see
 * orth_bjorck_opts.power_iters and .u). */
typedef enum { ORTH_PRESCALE_NONE = 0, ORTH_PRESCALE_FROBENIUS = 1, ORTH_PRESCALE_SPECTRAL = 2 } orth_prescale;

/* Per-matrix status written to status_dev. */
typedef enum {
  ORTH_MAT_OK = 0,
  ORTH_MAT_ZERO = 1,       /* Frobenius norm 0: output is all zeros */
  ORTH_MAT_NONFINITE = 2   /* NaN/Inf in the input: output is all NaN */
} orth_mat_status;

/* One matrix to orthogonalize. */
typedef struct {
  const void* in;   /* device, rows x cols, leading dim ld_in, opts.in_dtype */
  void* out;        /* device, rows x cols, leading dim ld_out, opts.out_dtype.
                       May equal `in` (in-place) when dtypes and leading
                       dims agree; otherwise the two must not overlap, and
                       no output may overlap another matrix's input or
                       output (an output can be written during the call). */
  int32_t rows, cols;   /* >= 1 */
  int64_t ld_in, ld_out;
} orth_mat;

typedef struct {
  int32_t iters;      /* number of Björck steps T >= 0 (no early exit) */
  float beta;         /* step size in (0, 0.5]; 0.5 is the usual choice */
  int32_t prescale;   /* orth_prescale */
  int32_t in_dtype;   /* orth_dtype of every mats[i].in */
  int32_t out_dtype;  /* orth_dtype of every mats[i].out */
  int32_t compute;    /* orth_compute */
  /* ORTH_PRESCALE_SPECTRAL only (ignored otherwise): */
  int32_t power_iters;  /* power steps q in [1, 1024] */
  float* u;             /* device, fp32: the cached vectors of all matrices
                           packed in batch order, min(rows, cols) values for
                           each; read, and overwritten with the new estimate
                           (left unchanged for a zero or non-finite matrix) */
  /* bf16 products only (ignored otherwise): tile edge of the matrices with
   * min(rows, cols) >= 1024.  0 chooses by occupancy (256 x 256 tiles when
   * those matrices hold at least 1024 of them, else 128 x 128); 128 or 256
   * forces that size.  The result does not depend on it beyond fp32
   * rounding order. */
  int32_t tile;
  /* orth_orthogonalize_vjp_batched only (must be 0 elsewhere, ignored by
   * orth_orthogonalize_batched): 1 = the workspace holds what a preceding
   * orth_orthogonalize_save_batched call left there for the same inputs,
   * shapes and options, and the forward recomputation is skipped. */
  int32_t saved;
} orth_bjorck_opts;

/*
 * Björck–Bowie orthogonalization of a batch of independent matrices
 * (Appendix A.5 of the paper: W <- (1+beta) W - beta W W^T W, after an
 * optional Frobenius pre-scaling W_0 = W / ||W||_F), exactly opts->iters
 * steps per matrix.  Tall matrices (rows >= cols) get orthonormal columns
 * in the limit, wide ones orthonormal rows.  All matrices of the batch are
 * processed by the same few launches per step, whatever their shapes.
 *
 * Spectral pre-scaling (App. A.5 and Section 2: spectral normalization by
 * batched power iteration, with the estimate of the top singular vector
 * cached across parameter updates): with X the tall orientation of W and
 * v the matrix's cached vector (N = min(rows, cols) values; a zero vector
 * starts as ones), q steps of x = X v, y = X^T x, sigma_hat = |y| / |x|,
 * v = y / |y| (fp64 arithmetic), then W_0 = W / max(sigma_hat,
 * ||W||_F / sqrt(N)) and v is written back.  Both terms are lower bounds of
 * the largest singular value, so W_0's is >= 1; convergence needs it below
 * sqrt(3), which a cached vector from the previous step gives.
 *
 * status_dev: optional device array of n int32 (orth_mat_status).  A zero
 * or non-finite matrix does not fail the call.
 * Workspace: the size depends on the output descriptors as well.  An fp32
 * output laid out as the matrix's fp32 iterate (rows >= cols, both
 * multiples of the tile edge: 64 for fp32 products, 128 or 256 for bf16
 * ones (see tile); ld_out == cols; a 16-byte aligned address) serves as
 * the iterate buffer that the last step writes, so it needs no workspace
 * and is written during the call, not only at its end.  Query the size
 * with the descriptors of the call.
 * Returns ORTH_EINVAL for n < 0, a NULL pointer, rows or cols < 1,
 * ld < cols, iters < 0, beta outside (0, 0.5], an unknown dtype, compute or
 * prescale mode, in == out with differing dtype/leading dim, tile not in
 * {0, 128, 256}, or (spectral) power_iters outside [1, 1024] or u == NULL.
 */
int orth_orthogonalize_workspace_size(const orth_mat* mats, int32_t n,
                                      const orth_bjorck_opts* opts, size_t* bytes);
int orth_orthogonalize_batched(const orth_mat* mats, int32_t n,
                               const orth_bjorck_opts* opts, void* workspace,
                               size_t workspace_bytes, int32_t* status_dev,
                               void* stream);

/*
 * For callers that cannot allocate (tight serving loops, harnesses that
 * forbid hipMalloc): the same
 * orthogonalization as orth_orthogonalize_batched, same arguments and
 * results, with the library's own device scratch in place of the
 * workspace.  The scratch is a fixed array of ORTH_NOALLOC_SCRATCH_BYTES
 * (64 MiB) that each GPU the library runs on holds until the process ends.
 * A batch whose orth_orthogonalize_workspace_size exceeds it fails with
 * ORTH_EWORKSPACE before anything is enqueued.  The call allocates
 * nothing: no device memory, no pinned staging (the descriptor tables are
 * copied from pageable host memory, which HIP may perform synchronously,
 * so the host can wait for earlier work on `stream`), no side streams
 * (every kernel runs on `stream`).  All calls on one GPU share its scratch,
 * which keeps the last call's contents (nothing in it needs to start at
 * zero): calls that overlap on one GPU (other streams or threads without
 * an ordering between them) race and must be serialized by the caller.
 * status_dev as for orth_orthogonalize_batched (NULL: the statuses stay in
 * the scratch).  The call cannot be captured into a HIP graph (its table
 * copies read host memory that lives only during the call): on a capturing
 * stream it returns ORTH_EUNSUPPORTED before anything is enqueued.
 * Errors: those of orth_orthogonalize_batched, ORTH_EWORKSPACE for a batch
 * larger than the scratch, and ORTH_EUNSUPPORTED under stream capture.
 */
#define ORTH_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int orth_orthogonalize_batched_noalloc(const orth_mat* mats, int32_t n,
                                       const orth_bjorck_opts* opts,
                                       int32_t* status_dev, void* stream);

/* One matrix of a Björck vector-Jacobian product. */
typedef struct {
  const void* w;         /* device, the raw parameter W the forward call was
                            given: rows x cols, leading dim ld_w, opts.in_dtype */
  const void* grad_out;  /* device, dL/d(output of the forward call), rows x
                            cols, leading dim ld_grad_out, opts.out_dtype */
  void* grad_in;         /* device, dL/dW, rows x cols, leading dim ld_grad_in,
                            opts.in_dtype.  May equal grad_out (equal dtypes
                            and leading dims) or w (equal leading dims);
                            otherwise it must not overlap either. */
  int32_t rows, cols;    /* >= 1 */
  int64_t ld_w, ld_grad_out, ld_grad_in;
} orth_vjp_mat;

/*
 * Vector-Jacobian product of orth_orthogonalize_batched: for every matrix,
 * dL/dW given dL/d(output), for the same opts (iters, beta, prescale,
 * compute).  Derivative of the Appendix A.5 step for tall X with upstream
 * gradient Y:
 *   dL/dX = Y + beta (Y E - X S),  E = I - X^T X,  S = X^T Y + Y^T X
 * (wide matrices through their transpose), chained from the last step to
 * the first, then through the pre-scaling W_0 = W / ||W||_F:
 *   dL/dW = (dL/dW_0 - <dL/dW_0, W_0> W_0) / ||W||_F.
 * Spectral pre-scaling (App. A.5; the estimate W_0 = W / sigma with sigma =
 * max(sigma_hat, ||W||_F / sqrt(N)) of orth_orthogonalize_batched): the
 * cached vector is state, not a function of W, and is held constant; with
 * G_0 = dL/dX_0 (tall orientation) and c = -<G_0, X_0> / sigma,
 *   floor branch:  dL/dX = G_0 / sigma + c X / (||X||_F sqrt(N)),
 *   power branch:  dL/dX = G_0 / sigma + the 2q rank-1 terms of the chain
 *                  rule through the q power steps (each step's vectors
 *                  depend on W; only the starting vector is constant).
 * opts.u then holds the cached vectors as the differentiated forward call
 * found them (before it wrote its new estimates back); they are read, never
 * written.  With opts.saved = 1 they are not read: the saving forward kept
 * the power steps and a copy of its starting vectors in the workspace.
 * power_iters may be at most 16 here (the workspace keeps every step's
 * vectors and the backward adds 2q rank-1 terms to every element).
 * The forward iterates are recomputed inside the call (or, with
 * opts.saved = 1, taken from a saving forward, see below) and every X_t and
 * E_t is kept in the workspace (about T (M N + N^2) elements per M x N
 * matrix, in fp32 or bf16 per opts.compute), so the workspace query grows
 * with T.
 * Matrices with N <= 64 and M <= 128 (tall orientation) use fp32 products
 * whatever opts.compute says, as the forward does.
 *
 * status_dev: optional, as for the forward (1: zero matrix -> zero gradient;
 * 2: non-finite input -> NaN gradient).
 * Returns ORTH_EINVAL for the argument errors of the forward call (u may
 * be NULL with opts.saved = 1), iters > 4096, or aliasing other than the
 * two allowed above; ORTH_EUNSUPPORTED for spectral pre-scaling with more
 * than 16 power steps.
 */
int orth_orthogonalize_vjp_workspace_size(const orth_vjp_mat* mats, int32_t n,
                                          const orth_bjorck_opts* opts, size_t* bytes);
int orth_orthogonalize_vjp_batched(const orth_vjp_mat* mats, int32_t n,
                                   const orth_bjorck_opts* opts, void* workspace,
                                   size_t workspace_bytes, int32_t* status_dev,
                                   void* stream);

/*
 * The forward of orth_orthogonalize_batched (Appendix A.5 steps, same
 * options and results up to fp32 rounding order) that keeps, in a
 * vector-Jacobian workspace, every X_t and E_t that the product above needs
 * (the training pattern: a forward that saves, a backward that reuses).  A
 * later orth_orthogonalize_vjp_batched call with opts.saved = 1, this
 * workspace, the same inputs (unchanged) and the same shapes and options
 * then skips its forward recomputation (about a third of its work); several
 * such calls may reuse one saving forward.  The workspace size is that of
 * orth_orthogonalize_vjp_workspace_size for matrices of the same shapes
 * (orth_orthogonalize_save_workspace_size gives it from these descriptors)
 * and holds the saved state until the caller reuses it.
 * Spectral pre-scaling: the cached vectors are read and the new estimates
 * written back as by orth_orthogonalize_batched; the vectors this call
 * started from are copied into the workspace for the saved product.
 * Errors: those of orth_orthogonalize_vjp_batched for these options
 * (ORTH_EUNSUPPORTED for spectral pre-scaling with more than 16 power
 * steps), ORTH_EINVAL for in == out (the product reads the input again) or
 * opts.saved != 0.
 */
int orth_orthogonalize_save_workspace_size(const orth_mat* mats, int32_t n,
                                           const orth_bjorck_opts* opts, size_t* bytes);
int orth_orthogonalize_save_batched(const orth_mat* mats, int32_t n,
                                    const orth_bjorck_opts* opts, void* workspace,
                                    size_t workspace_bytes, int32_t* status_dev,
                                    void* stream);

/* Options of the exponential map. */
typedef struct {
  int32_t terms;        /* p in [1, 64]: the series is truncated after Ahat^p / p! */
  int32_t power_iters;  /* power steps q in [1, 1024] of the spectral normalization */
  float* u;             /* device, fp32: cached vectors, C values per matrix packed in
                           batch order; read and overwritten with the new estimate */
  int32_t in_dtype;     /* orth_dtype of every mats[i].in */
  int32_t out_dtype;    /* orth_dtype of every mats[i].out */
} orth_exp_opts;

/*
 * Exponential map with spectral normalization (Appendix A.3, algorithm
 * "Exponential Map with Spectral Normalization"): for every square C x C
 * matrix W, A = W - W^T, Ahat = A / sigma, and
 *     What = I + sum_{k=1}^{p} P_k,   P_k = P_{k-1} Ahat / k,  P_0 = I,
 * an element of SO(C) up to the truncation error |Ahat|^(p+1) e^|Ahat| / (p+1)!.
 * sigma is the spectral-normalization estimate of orth_orthogonalize_batched's
 * ORTH_PRESCALE_SPECTRAL applied to A (power iteration from the cached
 * vector, at least ||A||_F / sqrt(C)).  fp32 products; a symmetric W (A = 0)
 * gives I and status 1 with its vector unchanged; a non-finite W gives NaN
 * and status 2.  Returns ORTH_EINVAL for non-square or NULL matrices, in ==
 * out, terms outside [1, 64], power_iters outside [1, 1024], u == NULL or
 * an unknown dtype.
 */
int orth_exp_map_workspace_size(const orth_mat* mats, int32_t n, const orth_exp_opts* opts,
                                size_t* bytes);
int orth_exp_map_batched(const orth_mat* mats, int32_t n, const orth_exp_opts* opts,
                         void* workspace, size_t workspace_bytes, int32_t* status_dev,
                         void* stream);

/* One explicit conv exponential. */
typedef struct {
  int32_t channels;     /* c: the kernel maps c channels to c channels */
  int32_t k;            /* odd kernel size, <= 15 */
  int32_t terms;        /* p in [1, 32] */
  float scale;          /* t: the exponential of t (K - K*) */
  const void* kernel;   /* device: K, c x c x k x k (OIHW), contiguous */
  void* out;            /* device: c x c x S x S, S = p (k - 1) + 1, contiguous */
} orth_conv_exp_desc;

/*
 * Explicit exponential of a skew-symmetric convolution (Appendix B.2,
 * theorem "Explicit conv exponential", the Adaptive-SOC layer): with
 * K*[o, i, a, b] = K[i, o, k-1-a, k-1-b] (the kernel of the adjoint of a
 * stride-1 circular conv with centred padding) and L = t (K - K*),
 *     E = sum_{j=0}^{p} L^(⊛j) / j!,
 * ⊛ the block-convolution operator, L^(⊛0) the identity, every term centred
 * in the S x S output.  conv(E, .) equals the per-input series
 * sum_j conv(L, .)^j / j!, so one convolution replaces p.  dtype is the
 * storage of kernel and out; arithmetic is fp32.  Returns ORTH_EINVAL for
 * NULL pointers, kernel == out, channels outside [1, 8192], terms outside
 * [1, 32], a non-finite scale or an unknown dtype; ORTH_EUNSUPPORTED for
 * an even kernel size (no centre) or k > 15.
 */
int orth_conv_exp_workspace_size(const orth_conv_exp_desc* descs, int32_t n, int32_t dtype,
                                 size_t* bytes);
int orth_conv_exp_batched(const orth_conv_exp_desc* descs, int32_t n, int32_t dtype,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Geometry of one orthogonal convolution (groups g, stride s, dilation d). */
typedef struct {
  int32_t cin, cout, k, stride, dilation, groups;
} orth_conv_geom;

/*
 * Shapes of the free parameters of one AOC layer (Appendix B.1: the kernel
 * is RKO composed with BCOP blocks; valid iff k >= stride).  Per group:
 * one RKO matrix of rko_rows x rko_cols = (cout/g) x (cin/g * s^2) and
 * n_proj = 2 (k - s) projector factors of proj_rows x proj_cols =
 * (cin/g) x floor(cin/g / 2).  Host only; launches nothing.
 * Returns ORTH_EINVAL for non-positive sizes or groups not dividing cin and
 * cout, ORTH_EUNSUPPORTED for k < s, s > 1 with gcd(s, d) != 1, or fewer
 * than 2 channels per group when k > s.
 */
int orth_aoc_param_shapes(const orth_conv_geom* geom, int32_t* rko_rows,
                          int32_t* rko_cols, int32_t* n_proj,
                          int32_t* proj_rows, int32_t* proj_cols);

/* One conv layer to build. */
typedef struct {
  orth_conv_geom geom;
  const void* rko;   /* device: g x rko_rows x rko_cols, contiguous, orthogonalized */
  const void* proj;  /* device: g x n_proj x proj_rows x proj_cols, contiguous,
                        orthogonalized; horizontal 1x2 blocks first, then the
                        vertical 2x1 blocks.  Ignored (may be NULL) if n_proj == 0. */
  void* kernel;      /* device: cout x (cin/g) x k x k (OIHW), contiguous */
} orth_conv_desc;

/*
 * Explicit AOC kernels (Appendix B.1, AOC = RKO ⊛ K_BCOP, with native
 * stride, groups and dilation).  For every group, the s x s RKO kernel
 * R[o, i, a, b] = M[o, i s^2 + a s + b] is composed with k - s horizontal
 * blocks (taps P, I - P) and k - s vertical blocks (taps Q, I - Q), where
 * P = V V^T for each projector factor V, by the block-convolution operator
 * (the kernel of the composition of two convolutions).  Group j fills
 * output channels [j cout/g, (j+1) cout/g).  Dilation does not change the
 * kernel; it is only validated.  `dtype` is the storage type of rko, proj
 * and kernel; arithmetic is fp32.  Errors as orth_aoc_param_shapes, plus
 * ORTH_EINVAL for NULL pointers or n < 0.
 */
int orth_build_conv_kernels_workspace_size(const orth_conv_desc* descs, int32_t n,
                                           int32_t dtype, size_t* bytes);
int orth_build_conv_kernels_batched(const orth_conv_desc* descs, int32_t n,
                                    int32_t dtype, void* workspace,
                                    size_t workspace_bytes, void* stream);
/* One conv layer of a composition vector-Jacobian product. */
typedef struct {
  orth_conv_geom geom;
  const void* rko;          /* device: the forward call's rko (orthogonalized factors) */
  const void* proj;         /* device: the forward call's proj (may be NULL if n_proj == 0) */
  const void* grad_kernel;  /* device: dL/dK, cout x (cin/g) x k x k (OIHW), contiguous */
  void* grad_rko;           /* device: dL/d rko, g x rko_rows x rko_cols, contiguous */
  void* grad_proj;          /* device: dL/d proj, g x n_proj x proj_rows x proj_cols,
                               contiguous (ignored, may be NULL, if n_proj == 0) */
} orth_conv_vjp_desc;

/*
 * Vector-Jacobian product of orth_build_conv_kernels_batched with respect to
 * the factors: given dL/dK, the gradients with respect to the (already
 * orthogonalized) RKO matrix and projector factors of every group.  Each ⊛
 * step with a block of taps P, I - P is bilinear, so its adjoint sends the
 * kernel gradient G to dT[a][b] = G[a][b] P + G[next] (I - P) and gives
 * dP = sum_taps T^T (G[a][b] - G[next]), with "next" the neighbouring tap
 * along the block's direction; P = V V^T gives dV = (dP + dP^T) V.  The
 * forward taps are recomputed inside the call (see the saving composition
 * below for the alternative).  Chain with
 * orth_orthogonalize_vjp_batched for the gradient with respect to the raw
 * parameters.  dtype is the storage type of every tensor; arithmetic is fp32.
 * Errors as orth_build_conv_kernels_batched.  grad_* must not overlap the
 * inputs.
 */
int orth_build_conv_kernels_vjp_workspace_size(const orth_conv_vjp_desc* descs, int32_t n,
                                               int32_t dtype, size_t* bytes);
int orth_build_conv_kernels_vjp_batched(const orth_conv_vjp_desc* descs, int32_t n,
                                        int32_t dtype, void* workspace,
                                        size_t workspace_bytes, void* stream);

/*
 * The composition of orth_build_conv_kernels_batched (Appendix B.1, same
 * kernels up to fp32 rounding order) that leaves, in a composition-VJP
 * workspace, the projectors and the input tap grid of every block step, so
 * that orth_build_conv_kernels_vjp_saved_batched (the product above without
 * its forward recomputation) can follow for the same layers, factors
 * (unchanged) and dtype, as often as needed.  The workspace size is that of
 * orth_build_conv_kernels_vjp_workspace_size for the same geometries
 * (orth_build_conv_kernels_save_workspace_size gives it from these
 * descriptors).  Errors as orth_build_conv_kernels_batched.
 */
int orth_build_conv_kernels_save_workspace_size(const orth_conv_desc* descs, int32_t n,
                                                int32_t dtype, size_t* bytes);
int orth_build_conv_kernels_save_batched(const orth_conv_desc* descs, int32_t n,
                                         int32_t dtype, void* workspace,
                                         size_t workspace_bytes, void* stream);
int orth_build_conv_kernels_vjp_saved_batched(const orth_conv_vjp_desc* descs, int32_t n,
                                              int32_t dtype, void* workspace,
                                              size_t workspace_bytes, void* stream);

/* Application of an explicit kernel (forward or transposed convolution). */
typedef struct {
  orth_conv_geom geom;     /* geometry of the FORWARD conv (cin -> cout, stride s) */
  const void* kernel;      /* device: cout x (cin/g) x k x k (OIHW), kernel_dtype */
  int32_t kernel_dtype;    /* orth_dtype */
  int32_t transposed;      /* 0: y = conv(K, x); 1: y = conv^T(K, x) */
  const float* x;          /* device fp32 NCHW: batch x cin x H x W (forward) or
                              batch x cout x H/s x W/s (transposed) */
  float* y;                /* device fp32 NCHW: batch x cout x H/s x W/s (forward)
                              or batch x cin x H x W (transposed); must not
                              overlap x */
  int32_t batch, height, width;   /* H, W: the forward conv's input grid */
} orth_conv_apply_args;

/*
 * Circular-padded convolution with an explicit kernel, natively strided,
 * dilated and grouped, or its transpose (Section 3: an AOC layer runs as one
 * convolution with the materialized kernel; transposed convolutions reuse
 * the same kernel for learnable upsampling).  Forward:
 *   y[b,o,u,v] = sum_{i,a,e} K[o,i,a,e] x[b, g(o) c + i, (s u + d a - pl) mod H, (s v + d e - pl) mod W],
 * c = cin/g, pl = floor((d (k-1) + 1 - s) / 2); transposed: the adjoint of
 * that map.  For an orthogonal kernel with cout/g <= c s^2 the forward map
 * has orthonormal rows, so the transposed map preserves norms and the
 * forward map inverts it.  fp32 arithmetic on fp32 MFMA.
 * Errors: the geometry errors of orth_aoc_param_shapes, ORTH_EINVAL for
 * NULL pointers, batch/height/width < 1, H or W not divisible by the
 * stride, x == y, or an unknown dtype.
 */
int orth_conv_apply(const orth_conv_apply_args* args, void* stream);

/* Single-layer convenience form of orth_build_conv_kernels_batched. */
int orth_build_conv_kernel(const void* rko, const void* proj, int32_t cin,
                           int32_t cout, int32_t k, int32_t stride,
                           int32_t dilation, int32_t groups, int32_t dtype,
                           void* kernel_out, void* workspace,
                           size_t workspace_bytes, void* stream);

typedef enum {
  ORTH_CHECK_GRAM = 0,          /* out[i] = max |G_i - I|, G the smaller Gram of mats[i].in */
  ORTH_CHECK_CONV = 1,          /* out[b] = ||conv(K, x_b)|| / ||x_b|| */
  ORTH_CHECK_CONV_ADJOINT = 2   /* out[b] = ||conv^T(K, x_b)|| / ||x_b|| */
} orth_check_mode;

/*
 * Verification quantities (Section 4 and Appendix C: orthogonality of
 * matrices, norm preservation of the circular-padded convolution).
 * CONV: x is batch x cin x height x width fp32; the convolution is the
 * circular-padded cross-correlation with stride s and dilation d, total
 * padding d (k - 1) + 1 - s split floor/ceil, output (height/s, width/s).
 * CONV_ADJOINT: x is batch x cout x height x width on the OUTPUT grid and
 * the transpose maps it to cin x (height s) x (width s).
 * height and width must be divisible by s (CONV).
 */
typedef struct {
  int32_t mode;             /* orth_check_mode */
  /* GRAM */
  const orth_mat* mats;     /* reads mats[i].in, rows, cols, ld_in */
  int32_t n_mats;
  int32_t mat_dtype;
  /* CONV / CONV_ADJOINT */
  const void* kernel;       /* cout x (cin/g) x k x k */
  int32_t kernel_dtype;
  orth_conv_geom geom;
  const float* x;
  int32_t batch, height, width;
} orth_check_args;

int orth_check_workspace_size(const orth_check_args* args, size_t* bytes);
int orth_check_norm(const orth_check_args* args, float* out_dev, void* workspace,
                    size_t workspace_bytes, void* stream);

/* Diagnostics. */
const char* orth_status_string(int status);
const char* orth_last_error(void);
int32_t orth_version(void);

/*
 * Per-kernel timing with HIP events recorded around every launch on the
 * launch stream (off by default; process-wide: the launches of every thread
 * and stream count together, each timed by two events on its own stream).
 * orth_timing_read synchronizes the recorded events and returns the total
 * milliseconds and launch count of the named kernel since the last reset.
 * orth_timing_span returns the wall-clock milliseconds covered by the
 * launches whose kernel name starts with one of the ';'-separated
 * prefixes (the union of their intervals: launches that overlap on
 * several streams count once) and their number, since the last reset.
 * orth_timing_names writes a ';'-separated list of the kernel names seen.
 * orth_timing_filter limits the timing to launches whose kernel name starts
 * with one of the ';'-separated prefixes (NULL or "": every launch); each
 * timed launch adds two event records to its stream (a few microseconds).
 */
int orth_timing_enable(int32_t on);
int orth_timing_filter(const char* prefixes);
int orth_timing_reset(void);
int orth_timing_read(const char* kernel_name, double* total_ms, int64_t* launches);
int orth_timing_span(const char* prefixes, double* covered_ms, int64_t* launches);
int orth_timing_names(char* buf, size_t buf_bytes);

#ifdef __cplusplus
}
#endif

#endif /* ORTH_H_ */
