/*
 * oaa.h - overlap-and-add (OaA) FFT convolution of one CNN layer on gfx950.
 *
 * The operation is that of T. Highlander and A. Rodriguez, "Very Efficient
 * Training of Convolutional Neural Networks using Fast Fourier Transform and
 * Overlap-and-Add", arXiv:1601.06815:
 *
 *   - Problem (Introduction; Section 3.2): an input of C channels, each N x N,
 *     and K kernels of C channels, each n x n; every kernel channel is
 *     convolved with its input channel and the C results are summed (K*C 2-D
 *     convolutions per layer).
 *   - Method (Section 2): each N x N plane is cut into ceil(N/n)^2 blocks of
 *     n x n, block and kernel are zero-padded (to 2n-1 per side, rounded up to
 *     a power of two, Sections 3.2-3.3) and transformed, multiplied bin by bin,
 *     transformed back, and the (2n-1)^2 block results are overlapped by n-1
 *     and added.
 *   - Backward (Section 3.2): two convolutions, one propagating the error
 *     through the layer (oaa_conv_backward_data), one forming the weight
 *     change (oaa_conv_backward_filter).
 *
 * Definitions computed (all tensors row-major NCHW float32, M = N - n + 1):
 *
 *   forward:          y[b,k,i,j]  = sum_c sum_{u,v<n} w[k,c,u,v] x[b,c,i+n-1-u,j+n-1-v]
 *   backward_data:    dx[b,c,p,q] = sum_k sum_{u,v<n} w[k,c,u,v] g[b,k,p-n+1+u,q-n+1+v]
 *                                   (g taken as 0 outside [0,M)^2)
 *   backward_filter:  dw[k,c,u,v] = sum_b sum_{i,j<M} g[b,k,i,j] x[b,c,i+n-1-u,j+n-1-v]
 *
 * i.e. a true convolution (kernel flipped; a cross-correlation layer passes
 * w flipped in both spatial axes), valid output, stride 1, and the exact
 * derivatives of <y, g> with respect to x and w. Outputs are overwritten.
 *
 * Memory and streams: every tensor pointer is a DEVICE pointer owned by the
 * caller; the plan owns only a small host structure. All intermediate
 * spectra live in a caller-allocated device workspace bound with
 * oaa_plan_bind_workspace. Compute calls only enqueue work on the given HIP
 * stream (NULL = the null stream) and return without synchronising. A plan is
 * used from one stream at a time and is not thread-safe; distinct plans are
 * independent. Inputs must not alias outputs or the workspace.
 *
 * Errors: every call returns a status. Arguments are validated before any
 * work is enqueued, so a non-OK status from validation means nothing ran.
 * OAA_ERR_HIP reports a launch failure; oaa_last_error_detail() gives a
 * thread-local human-readable reason for the last non-OK status.
 */
#ifndef OAA_H_
#define OAA_H_

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct oaa_plan_s* oaa_plan_t;

typedef enum {
  OAA_OK = 0,
  OAA_ERR_INVALID_ARG = 1,   /* bad dimension, NULL pointer, unknown enum   */
  OAA_ERR_UNSUPPORTED = 2,   /* valid but outside this library (n > 64)      */
  OAA_ERR_NO_WORKSPACE = 3,  /* no workspace bound, or the one bound is too small */
  OAA_ERR_NO_CACHE = 4,      /* a NULL input asks for a spectrum not yet computed */
  OAA_ERR_HIP = 5            /* the HIP runtime reported an error             */
} oaa_status_t;

/* Sizes derived from (B, C, K, N, n) and the tiling (L, b). */
typedef struct {
  int B, C, K, N, n;
  int M;      /* output side, N - n + 1                                      */
  int T;      /* blocks per side: ceil(N / b), or ceil(M / b) for overlap-save */
  int P;      /* blocks per plane, T * T                                     */
  int L;      /* transform side (oaa_plan_create: smallest power of two
                 >= 2n - 1, at least 2)                                      */
  int F;      /* stored frequency bins per tile, L * (L/2 + 1)               */
  int split;  /* partial sums of the weight-gradient contraction             */
  int b;      /* block pitch: blocks are b x b (oaa_plan_create: b = n)      */
  int method; /* oaa_method_t of the plan                                    */
  int fused;  /* 1 if the passes run fused (OAA_CONTRACTION_FUSED), else 0   */
} oaa_geometry_t;

/* How the passes are tiled (oaa_plan_create_method).
 *
 * OAA_METHOD_OVERLAP_ADD: the paper's method (Section 2). The forward pass
 *   cuts x into b x b blocks, T = ceil(N / b) per side, and overlap-adds the
 *   block results; the backward passes read g in windows of side up to 2b
 *   that start every b (the adjoint of the overlap-add).
 * OAA_METHOD_OVERLAP_SAVE: the alternative the paper names beside OaA
 *   (Introduction), every pass tiled by the output side M with hop
 *   h = L - n + 1 (reported as b), T = ceil(M / h) per side. The forward pass
 *   transforms L x L windows of x starting every h and keeps rows and columns
 *   [n-1, L) of each inverse (overlap-and-save); the error propagation cuts g
 *   into h x h blocks and overlap-adds their results into dx (OaA applied to
 *   that convolution); the weight gradient pairs the same windows and blocks.
 *   The X and G regions then hold window and block spectra respectively. */
typedef enum {
  OAA_METHOD_OVERLAP_ADD = 0,
  OAA_METHOD_OVERLAP_SAVE = 1
} oaa_method_t;

/* Workspace regions (see oaa_plan_region). Every spectrum is complex64
 * (re, im interleaved) and bin-major: bin f = u * (L/2 + 1) + v holds row
 * frequency u in [0, L) and column frequency v in [0, L/2], the Hermitian half
 * of a real L x L transform X[u][v] = sum_{r,s} t[r][s] exp(-2 pi i (ur+vs)/L).
 * Tile t of image b is b * P + P_row * T + Q_col. */
typedef enum {
  OAA_REGION_W_SPECTRUM = 0, /* [F][C][K]        kernel spectra                 */
  OAA_REGION_X_SPECTRUM = 1, /* [F][C][B*P]      input block spectra            */
  OAA_REGION_G_SPECTRUM = 2, /* [F][K][B*P]      upstream-gradient window spectra */
  OAA_REGION_PRODUCT = 3     /* after forward: [F][K][B*P] output spectra;
                                after backward_data: [F][C][B*P];
                                after backward_filter: [split][F][C][K] partial sums.
                                Bins (u, v) with u > L/2 and v in {0, L/2} are
                                the conjugates of bins (L-u, v), the spectra
                                being Hermitian there. Nothing reads them: they
                                are never written here, and the X and G
                                regions may omit them too.
                              With the fused passes (OAA_CONTRACTION_FUSED) the layouts
                              differ: W holds the kernels' bins contiguous
                              ([K][C][F]); X runs of a block row
                              ([B*T][C][F][T], block (P, Q) of image b in run b*T + P at
                              position Q); G and the forward product are never stored;
                              PRODUCT holds only the weight-gradient partial sums,
                              [split][F][C][K]. */
} oaa_region_t;

/* Contraction implementation (the per-bin complex matrix product). */
typedef enum {
  OAA_CONTRACTION_AUTO = 0,  /* library's choice by shape                        */
  OAA_CONTRACTION_VALU = 1,  /* LDS-tiled FMA on the vector ALUs                 */
  OAA_CONTRACTION_MFMA = 2,  /* fp32 matrix cores                                */
  OAA_CONTRACTION_NARROW = 3, /* streaming, for C <= 4 input channels only      */
  OAA_CONTRACTION_FUSED = 4   /* the contraction inside the transform kernels, so
                                 that the product spectra (forward) and the
                                 gradient window spectra (both backward passes)
                                 are never stored: overlap-add plans with L = 64,
                                 C <= 4 and T <= 8 (the library's choice there
                                 when B T^2 >= 512)                            */
} oaa_contraction_t;

/* Stages of the three passes, for per-stage timing. */
typedef enum {
  OAA_STAGE_W_SPECTRUM = 0,       /* kernel zero-pad + transform                   */
  OAA_STAGE_X_SPECTRUM = 1,       /* input block division + zero-pad + transform   */
  OAA_STAGE_G_SPECTRUM = 2,       /* gradient windows + zero-pad + transform       */
  OAA_STAGE_FWD_PRODUCT = 3,      /* forward per-bin contraction over C            */
  OAA_STAGE_FWD_INVERSE = 4,      /* inverse transform + overlap-add + valid crop  */
  OAA_STAGE_BWD_DATA_PRODUCT = 5, /* per-bin contraction over K with conj kernels  */
  OAA_STAGE_BWD_DATA_INVERSE = 6, /* inverse transform + block crop                */
  OAA_STAGE_BWD_FILTER_PRODUCT = 7, /* per-bin contraction over B and blocks       */
  OAA_STAGE_BWD_FILTER_INVERSE = 8, /* partial-sum reduce + inverse + crop         */
  OAA_STAGE_COUNT = 9
} oaa_stage_t;

/* Create a plan for x[B,C,N,N] and w[K,C,n,n] with the paper's tiling
 * (Section 2: blocks of the kernel's size, b = n; transform side L the
 * smallest power of two >= 2n - 1, Sections 3.2-3.3). Host-only: makes no
 * HIP call and allocates no device memory. Requires B, C, K >= 1 and
 * 1 <= n <= N (else OAA_ERR_INVALID_ARG); n <= 64 (transform sides up to
 * 128) and element counts within 2^31 blocks per spectrum row (else
 * OAA_ERR_UNSUPPORTED). On success *plan
 * is set; on failure *plan is set to NULL. */
oaa_status_t oaa_plan_create(oaa_plan_t* plan, int B, int C, int K, int N, int n);

/* Same, with blocks of b x b (pitch b) in L x L transforms. Block results
 * then have support b + n - 1 and the result is the same convolution for any
 * b with max(1, n-1) <= b <= L - n + 1 (up to L/2 the forward overlap-add is
 * done on the spectra; above, after the inverse). L must be a power of two
 * in [2, 128] (else OAA_ERR_UNSUPPORTED); a b outside that range is
 * OAA_ERR_INVALID_ARG.
 * L = b = 0 lets the library choose: L from L0 (the paper's side) up to 64,
 * or L0 = 128, and b, by an estimate of the step time of contractions and
 * transforms. Larger blocks mean fewer tiles: fewer spectra to transform,
 * store and contract. */
oaa_status_t oaa_plan_create_tiled(oaa_plan_t* plan, int B, int C, int K, int N, int n, int L, int b);

/* Same, with a choice of method (oaa_method_t). For OAA_METHOD_OVERLAP_ADD
 * this is oaa_plan_create_tiled. For OAA_METHOD_OVERLAP_SAVE, L is a power of
 * two in [max(2, 2n-1 rounded up), 128], or 0 for the library's choice between
 * that side and twice it; b must be 0 or L - n + 1 (the hop). An unknown
 * method is OAA_ERR_INVALID_ARG. */
oaa_status_t oaa_plan_create_method(oaa_plan_t* plan, int B, int C, int K, int N, int n, int L, int b,
                                    oaa_method_t method);

/* Release the host structure (and any timing events). NULL is a no-op.
 * Does not free the workspace. */
oaa_status_t oaa_plan_destroy(oaa_plan_t plan);

/* Copy the plan's derived sizes into *out. */
oaa_status_t oaa_plan_geometry(oaa_plan_t plan, oaa_geometry_t* out);

/* Device workspace the plan needs, in bytes (0 for a NULL plan): the four
 * regions below and, for L = 128 planes of several tiles per side, a scratch
 * after them that holds the real tile results of the overlap-add. */
size_t oaa_plan_workspace_bytes(oaa_plan_t plan);

/* Byte offset and size of one workspace region (layouts above). */
oaa_status_t oaa_plan_region(oaa_plan_t plan, oaa_region_t region, size_t* offset, size_t* bytes);

/* Bind caller-owned device memory of at least oaa_plan_workspace_bytes()
 * bytes, 256-byte aligned. Binding (or re-binding) discards cached spectra.
 * The memory must stay allocated while calls that use it are in flight. */
oaa_status_t oaa_plan_bind_workspace(oaa_plan_t plan, void* dev_ptr, size_t bytes);

/* Choose the contraction implementation for later calls. OAA_CONTRACTION_FUSED
 * on a plan that cannot take it is OAA_ERR_UNSUPPORTED. Switching between the
 * fused and the unfused passes discards the cached spectra (their layouts
 * differ). */
oaa_status_t oaa_plan_set_contraction(oaa_plan_t plan, oaa_contraction_t which);

/* Per-stage timing (the stage breakdown of Section 3.2's overhead
 * measurement). enable != 0: every later kernel launch is bracketed by two HIP
 * events recorded on the call's stream (a HIP call; events are created on
 * first use and released by oaa_plan_destroy). enable == 0 stops recording. */
oaa_status_t oaa_plan_set_timing(oaa_plan_t plan, int enable);

/* Wait for every recorded launch to finish, then add its duration (ms) into
 * total_ms[stage] and 1 into launches[stage] for stage < count (both arrays
 * are zeroed first), and forget the records. Either array may be NULL. */
oaa_status_t oaa_plan_stage_times(oaa_plan_t plan, double* total_ms, int* launches, int count);

/* Forward pass (Section 2): y[B,K,M,M] from x[B,C,N,N] and w[K,C,n,n].
 * w == NULL reuses the kernel spectra of the last call that computed them
 * (OAA_ERR_NO_CACHE if none). Leaves the input block spectra in the
 * workspace for a later backward_filter with x == NULL. */
oaa_status_t oaa_conv_forward(oaa_plan_t plan, const float* x, const float* w, float* y,
                              void* hip_stream);

/* Error propagation (Section 3.2): dx[B,C,N,N] from g[B,K,M,M] and
 * w[K,C,n,n]. w == NULL reuses the cached kernel spectra. Leaves the window
 * spectra of g in the workspace for a later backward_filter with g == NULL. */
oaa_status_t oaa_conv_backward_data(oaa_plan_t plan, const float* g, const float* w, float* dx,
                                    void* hip_stream);

/* Weight gradient (Section 3.2): dw[K,C,n,n] from x[B,C,N,N] and
 * g[B,K,M,M]. x == NULL reuses the block spectra of the last forward (or
 * backward_filter) call; g == NULL reuses the window spectra of the last
 * backward_data (or backward_filter) call. The fused passes keep no gradient
 * spectra: with them g == NULL is OAA_ERR_NO_CACHE. */
oaa_status_t oaa_conv_backward_filter(oaa_plan_t plan, const float* x, const float* g, float* dw,
                                      void* hip_stream);

/* Two stacked convolution layers with nothing between them, x -> conv(., w1)
 * -> conv(., w2), composed in the frequency domain (Conclusion: convolution
 * layers as products in the frequency domain, with no transform between
 * them). conv(conv(x, w1), w2) = conv(x, w12), where w12[k][c] = sum_j
 * w2[k][j] * w1[j][c] (full 2-D convolutions, side n1 + n2 - 1); its
 * spectrum is, bin by bin, W12[c][k] = sum_j W1[c][j] W2[j][k]. This call
 * transforms w1 and w2 at the plan's L, forms that product on the device and
 * stores it as the plan's cached kernel spectra, so that
 * oaa_conv_forward(plan, x, NULL, y) computes both layers, valid, without
 * the intermediate activation ever leaving the frequency domain, and
 * oaa_conv_backward_data(plan, g, NULL, dx) the gradient with respect to x
 * through both. (backward_filter then gives the gradient of the composite
 * kernel w12, not of w1 and w2.)
 *   - plan: bound workspace; C = w1's input channels, K = w2's output
 *     channels, n = n1 + n2 - 1 (else OAA_ERR_INVALID_ARG); not running the
 *     fused passes (their kernel spectra have another layout; else
 *     OAA_ERR_UNSUPPORTED: choose another contraction first).
 *   - w1: device, [J][C][n1][n1] fp32; w2: device, [K][J][n2][n2] fp32;
 *     J, n1, n2 >= 1.
 *   - scratch: device memory of at least oaa_plan_chain_scratch_bytes(plan,
 *     J) bytes, 256-byte aligned, owned by the caller, for the two layers'
 *     spectra; free to reuse once the call's work on `stream` is done.
 *   - stream: as for the passes. Validation happens before any launch.
 * Later oaa_conv_forward / backward_data calls with w == NULL use the
 * composed spectra until a call with w != NULL, a contraction switch or a
 * workspace bind replaces or discards them. */
size_t oaa_plan_chain_scratch_bytes(oaa_plan_t plan, int J);
oaa_status_t oaa_plan_set_kernel_chain(oaa_plan_t plan, const float* w1, int J, int n1, const float* w2, int n2,
                                       void* scratch, size_t scratch_bytes, void* hip_stream);

/* Forward pass without device allocation, for callers that cannot allocate:
 * code being captured into a HIP graph, tight serving loops, harnesses that
 * forbid hipMalloc. Same result as oaa_conv_forward(plan, x, w, y, stream)
 * (the same kernels), but the spectra live in a static scratch array inside
 * the library (64 MiB on each device, held until the process ends) instead
 * of the plan's bound workspace, so no workspace need be bound.
 *   - plan: a plan whose oaa_plan_workspace_bytes() is at most 64 MiB, else
 *     OAA_ERR_UNSUPPORTED before anything is enqueued.
 *   - x, w, y: device pointers as for oaa_conv_forward, all non-NULL
 *     (OAA_ERR_INVALID_ARG otherwise): no cached spectra are read, and none
 *     are recorded for later NULL arguments (the plan's own cache and
 *     workspace are left untouched).
 *   - stream: a stream of the current device (NULL = its null stream).
 * Makes no hipMalloc / hipFree call and allocates nothing; the first call on
 * a device looks up that device's copy of the array. Per-stage timing is
 * not recorded. Every call on one device shares that device's array, which
 * keeps the last call's contents (nothing in it needs to start at zero):
 * calls that overlap in time on one device, from any plan or stream, race. */
oaa_status_t oaa_conv_forward_noalloc(oaa_plan_t plan, const float* x, const float* w, float* y,
                                      void* hip_stream);

/* Static text for a status code. */
const char* oaa_status_string(oaa_status_t status);

/* Thread-local detail for the last non-OK status returned on this thread
 * ("" if none). Valid until the next call on this thread. */
const char* oaa_last_error_detail(void);

#ifdef __cplusplus
}
#endif

#endif /* OAA_H_ */
