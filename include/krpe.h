/*
 * krpe.h -- C ABI of the kernelized-attention-with-RPE library (libkrpe.so).
 *
 * The library computes, on one AMD Instinct MI355X (gfx950), the forward pass
 * of positive-random-feature kernelized attention with a relative positional
 * bias (Luo et al., "Stable, Fast and Accurate: Kernelized Attention with
 * Relative Positional Encoding", NeurIPS 2021), in O(n log n) per channel:
 *
 *   z_i = phi(q_i) sum_j c_{j-i} phi(k_j)^T v_j  /  phi(q_i) sum_j c_{j-i} phi(k_j)^T
 *                                                        (Section 3.2, Eq. (10))
 *   phi(x) = exp(W x^T - ||x||^2 / 2) / sqrt(m)          (Section 2.1, Eq. (5))
 *   c_t    = exp(b_t),  t = j - i in [-(n-1), n-1]       (Section 2.2, Eq. (6))
 *
 * The products with the Toeplitz matrix C = {c_{j-i}} of Eqs. (12)-(13) run as
 * zero-padded FFT convolutions (Section 3.2, the paragraph after Eq. (13)).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every array pointer is a DEVICE pointer (memory from hipMalloc or any
 *   allocator handing out device memory, e.g. a torch CUDA tensor), holding a
 *   dense row-major array, 16-byte aligned.  The caller owns all memory: the
 *   library never allocates, frees or keeps a pointer after returning.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *   work is enqueued asynchronously on it; buffers must stay alive until that
 *   work has completed.  Faults during execution surface at the caller's next
 *   synchronisation with the stream.
 * - b[h, s] stores b_t for t = s - (n - 1), i.e. the vector
 *   (b_{-(n-1)}, ..., b_{n-1}) of Algorithm 1, one vector of length 2n-1 per
 *   head.  b_t = -inf is allowed and gives c_t = 0 exactly; causal masking
 *   (Section 3.2, footnote on teacher forcing) is expressed this way, with
 *   b_t = -inf for t > 0.
 * - All argument checks run on the host before any HIP call.  A non-OK return
 *   means nothing was enqueued; krpe_last_error() then describes the problem.
 *   Launch failures return KRPE_ERR_HIP.  No exception or abort crosses the ABI.
 * - Inputs are read-only.  Outputs are fully overwritten and must not overlap
 *   any input or the workspace (KRPE_ERR_ALIAS).  Workspace contents are
 *   undefined on return.
 * - Supported sizes: 1 <= n <= 16384 (any n; the FFT length is 2N with N the
 *   next power of two >= n), except the attention forward pass
 *   (krpe_attention_fwd*, krpe_feature_map*) and the Toeplitz product
 *   (krpe_toeplitz_conv*): 1 <= n <= 65536, longer sequences taking the
 *   Toeplitz matrix in blocks of 16384 positions;
 *   1 <= d <= 128, 1 <= m <= 1024, B, H >= 0, C >= 0.
 *   B*H == 0 (or C == 0) is a valid empty call that enqueues nothing.
 * - Precondition (not checked: it would need to read device memory): every
 *   query row's window of b holds a finite entry (b_0 finite suffices), so
 *   every denominator of Eq. (10) is > 0.  Otherwise that row of z is NaN.
 * - Functions are stateless and thread-safe, except krpe_toeplitz_conv_noalloc,
 *   whose calls on one GPU share a static workspace (see its note).
 */
#ifndef KRPE_H_
#define KRPE_H_

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of q, k, v and x.  W, b, phi, a, y and z are always fp32. */
typedef enum {
  KRPE_F32 = 0,  /* IEEE binary32 */
  KRPE_BF16 = 1  /* bfloat16 bit patterns (uint16); converted exactly to fp32 */
} krpe_dtype_t;

typedef enum {
  KRPE_OK = 0,
  KRPE_ERR_NULL = 1,        /* a required pointer is NULL */
  KRPE_ERR_SHAPE = 2,       /* a size is negative or inconsistent */
  KRPE_ERR_UNSUPPORTED = 3, /* valid per the method, outside the supported sizes */
  KRPE_ERR_DTYPE = 4,       /* unknown krpe_dtype_t */
  KRPE_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than the query says */
  KRPE_ERR_ALIAS = 6,       /* an output overlaps an input or the workspace */
  KRPE_ERR_HIP = 7,         /* a HIP runtime call or kernel launch failed */
  KRPE_ERR_ALIGN = 8        /* a pointer is not 16-byte aligned */
} krpe_status_t;

/*
 * Option bits of the _ex entry points (other bits: KRPE_ERR_UNSUPPORTED).
 * KRPE_NPRF: divide every row of q and k (of x for the feature map) by its l2
 * norm before the feature map -- the first step of Algorithm 1, "Normalized
 * Kernelized Attention with RPE" (Section 3.3).  A zero row stays zero.
 */
#define KRPE_NPRF 1u
/*
 * Feature map options (Section 2; at most one of them; PRF of Eq. (5) when
 * neither is set).  The method is the same for every feature map: only phi
 * changes, and with it the number M of features per position.
 * KRPE_FEAT_TRF: the trigonometric random features of Section 2,
 *   phi(x) = exp(||x||^2/2) / sqrt(m) [sin(w_1 x), .., sin(w_m x),
 *                                      cos(w_1 x), .., cos(w_m x)],
 *   M = 2m signed features from the m rows of W (so m <= 512).  The
 *   denominator of Eq. (10) can then be small or negative: rows whose FFT
 *   result cannot be certified to 1e-4 (a vanishing denominator among them)
 *   are evaluated directly, and a zero denominator gives inf / nan as the
 *   formula does.
 * KRPE_FEAT_ELU: elu(x) + 1 elementwise, the linear transformer's map the
 *   paper compares with; M = d, m must equal d, W is not read (may be NULL).
 * Sphere-PRF and ORF (the paper's appendix comparison) are PRF with W drawn
 * from the sphere of radius sqrt(d) or with orthogonal rows: no option, the
 * caller passes that W.
 */
#define KRPE_FEAT_TRF 2u
#define KRPE_FEAT_ELU 4u
/*
 * Route of the forward pass (at most one; neither: chosen by the measured
 * cost model of krpe_attention_fwd_route, from the sizes and the head
 * count).  KRPE_ROUTE_FFT: the O(n log n) FFT
 * convolution of Section 3.2 (rows it cannot certify evaluated directly).
 * KRPE_ROUTE_DIRECT: every row evaluated directly from Eq. (10) as
 * (phi(Q) phi(K)^T o C) [v, 1] on fp32 MFMA tiles with fp64 totals, O(n^2);
 * faster than the FFT route for short sequences and many heads.  Same results to the
 * tolerance of the FFT route (the direct route is the more accurate).
 */
#define KRPE_ROUTE_DIRECT 8u
#define KRPE_ROUTE_FFT 16u
/*
 * KRPE_HINT_CAUSAL: the caller states that b[h][t + n - 1] = -inf for every
 * t > 0 (query i attends to keys j <= i only, the causal mask of Sec. 3.2's
 * relative-position view).  Read by the route choice alone: the direct route
 * visits only the keys inside each row's finite-b range, so with the hint
 * its cost model counts n (n + 1) / 2 query/key pairs instead of n^2.
 * Results do not depend on it (both routes evaluate Eq. (10) for the b
 * given), and a wrong hint only costs time.
 */
#define KRPE_HINT_CAUSAL 32u

/* Version of this ABI (incremented on any incompatible change). */
int krpe_abi_version(void);

/* Static text for a status code; never NULL. */
const char* krpe_status_str(int status);

/* Detail of the last non-OK return on the calling thread ("" if none). */
const char* krpe_last_error(void);

/*
 * Positive random feature map, Section 2.1, Eq. (5):
 *   phi[beta, h, i, l] = exp( sum_a W[h, l, a] x[beta, h, i, a]
 *                             - 0.5 sum_a x[beta, h, i, a]^2 ) / sqrt(m)
 * x   : [B, H, n, d] in x_dtype        W : [H, m, d] fp32 (rows w_l)
 * phi : [B, H, n, m] fp32 (output)
 * Runs as an fp32 MFMA contraction with the exponential fused into its epilogue.
 */
krpe_status_t krpe_feature_map(const void* x, int x_dtype, const float* W, float* phi,
                               int B, int H, int n, int d, int m, void* stream);
/*
 * krpe_feature_map with option bits: KRPE_NPRF (phi of x / ||x||), one of
 * KRPE_FEAT_TRF / KRPE_FEAT_ELU.  phi is then [B, H, n, M] with M = 2m (TRF,
 * sin features first) or d (elu + 1; W not read).
 */
krpe_status_t krpe_feature_map_ex(const void* x, int x_dtype, const float* W, float* phi,
                                  int B, int H, int n, int d, int m, unsigned flags, void* stream);

/*
 * Bytes of workspace krpe_toeplitz_conv needs for B x H heads of C channels of
 * length n (0 if the sizes are invalid or unsupported).
 */
size_t krpe_toeplitz_conv_workspace(int B, int H, int C, int n);

/*
 * Product with the Toeplitz matrix C = {c_{j-i}} of Eqs. (12)-(13), per channel:
 *   y[beta, h, ch, i] = sum_{j<n} exp(b[h, j - i + n - 1]) * a[beta, h, ch, j]
 * b : [H, 2n-1] fp32     a, y : [B, H, C, n] fp32 (sequence-contiguous channels)
 * Computed as a zero-padded length-2N FFT convolution (split into residue
 * classes of its frequency bins, each a transform of at most 8192 points).
 * For n > 16384 the matrix is taken in blocks of 16384 positions, y_I =
 * sum_J C_IJ a_J, each block of C itself Toeplitz (its window of b); blocks
 * of C that are all zero (b = -inf throughout, e.g. above the diagonal under
 * a causal mask) cost no transforms.
 */
krpe_status_t krpe_toeplitz_conv(const float* b, const float* a, float* y,
                                 int B, int H, int C, int n,
                                 void* ws, size_t ws_bytes, void* stream);

/*
 * krpe_toeplitz_conv for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
 * the same product with no workspace argument.  Its workspace is a static
 * device array of KRPE_NOALLOC_SCRATCH_BYTES bytes inside the library, one
 * copy per GPU, held from the library's load until the process ends; the call
 * allocates and frees nothing.  Sizes whose workspace (the value of
 * krpe_toeplitz_conv_workspace) exceeds it return KRPE_ERR_UNSUPPORTED before
 * any HIP call.  Every call on a GPU shares that GPU's array: calls that
 * overlap on one GPU (two streams, or two threads) race and must be
 * serialised by the caller.  The array keeps the last call's contents; every
 * call writes all of the workspace it reads.  The first call on a device
 * looks the array's address up (hipGetSymbolAddress), briefly making the
 * stream's device current if it is not.
 */
#define KRPE_NOALLOC_SCRATCH_BYTES (64u << 20)
krpe_status_t krpe_toeplitz_conv_noalloc(const float* b, const float* a, float* y,
                                         int B, int H, int C, int n, void* stream);

/*
 * Bytes of workspace krpe_attention_fwd needs (0 if the sizes are invalid or
 * unsupported).
 */
size_t krpe_attention_fwd_workspace(int B, int H, int n, int d, int m);
/* The same for krpe_attention_fwd_ex with option bits (TRF needs more). */
size_t krpe_attention_fwd_workspace_ex(int B, int H, int n, int d, int m, unsigned flags);

/*
 * The route krpe_attention_fwd_ex takes for these sizes and option bits:
 * KRPE_ROUTE_DIRECT or KRPE_ROUTE_FFT (0 if the sizes or bits are invalid).
 * Without a route bit it follows a cost model of both routes measured on
 * MI355X (work over the B*H heads plus each route's fixed cost); it counts
 * all n^2 query/key pairs (b is not read on the host), n (n + 1) / 2 with
 * KRPE_HINT_CAUSAL.
 */
int krpe_attention_fwd_route(int B, int H, int n, int d, int m, unsigned flags);

/*
 * Kernelized attention with RPE, Section 3.2, Eq. (10), with phi from Eq. (5)
 * using W[h] for head h and c = exp(b[h]):
 * q, k, v : [B, H, n, d] in qkv_dtype (the already-projected x W^Q, x W^K, x W^V)
 * b       : [H, 2n-1] fp32            W : [H, m, d] fp32
 * z       : [B, H, n, d] fp32 (output)
 * ws      : device workspace of at least krpe_attention_fwd_workspace() bytes.
 * Queries and keys are used as given (no normalisation, no 1/sqrt(d) scale).
 */
krpe_status_t krpe_attention_fwd(const void* q, const void* k, const void* v, int qkv_dtype,
                                 const float* b, const float* W, float* z,
                                 int B, int H, int n, int d, int m,
                                 void* ws, size_t ws_bytes, void* stream);

/*
 * krpe_attention_fwd with option bits: KRPE_NPRF normalises the rows of q
 * and k first (Algorithm 1's NPRF attention); KRPE_FEAT_TRF / KRPE_FEAT_ELU
 * select the feature map (W [H, m, d] as above; not read for elu + 1, where
 * m == d); KRPE_ROUTE_DIRECT / KRPE_ROUTE_FFT force a route and
 * KRPE_HINT_CAUSAL informs the route choice.  Workspace:
 * krpe_attention_fwd_workspace_ex with the same flags.
 */
krpe_status_t krpe_attention_fwd_ex(const void* q, const void* k, const void* v, int qkv_dtype,
                                    const float* b, const float* W, float* z,
                                    int B, int H, int n, int d, int m, unsigned flags,
                                    void* ws, size_t ws_bytes, void* stream);

/*
 * krpe_attention_fwd_ex with per-stage timing: when `events` is not NULL it points
 * to KRPE_STAGE_EVENTS hipEvent_t handles (as void*), recorded on `stream`
 * before the spectrum of c, before the feature maps, before the FFT
 * convolution + contraction kernel, before the final division and after it.
 * The events are created and owned by the caller.
 */
#define KRPE_STAGE_EVENTS 5
krpe_status_t krpe_attention_fwd_profiled(const void* q, const void* k, const void* v,
                                          int qkv_dtype, const float* b, const float* W,
                                          float* z, int B, int H, int n, int d, int m,
                                          unsigned flags, void* ws, size_t ws_bytes, void* stream,
                                          void* const* events);

/*
 * Bytes of workspace krpe_attention_bwd needs (0 if the sizes or flags are
 * invalid or unsupported).
 */
size_t krpe_attention_bwd_workspace(int B, int H, int n, int d, int m, unsigned flags);

/*
 * Backward pass of krpe_attention_fwd_ex (PRF features of Eq. (5), optional
 * KRPE_NPRF, the route bits and KRPE_HINT_CAUSAL for the recomputed forward;
 * W fixed): the gradients of L = sum(dz * z) with respect to q, k,
 * v and b, z from Eq. (10).  The paper states no backward pass; these are the
 * derivatives of its forward definition.  With A = C o (phi(Q) phi(K)^T),
 * den = A 1 and Gh = [dz / den, -(dz . z) / den] per row:
 *   dv = A^T Gh[:, :d],  dphi(Q) = ((Gh [v, 1]^T) o C) phi(K),
 *   dphi(K) = ((Gh [v, 1]^T) o C)^T phi(Q),  dx = (dphi o phi) W - x rowsum(dphi o phi)
 * (through the row normalisation when KRPE_NPRF).  Each of the three
 * products is one run of the forward's FFT convolution kernel, with the
 * transposed Toeplitz matrix (the reversed b) where C^T appears; the forward
 * pass is recomputed inside (its exact-row evaluation included).
 * q, k, v : [B, H, n, d] in qkv_dtype    b : [H, 2n-1]    W : [H, m, d]
 * dz      : [B, H, n, d] fp32             dq, dk, dv : [B, H, n, d] fp32 (outputs)
 * db      : [H, 2n-1] fp32 (output, summed over the batch), or NULL to skip it:
 *           db_t = c_t sum_{l,c} corr(phi_l(q) o Gh_c, phi_l(k) o [v, 1]_c)(t), one
 *           spectrum per head accumulated over all channels (FFT cross-correlation);
 *           0 where b_t = -inf.
 * ws      : device workspace of at least krpe_attention_bwd_workspace() bytes.
 * Outputs must not overlap each other, an input or the workspace.
 */
krpe_status_t krpe_attention_bwd(const void* q, const void* k, const void* v, int qkv_dtype,
                                 const float* b, const float* W, const float* dz,
                                 float* dq, float* dk, float* dv, float* db,
                                 int B, int H, int n, int d, int m, unsigned flags,
                                 void* ws, size_t ws_bytes, void* stream);

/*
 * Rows of the last krpe_attention_fwd / _ex call (with this workspace and
 * these sizes, whatever its option bits) that were evaluated exactly instead
 * of through the FFT.
 *
 * The FFT path's fp32 rounding error is spread over a whole sequence, so a
 * row whose denominator of Eq. (10) is small next to the sequence's total
 * (the first rows under a causal mask, for example) cannot be resolved by it.
 * krpe_attention_fwd bounds that error for every row and recomputes the rows
 * it cannot certify directly from Eq. (10) with fp64 accumulation.  This call
 * waits for `stream`, then copies the number of such rows into *fixed_rows.
 */
krpe_status_t krpe_attention_fwd_stats(const void* ws, size_t ws_bytes, int B, int H, int n, int d, int m,
                                       unsigned* fixed_rows, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KRPE_H_ */
