/*
 * cgconv.h - C ABI of the MI355X (gfx950) global Clebsch-Gordan convolution.
 *
 * The operation (arXiv 2509.24093, §4.1, Eq. (EquiConv) summed over every
 * path as in the path sum that follows it; FFT / tensor product / inverse FFT
 * as in Algorithm 1):
 *
 *   out[b,i,(J,M),c] = sum_{l1,l2} sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
 *                      * sum_j q[b,j,(l1,m1),c] * k[b,(i-j) mod N,(l2,m2),c]
 *
 * for every output degree J = 0..L_max and every triangle-allowed path
 * (|l1-l2| <= J <= l1+l2, l1,l2 <= L_max, odd l1+l2+J included), with unit
 * path weights, a cyclic token boundary and depthwise channels (channel c of q
 * meets only channel c of k; §4.1 "intra-channel").  R is the real-basis
 * Clebsch-Gordan tensor: real harmonics with Y_1 ~ (y, z, x), sign fixed so
 * that the (1,1 -> 1) path is +(1/sqrt 2) q x k (§4.4).  Sparsity follows
 * §4.3: only coefficients obeying the selection rule M = m1 + m2 (complex
 * basis) are evaluated.
 *
 * Layout of q, k, out: contiguous [batch][N][(L_max+1)^2][C], component index
 * l*l + l + m, channel fastest.  All pointers are DEVICE pointers, 16-byte
 * aligned.  Ownership: the caller owns q, k, out and the stream; a plan owns
 * its device workspace and tables.
 *
 * Errors: functions returning int give 0 on success or a negative
 * cgconv_status; cgconv_last_error() returns a thread-local message for the
 * last failure on the calling thread.  No C++ exception crosses this ABI.
 * Kernel faults are asynchronous and surface at the caller's next
 * synchronisation of the stream.
 *
 * Graph capture: every device allocation and upload happens at plan
 * creation; the compute entry points only enqueue kernels on the given
 * stream (no allocation, memset, copy or host synchronisation), so a call
 * may be captured into a HIP graph and replayed while its buffers live.
 * Per-stage timing (cgconv_plan_enable_timing) records events and is for
 * eager calls only.
 */
#ifndef CGCONV_H
#define CGCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t; /* same opaque type as HIP's */
typedef struct cgconv_plan* cgconv_plan_t;

enum cgconv_status {
  CGCONV_OK = 0,
  CGCONV_ERR_INVALID_ARG = -1,   /* null handle/pointer, bad size */
  CGCONV_ERR_UNSUPPORTED = -2,   /* N not a power of two, N too large, L_max too large */
  CGCONV_ERR_ALIGNMENT = -3,     /* a pointer is not 16-byte aligned */
  CGCONV_ERR_OUT_OF_MEMORY = -4, /* workspace allocation failed */
  CGCONV_ERR_HIP = -5            /* a HIP runtime call failed */
};

/* Largest supported degree and token count. */
#define CGCONV_LMAX 8
#define CGCONV_NMAX 65536
/* Largest node count of a graph plan (its bases are N x N per batch element). */
#define CGCONV_GRAPH_NMAX 16384

/*
 * Create a plan for q, k, out of shape [batch][N][(L_max+1)^2][C].
 * batch >= 1; N >= 2 and a power of two, N <= CGCONV_NMAX; 0 <= L_max <=
 * CGCONV_LMAX; C >= 1.  Builds the sparse CG table (§4.3) and the FFT
 * twiddles on the host, allocates the device workspace (hipMalloc on the
 * current device: 2 * batch*N*(L_max+1)^2*C*8 bytes for the spectra, the
 * gating partials, 8 * batch*ceil(N/64)*(L_max+1)*C bytes, 4 KiB per path
 * for the channel-mixing weights when L_max <= 6 and C <= 32, and small
 * tables; cgconv_plan_info reports the total) and uploads the tables.
 * Synchronous.  Returns NULL on failure (see cgconv_last_error()).
 *
 * Environment switches, read when a plan is created (all results stay within
 * the same accuracy; they exist for cross-checks and tests):
 *   CGCONV_UNFUSED=1        the modular five-kernel pipeline instead of the
 *                           fused middle kernel;
 *   CGCONV_NO_SMALL=1       for DFT lengths <= 256, the three single-pass
 *                           kernels instead of the one-block kernel;
 *   CGCONV_FORCE_GENERIC=1  the table-driven contraction kernel instead of the
 *                           generated per-L_max bodies (modular pipeline);
 *   CGCONV_TEST_FAIL_ALLOC=1  token plans return NULL with the message of a
 *                           failed workspace allocation (tests of that path).
 */
cgconv_plan_t cgconv_plan_create(int64_t batch, int64_t N, int32_t L_max, int64_t C);

/* Token boundary of a plan. */
enum cgconv_boundary {
  CGCONV_BOUNDARY_CYCLIC = 0, /* k index (i - j) mod N, as cgconv_plan_create */
  CGCONV_BOUNDARY_LINEAR = 1  /* zero padding: terms with i - j < 0 are absent (causal sum) */
};

/*
 * As cgconv_plan_create, with a choice of token boundary.  The paper's
 * Eq. (EquiConv) gives only the token sum; CGCONV_BOUNDARY_LINEAR reads it
 * with zero padding, the boundary of causal long convolutions:
 *
 *   out[b,i,(J,M),c] = sum_paths sum R^{(l1 l2 J)}[M,m1,m2]
 *                      * sum_{j=0}^{i} q[b,j,(l1,m1),c] * k[b,i-j,(l2,m2),c]
 *
 * computed exactly by DFTs of length Nf = the smallest power of two >= 2N-1
 * over the zero-padded tokens (no term wraps around).  With the linear
 * boundary N may be any value 1 <= N <= CGCONV_NMAX/2 (not only a power of
 * two); q, k, out keep N rows, and the workspace is sized for Nf rows.
 * Every entry point taking a plan follows its boundary: cgconv_forward,
 * cgconv_forward_bf16, cgconv_forward_mixed, cgconv_backward (the gradients
 * of the causal sum) and cgconv_gate_value (softmax over the N tokens).
 */
cgconv_plan_t cgconv_plan_create_boundary(int64_t batch, int64_t N, int32_t L_max, int64_t C,
                                          int32_t boundary);

/*
 * Enqueue one CG convolution on `stream` (NULL = the legacy default stream),
 * fp32 in, fp32 out, fp32 arithmetic.  Asynchronous: no host synchronisation.
 * out must not alias q or k; q == k is allowed.  The plan's workspace is
 * shared by its calls: do not have two forwards of one plan in flight on
 * different streams.  The device current at plan creation must be current.
 */
int cgconv_forward(cgconv_plan_t plan, const float* q, const float* k, float* out,
                   hipStream_t stream);

/*
 * As cgconv_forward, with q, k, out stored as bfloat16 bit patterns (uint16)
 * and all arithmetic in fp32; the output is rounded to bfloat16 to nearest,
 * ties to even.
 */
int cgconv_forward_bf16(cgconv_plan_t plan, const uint16_t* q, const uint16_t* k,
                        uint16_t* out, hipStream_t stream);

/*
 * CG convolution with per-path channel mixing (the inter-channel form of
 * §4.1: the depthwise product of every path is mixed over channels by one
 * dense weight matrix per path before the paths are summed):
 *
 *   out[b,i,(J,M),c] = sum_{p=(l1,l2,J)} sum_{c'} W_p[c,c']
 *                      * sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
 *                      * sum_j q[b,j,(l1,m1),c'] * k[b,(i-j) mod N,(l2,m2),c']
 *
 * weights: DEVICE pointer, fp32 [n_paths][C][C] (row = output channel c,
 * column = input channel c'), 16-byte aligned, paths in the order of
 * cgconv_paths.  W_p = identity for every p gives cgconv_forward.  q, k, out
 * as for cgconv_forward (fp32).  The dense mixing runs on the bfloat16
 * matrix cores with both operands split into bfloat16 high and low parts
 * (three products per tile, fp32 accumulation; relative error about 2^-17
 * per product); the unfused FFT passes are used.  Needs L_max <= 6 and C <= 32
 * (CGCONV_ERR_UNSUPPORTED otherwise).  Same stream and workspace rules as
 * cgconv_forward; the weights are read during the call only.
 */
int cgconv_forward_mixed(cgconv_plan_t plan, const float* q, const float* k, const float* weights,
                         float* out, hipStream_t stream);

/*
 * Inter-channel CG convolution with a per-degree channel reduction (§4.1:
 * query features with m channels and key features with m' channels give a
 * product with (2J+1) m m' components per degree, heads do not interact, and
 * the multiplicity is reduced again by a learned equivariant map, read here
 * as one real matrix per head and output degree):
 *
 *   out[b,i,(J,M),h*m_out+o] = sum_{c1,c2} weights[h][J][o][c1*m+c2]
 *        * sum_paths sum R^{(l1 l2 J)}[M,m1,m2]
 *          * sum_j q[b,j,(l1,m1),h*m+c1] * k[b,(i-j) mod N,(l2,m2),h*m+c2]
 *
 * with the plan's C = heads * m channels in heads of m (channel c = h*m + c'),
 * and its token boundary.  q, k: DEVICE fp32 [batch][N][(L_max+1)^2][C];
 * weights: DEVICE fp32 [heads][L_max+1][m_out][m*m], 16-byte aligned;
 * out: DEVICE fp32 [batch][N][(L_max+1)^2][heads*m_out], not aliasing q, k or
 * weights.  Needs L_max <= 6, m <= 8, m_out even and <= m
 * (CGCONV_ERR_UNSUPPORTED otherwise; heads must divide C).  Every channel
 * pair's product is evaluated by the generated contraction on the vector
 * units and reduced per degree on the matrix cores (fp32
 * v_mfma_f32_16x16x4f32), between the unfused FFT passes.  Same stream and
 * workspace rules as cgconv_forward; the weights are read during the call.
 */
int cgconv_forward_interchannel(cgconv_plan_t plan, int32_t heads, int32_t m_out, const float* q, const float* k,
                                const float* weights, float* out, hipStream_t stream);

/*
 * CG convolution in a graph Fourier basis (appendix "Fourier Space
 * Attention": the eigenvectors U of a graph's normalised Laplacian define the
 * transform x_hat = U^T x, inverse x = U x_hat, and a spectral convolution
 * multiplies the transforms frequency by frequency; the result permutes with
 * the nodes when U does).  With the CG product of §4.1 per graph frequency:
 *
 *   q_hat[b,f] = sum_i U[b,i,f] q[b,i],   k_hat[b,f] = sum_i U[b,i,f] k[b,i]
 *   out[b,i,(J,M),c] = sum_f U[b,i,f] sum_paths sum R^{(l1 l2 J)}[M,m1,m2]
 *                      * q_hat[b,f,(l1,m1),c] * k_hat[b,f,(l2,m2),c]
 *
 * cgconv_plan_create_graph(batch, N, L_max, C): N = nodes per batch element,
 * 1 <= N <= CGCONV_GRAPH_NMAX (any N); allocates the split operands of the
 * two transforms (about 8 batch*N^2 + 24 batch*N*K*C bytes).  Such a plan
 * serves cgconv_forward_graph, cgconv_backward_graph and cgconv_gate_value
 * only.
 * cgconv_forward_graph: U DEVICE fp32 [batch][N][N] (row i = node, column f
 * = graph frequency; orthonormal columns are the caller's responsibility,
 * the library applies U^T and U as given), q, k, out as for cgconv_forward;
 * out must not alias U, q or k.  The dense transforms run on the bfloat16
 * matrix cores with both operands split into high and low parts (relative
 * error about 2^-16 per product, fp32 accumulation); the per-frequency
 * product is the generated real-basis contraction.  Same stream and
 * workspace rules as cgconv_forward.
 */
cgconv_plan_t cgconv_plan_create_graph(int64_t batch, int64_t N, int32_t L_max, int64_t C);
int cgconv_forward_graph(cgconv_plan_t plan, const float* U, const float* q, const float* k, float* out,
                         hipStream_t stream);
/*
 * Backward of cgconv_forward_graph: given grad_out = dL/dout, the gradients
 * with respect to q and k (the chain rule through U^T, the per-frequency
 * product and U; valid for any U).  As for cgconv_backward, each gradient
 * is one forward pipeline of the same kernels with per-degree scales on the
 * per-frequency product (the transposition identity of the real-basis
 * tensor); the bases are split once for both.  Arguments and aliasing rules
 * as cgconv_backward, plus U as for cgconv_forward_graph.
 */
int cgconv_backward_graph(cgconv_plan_t plan, const float* U, const float* q, const float* k,
                          const float* grad_out, float* grad_q, float* grad_k, hipStream_t stream);

/*
 * Backward of cgconv_forward (the models of §5 are trained by gradient
 * descent through this operation): given grad_out = dL/dout for a scalar L,
 *
 *   grad_q[b,j,(l1,m1),c] = sum_i sum_{J,M,l2,m2} R^{(l1 l2 J)}[M,m1,m2]
 *                           * grad_out[b,i,(J,M),c] * k[b,(i-j) mod N,(l2,m2),c]
 *   grad_k[b,n,(l2,m2),c] = sum_i sum_{J,M,l1,m1} R^{(l1 l2 J)}[M,m1,m2]
 *                           * grad_out[b,i,(J,M),c] * q[b,(i-n) mod N,(l1,m1),c]
 *
 * (cyclic correlations with the transposed tensor).  Computed as two
 * forward convolutions on the same kernels: per path the real-basis tensor
 * satisfies R^{(J l2 l1)}[m1,M,m2] = (-1)^l2 sqrt((2 l1+1)/(2J+1))
 * R^{(l1 l2 J)}[M,m1,m2], so grad_q = s_o * conv(s_a * grad_out, s_b *
 * reverse(k)) with per-degree scales and reverse(x)[n] = x[-n mod N], and
 * likewise grad_k.  q, k, grad_out: DEVICE pointers, fp32, the layout of
 * cgconv_forward; grad_q, grad_k: outputs of the same layout, either may be
 * NULL (that gradient is skipped), not both; they must not alias q, k,
 * grad_out or each other.  q == k is allowed: the gradient with respect to
 * the shared tensor is then grad_q + grad_k (the caller adds them).  Same
 * stream and workspace rules as cgconv_forward; the two gradients are
 * computed one after the other in the plan's workspace.
 */
int cgconv_backward(cgconv_plan_t plan, const float* q, const float* k, const float* grad_out,
                    float* grad_q, float* grad_k, hipStream_t stream);

/*
 * Invariant softmax gating and the real-space value tensor product (§4.1.1
 * Invariant Gating; Algorithm 1, step 5), for the plan's batch, N, L_max, C:
 *
 *   I[b,i,l,c]     = || u[b,i,(l,.),c] ||_2          (norm over the 2l+1 components)
 *   g[b,i,l,c]     = exp(I[b,i,l,c]) / sum_j exp(I[b,j,l,c])   (softmax over tokens)
 *   f[b,i,(J,M),c] = sum_{paths} sum_{m1,m2} R^{(l1 l2 J)}[M,m1,m2]
 *                    * g[b,i,l1,c] u[b,i,(l1,m1),c] * v[b,i,(l2,m2),c]
 *
 * (the paper leaves the invariant map gamma and the softmax axis open; these
 * are the readings taken).  u (typically the convolution output), v (the
 * values) and f: DEVICE pointers, fp32 [batch][N][(L_max+1)^2][C], 16-byte
 * aligned; f must not alias u or v.  Uses a small plan-owned workspace; same
 * stream rules as cgconv_forward.
 */
int cgconv_gate_value(cgconv_plan_t plan, const float* u, const float* v, float* f, hipStream_t stream);

/*
 * cgconv_gate_value for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same operation and kernels with no plan.  The softmax
 * partials and statistics live in a library-owned static device array of
 * 16 MiB, which each device the library runs on holds until the process
 * ends; this call allocates nothing (no hipMalloc, hipFree or allocating
 * library routine).  batch, N (tokens), L_max, C: sizes of u, v, f, DEVICE
 * fp32 [batch][N][(L_max+1)^2][C], 16-byte aligned, f not aliasing u or v;
 * 1 <= batch <= 65535, N >= 1, 0 <= L_max <= CGCONV_LMAX, C >= 1, and
 * batch * (ceil(N/64) + 1) * (L_max+1) * C * 8 bytes must fit in the array
 * (CGCONV_ERR_UNSUPPORTED otherwise; e.g. batch=8, N=16384, L_max=6, C=32
 * needs 3.7 MB).  Every call on a device shares that device's array: calls
 * that overlap on one device (two streams, two threads) race and must be
 * ordered by the caller.  Enqueues on `stream`; the first call on a device
 * also looks up the array's address there (host-only).
 */
int cgconv_gate_value_noalloc(int64_t batch, int64_t N, int32_t L_max, int64_t C, const float* u, const float* v,
                              float* f, hipStream_t stream);

/*
 * Backward of cgconv_gate_value (the models of §5 are trained through this
 * step too): given grad_f = dL/df, the gradients with respect to u and v by
 * the chain rule through the definition above, with a = g u:
 *
 *   grad_v = R-transposed contraction of (grad_f, a), grad_a = that of (grad_f, v)
 *   h[b,i,l,c] = g sum_m u grad_a                   (the gate's gradient times g)
 *   grad_u = g grad_a + (h - g sum_j h[b,j,l,c]) u / I   (softmax and norm; no term where I = 0)
 *
 * Both contractions are forward token-wise products under the per-degree
 * scales of cgconv_backward.  u, v, grad_f: DEVICE pointers, fp32, the layout
 * of cgconv_gate_value; grad_u, grad_v: outputs of the same layout, either
 * may be NULL (skipped), not both; they must not alias the inputs or each
 * other.  Uses the plan's gating workspace (about 4 batch*N*(L_max+1)*C
 * bytes more than the forward); same stream rules as cgconv_forward.
 */
int cgconv_gate_value_backward(cgconv_plan_t plan, const float* u, const float* v, const float* grad_f,
                               float* grad_u, float* grad_v, hipStream_t stream);

/*
 * Host-only (no GPU needed): the CG paths at L_max in the order the mixing
 * weights use, every triangle-allowed (l1, l2, J) with l1, l2, J <= L_max
 * (odd l1+l2+J included), lexicographic in (l1, l2, J).  Writes up to cap
 * triples to l1l2J[3*p .. 3*p+2] (may be NULL when cap == 0) and returns the
 * number of paths, or a negative status.
 */
int64_t cgconv_paths(int32_t L_max, int32_t* l1l2J, int64_t cap);

/* Free the plan's device workspace and tables.  NULL is a no-op. */
void cgconv_plan_destroy(cgconv_plan_t plan);

/*
 * Plan introspection: number of CG paths (l1,l2,J) (§4.1, the path sum);
 * number of non-zero real-basis coefficients of the tensor the plan's
 * kernels evaluate (the entries cgconv_plan_export_table writes; §4.3 and
 * the appendix on sparsity, real basis); workspace bytes.  Any output
 * pointer may be NULL.  Returns 0, or CGCONV_ERR_INVALID_ARG for a NULL plan.
 */
int cgconv_plan_info(cgconv_plan_t plan, int64_t* n_paths, int64_t* nnz, size_t* workspace_bytes);

/*
 * The form in which the kernels of a token plan evaluate that tensor: the
 * number of complex-basis terms (selection rule M = m1 + m2, §4.3) and of
 * distinct complex products q[l1,m1] * k[l2,m2] among them, per frequency
 * and channel.  (A graph plan reports the same counts; its per-frequency
 * product runs on the real-basis entries.)  Either pointer may be NULL.
 */
int cgconv_plan_contraction_info(cgconv_plan_t plan, int64_t* nnz_complex, int64_t* n_products);

/*
 * Export the real-basis CG tensor R^{(l1 l2 J)}[M,m1,m2] that the plan's
 * kernels evaluate (§4.1 Eq. (EquiConv) summed over the paths; the sparse
 * entries of §4.3).  For a token plan it is recovered from the plan's
 * complex-basis contraction terms (the table the generated and the
 * table-driven kernels are built from) by expanding them back to the real
 * basis; for a graph plan it is the real table of its per-frequency
 * product.  Writes up to `cap` entries: l1m1l2m2JM[6*e .. 6*e+5] =
 * (l1, m1, l2, m2, J, M) and coef[e] (double), every |coef| > 1e-12, sorted
 * by (J, M, l1, m1, l2, m2); both buffers are HOST memory owned by the
 * caller and may be NULL when cap == 0.  Returns the total number of entries
 * (= cgconv_plan_info's nnz; it may exceed cap, nothing beyond cap is
 * written), or CGCONV_ERR_INVALID_ARG (NULL plan, cap < 0, NULL buffer with
 * cap > 0).  Host-only: no device work.
 */
int64_t cgconv_plan_export_table(cgconv_plan_t plan, int32_t* l1m1l2m2JM, double* coef, int64_t cap);

/*
 * Host-only (no GPU needed): the real-basis CG tensor R for degrees 0..L_max
 * as the library builds it (§4.3 and the appendix on sparsity, real basis).
 * Writes up to `cap` entries: idx[6*e .. 6*e+5] = (l1, m1, l2, m2, J, M) and
 * coef[e], for every path and every |coefficient| > 1e-12, sorted by
 * (J, M, l1, m1, l2, m2).  Returns the total number of entries (which may
 * exceed cap; nothing beyond cap is written), or a negative status.
 * idx/coef may be NULL when cap == 0.
 */
int64_t cgconv_cg_table(int32_t L_max, int32_t* idx, double* coef, int64_t cap);

/*
 * Host-only (no GPU needed) self-check of the frequency-domain contraction
 * the kernels evaluate: given the spectra of q and k at one frequency for one
 * channel (K complex values each, interleaved re,im, real-basis component
 * order), writes the K complex output values.  It applies the same
 * coefficient table, in double precision, that the generated GPU code
 * carries.  cgconv_forward never calls it.
 */
int cgconv_contract_host(int32_t L_max, const double* qhat, const double* khat, double* uhat);

/*
 * Per-stage timing for profiling.  After cgconv_plan_enable_timing(plan, n),
 * the next n forwards of the plan record HIP events before and after each
 * kernel stage on the forward's own stream (a few microseconds per call);
 * calls beyond n are not timed.  Enabling again resets the record.
 * cgconv_plan_stage_times waits for the timed calls to finish and writes the
 * summed time of each stage in milliseconds to ms[0 .. min(cap, n_stages)-1];
 * n_stages and n_calls (may be NULL) receive the stage count (3 for N <= 256:
 * fft_fwd, cg, fft_inv; 5 above: fft_fwd_1, fft_fwd_2, cg, fft_inv_1,
 * fft_inv_2; for plans with 512 <= N <= 32768 and L_max <= 6: fft_fwd_1,
 * cg_fused, fft_inv_2) and the number of timed calls.  The first timed call
 * fixes which kind is timed: plain forwards, mixed forwards (cg_mix replaces
 * cg and the unfused passes are listed), inter-channel forwards (cg_inter
 * likewise), backwards (each of the two
 * gradients is one timed call with the plain stages), gating calls
 * (gate_partials, gate_finalize, gate_value), gating backwards (gate_stats,
 * gate_bwd, gate_sums, gate_bwd_du) or graph forwards
 * (gft_split_u, gft_split_x, gft_gemm_fwd, gft_product, gft_split_uhat,
 * gft_gemm_inv); calls of the other kinds are not timed.
 * cgconv_plan_stage_name returns a stage's name ("" if out of range).
 */
int cgconv_plan_enable_timing(cgconv_plan_t plan, int32_t max_calls);
int cgconv_plan_stage_times(cgconv_plan_t plan, double* ms, int32_t cap, int32_t* n_stages, int32_t* n_calls);
const char* cgconv_plan_stage_name(cgconv_plan_t plan, int32_t stage);

/* Thread-local message describing the last error on this thread ("" if none). */
const char* cgconv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CGCONV_H */
