/*
 * sata.h - C ABI of the MI355X (gfx950) implementation of symmetry-aware Taylor
 * attention (Heinsen & Kozachkov, "Self-Attention at Constant Cost per Token via
 * Symmetry-Aware Taylor Approximation", arXiv 2602.00294).
 *
 * The method replaces exp(q.k / sqrt(d_k)) in causal attention by its P-term
 * Taylor series f_P (degrees 0..P-1, Sec. 2.1 and the truncation of Sec. 2.4),
 * and evaluates the series as an inner product of feature vectors over the
 * minimal symmetric monomial basis (Sec. 2.3-2.4): D = C(d_k+P-1, P-1) features.
 * Attention then runs as linear attention over the constant-size state
 *     S = sum_t phi(k_t) (x) [v_t, 1]        ([D][d_v+1] per head, App. A2)
 * with y_T = (phi(q_T)^T S_T)[0:d_v] / (phi(q_T)^T S_T)[d_v].
 *
 * Conventions fixed by this library (the paper leaves them open):
 *  - Feature order: degree-major; inside degree p the non-decreasing index tuples
 *    i1 <= ... <= ip (0-based) in lexicographic order.  Feature 0 is degree 0.
 *  - Feature weights: phi_m(x) = prod_j x[m_j] / (d^(p/4) * sqrt(prod_c c!)),
 *    i.e. sqrt(alpha_p * C_p[m]) with alpha_p = 1/(p! d^(p/2)) and C_p[m] the
 *    permutation count of m; so phi(q).phi(k) = f_P(q.k / sqrt(d)).
 *  - State layout: [B][H][D][d_v+1] float32, row-major; column d_v holds the
 *    normaliser Z = sum_t phi(k_t).
 *  - Causality is inclusive: output T sees tokens 0..T.
 *
 * Common rules for every call below:
 *  - Tensor arguments are device pointers to caller-owned, contiguous, row-major
 *    memory on the current HIP device.  Activations (q, k, v, y) use the layout
 *    [B][H][n][d] (prefill) or [B][H][d] (decode).  Outputs must not alias inputs.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *    asynchronous on that stream.  The host waits for the stream in two cases
 *    only: the first call on a device that needs a given (d_k, P) feature
 *    table (it uploads the table and waits for the copy, since every stream of
 *    the device shares it), and a call whose workspace on that stream must grow
 *    (it waits before freeing the smaller one).  A caller that captures calls
 *    into a graph makes one call of each shape first, outside the capture.
 *  - Arguments are validated on the host before anything is launched; on any
 *    error return nothing has been written and sata_last_error() explains it.
 *  - The library owns only per-device caches (feature tables, workspaces),
 *    created on first use and freed by sata_release().  Calls made concurrently
 *    on one device from different streams get separate workspaces.
 *  - Sizes: 1 <= d_k, d_v <= 255, 1 <= P <= 8, B*H <= 65535, and at most 2^26
 *    features per head (SATA_ERR_TOO_LARGE beyond).
 *  - Results are deterministic: identical inputs give bitwise-identical outputs
 *    (no floating-point atomics).
 */
#ifndef SATA_H
#define SATA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SATA_OK = 0,
  SATA_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, bad enum        */
  SATA_ERR_UNSUPPORTED = -2, /* valid request this implementation does not do    */
  SATA_ERR_TOO_LARGE = -3,   /* feature count / state too large for the kernels  */
  SATA_ERR_HIP = -4          /* a HIP runtime call or kernel launch failed       */
} sata_status;

typedef enum {
  SATA_F32 = 0,  /* IEEE binary32                          */
  SATA_BF16 = 1  /* bfloat16 (upper half of binary32 bits) */
} sata_dtype;

/* Number of features D = C(d+P-1, P-1) of degrees 0..P-1 over d coordinates
 * (Sec. 2.6, hidden state size).  Host only.  -1 if d < 1, P < 1, or overflow. */
int64_t sata_feature_count(int d, int P);

/* Elements of one head's state, (d_v+1) * C(d_k+P-1, P-1) (Sec. 2.6).
 * Host only.  -1 on invalid arguments or overflow. */
int64_t sata_state_elems(int d_k, int d_v, int P);

/* Which monomial feature f is (the rows of the constant index matrix M_p,
 * Sec. 2.4): writes its degree p to *degree and its indices i1 <= ... <= ip
 * (0-based) to idx[0..p-1]; idx must hold P-1 ints.  Host only, no GPU use.
 * SATA_ERR_INVALID_ARG if f is out of range or a pointer is NULL. */
sata_status sata_feature_index(int d, int P, int64_t f, int* degree, int* idx);

/* Feature map phi (Sec. 2.4, "Efficient Computation", with degree 0 from App. A1).
 *   x   : [rows][d] of dtype xt (device)
 *   phi : [rows][D] float32 (device, written)
 * rows = 0 is a no-op.  Supports 1 <= d <= 255, 1 <= P <= 8. */
sata_status sata_feature_map(const void* x, sata_dtype xt, int64_t rows, int d, int P,
                             float* phi, void* stream);

/* Causal prefill over n tokens from an empty state (App. A2: the accumulated
 * states and their readout; evaluated as a chunked scan).
 *   q, k : [B][H][n][d_k], v : [B][H][n][d_v], dtype dt (device)
 *   y    : [B][H][n][d_v], dtype dt (device, written): y_T = S_T / Z_T
 *   S_out: [B][H][D][d_v+1] float32 (device, written) or NULL: the state after
 *          token n-1, ready for sata_decode_step.
 * chunk: tokens per scan block, one of 16, 32, 64, 128.  The result does not
 * depend on it beyond float rounding.  n = 0 writes a zero S_out and no y.
 * Intermediate arithmetic is float32 or on the matrix cores with float32
 * accumulation (sata_prefill_operands tells which); the state is always float32.
 * Workspace: the tuned matrix-core kernels (bf16, P = 4, d_k = d_v in
 * {16, 32}) keep every token's float32 partial readouts (576 bytes per head
 * and token at d_k = 32, chunk 64) and serve a call only while those fit in
 * 4 GB; longer calls, and every other shape, work in segments whose partial
 * sums take at most 2 GB (512 MB on the float32 vector path), so the
 * workspace stays bounded for any n.
 * SATA_ERR_HIP if the workspace cannot be allocated; SATA_ERR_UNSUPPORTED if
 * a chunk's tiles do not fit on chip (for example d_k = 255 with chunk 64). */
sata_status sata_prefill(const void* q, const void* k, const void* v, sata_dtype dt,
                         int B, int H, int n, int d_k, int d_v, int P, int chunk,
                         void* y, float* S_out, void* stream);

/* Causal prefill with grouped query heads: each of the B*H_kv key/value heads
 * serves G consecutive query heads (query head g + G*h reads key/value head h),
 * the sharing of one key/value head by several query heads that a footnote of
 * Sec. 3.3 says carries over to this formulation.  Each query head's output is
 * sata_prefill's for its own queries and the shared keys and values:
 *   q    : [B][H_kv*G][n][d_k], k : [B][H_kv][n][d_k], v : [B][H_kv][n][d_v]
 *   y    : [B][H_kv*G][n][d_v], dtype dt (device, written)
 *   S_out: [B][H_kv][D][d_v+1] float32 or NULL: each key/value head's state,
 *          ready for sata_decode_step_grouped.
 * G = 1 is sata_prefill.  Each member of a group runs the prefill kernels of
 * sata_prefill with the shared keys and values, so the state contraction is
 * repeated G times (the readouts differ per member).  B*H_kv*G <= 65535;
 * other rules as sata_prefill. */
sata_status sata_prefill_grouped(const void* q, const void* k, const void* v, sata_dtype dt,
                                 int B, int H_kv, int G, int n, int d_k, int d_v, int P, int chunk,
                                 void* y, float* S_out, void* stream);

/* Gradients of the causal prefill: given dL/dy for every output, writes
 * dL/dq, dL/dk and dL/dv (training is the next step the paper names, Sec. 4;
 * the derivative is that of the causal output of App. A2).  The chunked scans
 * run over the same constant-size states as the forward: the forward scan
 * with S_T = sum_{t<=T} phi(k_t) (x) [v_t, 1] gives
 *     dL/dq_T = J_phi(q_T)^T S_T h_T,   h_T = [dy_T / Z_T, -(dy_T . y_T) / Z_T],
 * and the reverse scan with U_t = sum_{T>=t} phi(q_T) (x) h_T gives
 *     dL/dk_t = J_phi(k_t)^T U_t [v_t, 1],   dL/dv_t = (U_t^T phi(k_t))[0:d_v],
 * J_phi being the Jacobian of the feature map; inside a chunk the gradient of
 * f_P(q.k / sqrt(d_k)), f_{P-1}(s) k / sqrt(d_k), is used directly.
 *   q, k  : [B][H][n][d_k], v, dy : [B][H][n][d_v], dtype dt (device)
 *   dq, dk: [B][H][n][d_k], dv : [B][H][n][d_v], dtype dt (device, written)
 * All arithmetic is float32 (the forward is recomputed, not passed in).
 * chunk: 16, 32 or 64; d_k, d_v <= 64 (SATA_ERR_UNSUPPORTED otherwise).
 * Workspace: float32 dL/d[N|Z] for every token (4 (d_v+1) bytes per
 * head-token), one state, and per-segment partial sums of at most 2 GB.
 * n = 0 writes nothing. */
sata_status sata_backward(const void* q, const void* k, const void* v, const void* dy, sata_dtype dt,
                          int B, int H, int n, int d_k, int d_v, int P, int chunk,
                          void* dq, void* dk, void* dv, void* stream);

/* Operand precision of the state contractions (sata_prefill_operands). */
typedef enum {
  SATA_OPERANDS_F32 = 0,   /* every product formed in float32 (vector units)              */
  SATA_OPERANDS_BF16 = 1,  /* bfloat16 operands, float32 accumulation (matrix cores)       */
  SATA_OPERANDS_SPLIT = 2  /* float32 operands carried as bfloat16 pairs hi + lo, each
                              product as hi*hi + hi*lo + lo*hi (matrix cores)             */
} sata_operands;

/* Precision of the operands of the state contractions that sata_prefill uses
 * for these arguments (host only, no GPU use; same validation as sata_prefill).
 * The state is float32 in every case; callers use this to know the accuracy
 * to expect: about 2^-8 relative per term with bfloat16 operands, 2^-16 with
 * split operands, 2^-24 with float32 ones.  bfloat16 inputs take bfloat16
 * operands, float32 inputs split operands, where a matrix-core kernel covers
 * the shape (chunk 64 and d_k, d_v <= 64 with P >= 2; other chunks only for
 * the tuned bfloat16 P = 4, d in {16, 32} kernels); float32 arithmetic
 * otherwise. */
sata_status sata_prefill_operands(sata_dtype dt, int B, int H, int n, int d_k, int d_v, int P, int chunk,
                                  sata_operands* operands);

/* Number of parts of the sequence that sata_prefill runs side by side for
 * these arguments (host only, no GPU use; same validation as sata_prefill).
 * 1: the chunked scan of App. A2 runs token after token.  k > 1 (a call with
 * few heads and few features on the matrix-core path, whose sequence fits one
 * segment): a first pass forms each part's state increment, sum over its
 * tokens of phi(k) (x) [v, 1], and the scan of part g then starts from the sum
 * of the increments of parts 0..g-1, the same state up to the order of the
 * float32 additions; the workspace grows by (k - 1) states. */
sata_status sata_prefill_parts(sata_dtype dt, int B, int H, int n, int d_k, int d_v, int P, int chunk,
                               int* parts);

/* One decode step for every (b, h) (App. A2, the linear recurrences for Z_{p,T}
 * and S_{p,T}, then the readout at q_T): S += phi(k) (x) [v, 1], then
 * y = (phi(q)^T S)[0:d_v] / (phi(q)^T S)[d_v].  The update comes first, so the
 * new token attends to itself.
 *   S    : [B][H][D][d_v+1] float32 (device, read and written in place)
 *   q, k : [B][H][d_k], v : [B][H][d_v], dtype dt (device)
 *   y    : [B][H][d_v], dtype dt (device, written) */
sata_status sata_decode_step(float* S, const void* q, const void* k, const void* v,
                             sata_dtype dt, int B, int H, int d_k, int d_v, int P,
                             void* y, void* stream);

/* sata_decode_step for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, kernels and results (bitwise) as
 * sata_decode_step; it calls no hipMalloc, hipFree or allocating library
 * routine.  The partial sums and arrival counters of the split decode live in
 * a static 4 MB array per device, held until the process ends (the first call
 * on a device looks up its address and clears its counters with a kernel on
 * `stream`).  Every call on a device shares that array, so calls that overlap
 * on one device (other streams, other threads) race; serialise them.
 * SATA_ERR_TOO_LARGE if a call needs more than 4 MB - 256 KB of partial sums
 * (B*H * pieces * (d_v+1) floats; 67.6 KB at B*H = 256, d_k = d_v = 32, P = 4);
 * SATA_ERR_UNSUPPORTED if the (d_k, P) feature table does not exist on the
 * device yet: any earlier sata_decode_step, sata_prefill or sata_feature_map
 * call with that d_k and P creates it. */
sata_status sata_decode_step_noalloc(float* S, const void* q, const void* k, const void* v,
                                     sata_dtype dt, int B, int H, int d_k, int d_v, int P,
                                     void* y, void* stream);

/* Elements of one head's residual array for sata_decode_step_compensated:
 * D + (d_k+1)*d_v with D = C(d_k+P-1, P-1).  Host only.  -1 on invalid
 * arguments or overflow. */
int64_t sata_residual_elems(int d_k, int d_v, int P);

/* sata_decode_step with compensated summation of the state entries that stop
 * registering their per-token increments first as the context grows.  The
 * paper's decode costs the same for every token however long the context
 * (Sec. 1, Sec. 3.2); a float32 entry that grows with every token, such as
 * the degree-0 normaliser (the token count), absorbs increments below half
 * its ulp once about 2^24 tokens have been summed, so the outputs drift from
 * the method's.  This call keeps those entries as unevaluated float pairs:
 *   R : [B][H][D + (d_k+1)*d_v] float32 (device, read and written in place),
 *       per head R[f] for the normaliser column of row f (all D rows), then
 *       R[D + f*d_v + j] for value column j of rows f <= d_k (degrees 0 and 1).
 *       Zero it when the state is created (sata_prefill's state needs no
 *       residual: it adds whole chunks at a time).
 * After each call S holds the rounded pair sums, so S alone is the state to
 * float32 accuracy and may also be passed to sata_decode_step; the other
 * entries are updated as there.  The extra traffic is 8 bytes per residual
 * per step (3.5% of the state traffic at d_k = d_v = 32, P = 4).
 * SATA_ERR_UNSUPPORTED unless S is 16-byte aligned and d_v <= 127;
 * SATA_ERR_INVALID_ARG for a NULL R; otherwise as sata_decode_step. */
sata_status sata_decode_step_compensated(float* S, float* R, const void* q, const void* k, const void* v,
                                         sata_dtype dt, int B, int H, int d_k, int d_v, int P,
                                         void* y, void* stream);

/* One decode step with grouped query heads: each of the B*H_kv key/value
 * heads keeps one state and serves G consecutive query heads (query head
 * g + G*h reads key/value head h).  Sharing one key/value head among several
 * query heads is among the reuse schemes that a footnote of Sec. 3.3 says carry
 * over to this formulation; the update and readout are those of
 * sata_decode_step (App. A2), with the readout done for every query head:
 *   S += phi(k_h) (x) [v_h, 1];  y_{g+G h} = (phi(q_{g+G h})^T S)[0:d_v] / (...)[d_v]
 *   S    : [B][H_kv][D][d_v+1] float32 (device, read and written in place;
 *          16-byte aligned for G > 1)
 *   q    : [B][H_kv*G][d_k], k : [B][H_kv][d_k], v : [B][H_kv][d_v], dtype dt
 *   y    : [B][H_kv*G][d_v], dtype dt (device, written)
 * G = 1 is sata_decode_step.  G in {2, 4, 8} streams each state once for its
 * G query heads; other G, d_v large enough that no plan fits on chip (at
 * most 127 for large heads), or an unaligned state give SATA_ERR_UNSUPPORTED.
 * B*H_kv*G <= 65535. */
sata_status sata_decode_step_grouped(float* S, const void* q, const void* k, const void* v,
                                     sata_dtype dt, int B, int H_kv, int G, int d_k, int d_v, int P,
                                     void* y, void* stream);

/* Static text for a status code. */
const char* sata_status_string(sata_status s);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* sata_last_error(void);

/* Frees every cached table and workspace on every device.  Must not be called
 * while work issued by this library is still running. */
void sata_release(void);

#ifdef __cplusplus
}
#endif

#endif /* SATA_H */
