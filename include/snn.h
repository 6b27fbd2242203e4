/*
 * snn.h -- C ABI of the MI355X (gfx950) sparse spiking BPTT library (libsnn.so).
 *
 * Method: Perez-Nieves & Goodman, "Sparse Spiking Gradient Descent", NeurIPS 2021.
 * One fully connected layer of leaky integrate-and-fire (LIF) neurons at a time:
 *   forward       V[t+1] = alpha V[t] + sum_i S_in[t,i] W[i,j] - S_out[t,j]   (Sec. 2.1, Eq. (lif),
 *                 V_rest = V_r = 0, V[0] = 0), S_out[t,j] = V[t,j] > theta    (Eq. (spike_fn))
 *   active set    |V[t,j] - theta| < b_th                                      (Definition 1)
 *   spike deriv.  g(V) = 1/(beta |V - theta| + 1)^2 on the active set, else 0  (Definition 2; Sec. 3)
 *   backward      dW_ij = sum_t G_j[t] trace_i[t],  G = eps * dS/dV           (Eq. (w_grad))
 *                 eps_in_i[t] = sum_j W_ij delta_j[t], only where the input
 *                 neuron i is active at t                                      (Eq. (s_grad), Sec. 2.2)
 *                 delta_j[t] = alpha delta_j[t+1] + G_j[t+1], delta[T-1] = 0   (Proposition 1, App. B)
 *
 * Conventions shared by every entry point
 *   Layout       Time-major, row-major, contiguous: a [T,B,N] tensor holds element (t,b,n) at
 *                (t*B + b)*N + n. A "row" is one (t,b) pair, r = t*B + b. W is [N_in, N_out].
 *                Spikes are uint8, any nonzero byte is a spike. Real tensors are float32.
 *   Memory       Every tensor pointer is DEVICE memory owned by the caller; labels too.
 *                The library allocates and frees nothing. Scratch memory comes from the
 *                caller's workspace (device memory, at least the size the matching
 *                *_workspace() query returns, 256-byte aligned).
 *   Streams      `stream` is a hipStream_t (NULL = the default stream). Every call only
 *                enqueues work on it and returns; nothing synchronises the host.
 *   Errors       Arguments are checked on the host before any HIP call; a bad argument
 *                returns SNN_ERR_INVALID_ARG and enqueues nothing. Sizes outside what the
 *                kernels support return SNN_ERR_UNSUPPORTED. A failed launch returns
 *                SNN_ERR_HIP. Checked: null required pointers, dimensions <= 0, element
 *                counts T*B*N >= 2^31, alpha outside (0,1] or NaN, NaN theta, NaN or
 *                negative beta and b_th, a workspace smaller than the query's size.
 *   State        The library keeps no state between calls; calls on different streams
 *                may run concurrently if their outputs do not overlap.
 */
#ifndef SNN_H
#define SNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SNN_OK = 0,
  SNN_ERR_INVALID_ARG = -1,
  SNN_ERR_UNSUPPORTED = -2,
  SNN_ERR_HIP = -3
} snn_status;

/* Human-readable name of a status code (static string, never NULL). */
const char* snn_status_string(int status);

/*
 * LIF forward of one layer (Sec. 2.1, Eqs. (lif), (spike_fn), (lif_unrolled)).
 *   s_in     [T,B,N_in]  uint8 input spikes (read)
 *   W        [N_in,N_out] float32 weights (read)
 *   alpha    leak factor exp(-dt/tau), in (0,1]
 *   theta    threshold V_th; +INFINITY gives the non-spiking readout of Sec. 3
 *   V        [T,B,N_out] float32 membrane potential (written), V[0] = 0
 *   s_out    [T,B,N_out] uint8 output spikes (written), s_out[t] = V[t] > theta
 *   trace_in [T,B,N_in]  float32 input trace (written unless NULL):
 *            trace[0] = 0, trace[t+1] = alpha*trace[t] + s_in[t]  (the filtered input that
 *            Eq. (w_grad) reuses from the forward)
 * Arithmetic is float32 with every operation rounded separately (no fused multiply-add) and
 * the weighted input of a row summed over its spiking inputs in ascending input index starting
 * from +0.0, so V and s_out are a deterministic function of the inputs.
 * s_in[T-1] does not enter V. V doubles as scratch during the call (the weighted inputs are
 * parked in it before the recurrence overwrites them). Supported: N_out <= 4096; larger N_out
 * returns SNN_ERR_UNSUPPORTED.
 */
snn_status snn_lif_forward(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                           float alpha, float theta, float* V, uint8_t* s_out, float* trace_in,
                           void* stream);

/*
 * The forward with the active set of Definition 1 marked on the way (the band test runs on each
 * V value while it is in a register, so compaction need not read V again).
 *   b_th         backprop band; bit (t,b,j) is set iff |V[t,b,j] - theta| < b_th, in float32
 *                exactly as snn_active_compact evaluates it
 *   active_bits  uint64 bitset of snn_active_bits_words(T,B,N_out) words (written): bit (t, k),
 *                k = b*N_out + j, is bit k % 64 of word t*W64 + k/64, W64 = ceil(B*N_out/64)
 * Everything else as snn_lif_forward. NaN or negative b_th -> SNN_ERR_INVALID_ARG.
 */
size_t snn_active_bits_words(int T, int B, int N);
snn_status snn_lif_forward_active(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                  float alpha, float theta, float b_th, float* V, uint8_t* s_out,
                                  float* trace_in, uint64_t* active_bits, void* stream);

/*
 * The forward that also writes the trace of its own output spikes, which the next layer (a
 * readout, say) reads as its input trace (Eq. (w_grad)), so that layer's forward can be called
 * with trace_in = NULL instead of walking the spikes again.
 *   trace_out    [T,B,N_out] float32 (written unless NULL): trace_out[0] = 0,
 *                trace_out[t+1] = alpha_next*trace_out[t] + s_out[t], bit-identical to the
 *                trace_in that a forward of the next layer writes from s_out
 *   alpha_next   the leak of that trace (the next layer's alpha), in (0,1]; checked only when
 *                trace_out is not NULL
 *   active_bits  as snn_lif_forward_active, or NULL for no active set (b_th is then ignored)
 * Everything else as snn_lif_forward; trace_out must not overlap the other buffers.
 */
snn_status snn_lif_forward_traces(const uint8_t* s_in, const float* W, int T, int B, int N_in, int N_out,
                                  float alpha, float theta, float b_th, float* V, uint8_t* s_out,
                                  float* trace_in, float* trace_out, float alpha_next, uint64_t* active_bits,
                                  void* stream);

/*
 * Active-set compaction (Definition 1) with the truncated spike derivative (Definition 2).
 *   V        [T,B,N] float32 (read)
 *   active   |V - theta| < b_th in float32, strictly (b_th = +INFINITY: every finite V)
 *   row_ptr  int32 [T*B + 1] (written): exclusive prefix of per-row counts, row_ptr[T*B] = nnz
 *   col_idx  int32 [capacity] (written): neuron index n of each active entry, ascending in a row
 *   g_act    float32 [capacity] (written unless NULL): 1/(beta |V - theta| + 1)^2 at each entry
 *   capacity length of col_idx / g_act; entries at positions >= capacity are not written
 *   nnz_dev  int64 [1] device (written): the true nnz, even when it exceeds capacity. The
 *            caller checks nnz <= capacity after the stream has run.
 * Integer outputs are a deterministic function of V.
 */
size_t snn_active_compact_workspace(int T, int B, int N);
snn_status snn_active_compact(const float* V, int T, int B, int N, float theta, float b_th, float beta,
                              int32_t* row_ptr, int32_t* col_idx, float* g_act, int64_t capacity,
                              int64_t* nnz_dev, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Compaction from the bitset of snn_lif_forward_active: the same CSR as snn_active_compact with
 * the band used for the bitset (row_ptr, col_idx ascending, g_act = 1/(beta|V-theta|+1)^2 read
 * from V at the active entries only). V may be NULL when g_act is NULL. Capacity, nnz and
 * overflow behave as in snn_active_compact. SNN_ERR_UNSUPPORTED when T*B > 8,388,608 rows.
 */
size_t snn_active_compact_bits_workspace(int T, int B, int N);
snn_status snn_active_compact_bits(const uint64_t* active_bits, const float* V, int T, int B, int N,
                                   float theta, float beta, int32_t* row_ptr, int32_t* col_idx,
                                   float* g_act, int64_t capacity, int64_t* nnz_dev, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * snn_active_compact_bits without a workspace argument and without any allocation, for callers
 * that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments (minus workspace) and results. The row
 * counts and scan temporaries live in a device array of the library, 8 MiB, one per GPU, held
 * until the process ends; its address is looked up on the first call on each device.
 *   SNN_ERR_UNSUPPORTED when snn_active_compact_bits_workspace(T, B, N) exceeds 8 MiB (about
 *   T*B > 2,000,000 rows); SNN_ERR_HIP when the array's address cannot be had.
 * Every call on one GPU shares that array: calls that overlap on a GPU (on different streams or
 * host threads) race and give wrong results; calls in order on one stream are safe.
 */
snn_status snn_active_compact_bits_noalloc(const uint64_t* active_bits, const float* V, int T, int B, int N,
                                           float theta, float beta, int32_t* row_ptr, int32_t* col_idx,
                                           float* g_act, int64_t capacity, int64_t* nnz_dev, void* stream);

/*
 * Sparse backward of one layer (Sec. 2.2: sparse dW and sparse spike gradient, Proposition 1).
 *   W          [N_in,N_out] float32 (read)
 *   trace_in   [T,B,N_in]  float32 input trace from snn_lif_forward (read)
 *   alpha      the layer's leak factor
 *   out_*      CSR of this layer's active set (from snn_active_compact, or from snn_readout_ce
 *              for the readout): out_row_ptr [T*B+1], out_col_idx / out_g / eps_out [out_cap].
 *              out_g NULL means a derivative factor of 1 (the readout). eps_out is the loss
 *              gradient w.r.t. this layer's spikes at each entry. G = eps_out * out_g.
 *   in_*       CSR of the INPUT layer's active set, in_row_ptr [T*B+1], in_col_idx [in_cap];
 *              NULL for the first layer (no spike gradient is propagated to the data).
 *   eps_in     float32 [in_cap] (written unless in_* is NULL): sum_j W_ij delta_j[t] at each
 *              input-active entry (t,b,i), aligned with in_col_idx -- the next call's eps_out.
 *   dW         [N_in,N_out] float32 (overwritten).
 *   out_cap / in_cap are the allocated lengths of the entry arrays; entries at or beyond them
 *   are ignored, so a CSR whose compaction overflowed its capacity is read safely (and gives
 *   a truncated result). The CSRs are expected as the compaction writes them: row_ptr
 *   non-decreasing, columns strictly ascending inside a row. Entries with a column outside
 *   [0, N) are skipped; for other malformed input the results are unspecified, but every memory
 *   access stays inside the arrays and workspace given (indices are clamped).
 *   Workspace: for layers of 33..300 outputs and at most 1024 inputs it holds per-chunk partial
 *   dW only (the dW kernel reads the CSR directly) and does not depend on out_cap; for other
 *   layers of more than 32 outputs its size depends on out_cap (a slab-major or window-sorted
 *   copy of the active entries is built in it); for N_out <= 32 (narrow layers: G written
 *   densely, padded to 8, 16 or 32 columns) it holds that G and delta (T*B*ld floats each), a
 *   bitset of the rows with an entry and per-chunk partial dW, and does not depend on out_cap.
 *   aux_stream (may be NULL): a second hipStream_t. When given, the spike-gradient part runs on
 *   it beside the dW part on `stream`; the call makes aux_stream wait for the work already on
 *   `stream`, and `stream` wait for the aux work, so work enqueued on `stream` afterwards sees
 *   both results. The fork and join use two HIP events per device and host thread, created by
 *   the first such call and kept until the thread ends; no call creates or destroys events or
 *   synchronises the host. SNN_ERR_HIP when the fork or the join cannot be enqueued (after a
 *   failed join, work enqueued later on `stream` is not ordered after eps_in).
 * Supported: N_out <= 4096.
 */
size_t snn_sparse_backward_workspace(int T, int B, int N_in, int N_out, int64_t out_cap);
snn_status snn_sparse_backward(const float* W, const float* trace_in, int T, int B, int N_in, int N_out,
                               float alpha, const int32_t* out_row_ptr, const int32_t* out_col_idx,
                               const float* out_g, const float* eps_out, int64_t out_cap,
                               const int32_t* in_row_ptr, const int32_t* in_col_idx, int64_t in_cap,
                               float* eps_in, float* dW, void* workspace, size_t workspace_bytes,
                               void* stream, void* aux_stream);

/*
 * The two halves of snn_sparse_backward as calls of their own, for callers that schedule them
 * on different streams (the combined call does this itself when given aux_stream). Arguments
 * mean the same as in snn_sparse_backward; the results are the same as its results.
 *
 * snn_sparse_dw: dW of one layer (sparse form of Eq. (w_grad)), overwriting dW [N_in,N_out].
 *   Needs no W. Workspace from snn_sparse_dw_workspace (depends on out_cap).
 * snn_sparse_grad_in: the spike gradient eps_in at the input layer's active entries (sparse
 *   form of Eq. (s_grad) with Proposition 1's recurrence). in_row_ptr is required; nothing is
 *   written when in_cap = 0. share_cu != 0 keeps the walk to two blocks per compute unit, so
 *   that a kernel launched beside it on another stream (dW) finds room; 0 uses the whole GPU.
 *   Workspace from snn_sparse_grad_in_workspace.
 * The two calls use separate workspaces and may run concurrently.
 */
size_t snn_sparse_dw_workspace(int T, int B, int N_in, int N_out, int64_t out_cap);
snn_status snn_sparse_dw(const float* trace_in, int T, int B, int N_in, int N_out,
                         const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* out_g,
                         const float* eps_out, int64_t out_cap, float* dW, void* workspace,
                         size_t workspace_bytes, void* stream);
/*
 * snn_sparse_dw in two parts, so that the part that needs only the active set's structure can
 * run early (right after compaction, before any eps exists) and off the critical path:
 * snn_sparse_dw_layout reads out_row_ptr and out_col_idx only and writes the per-(row, column
 * slab) entry counts and offsets (or, for N_out <= 32, the bitset of rows with an entry; for
 * layers that take the CSR-direct dW, nothing) into the workspace; snn_sparse_dw_prepared then does the rest of snn_sparse_dw (arguments as there) and
 * gives the same dW bit for bit, provided the layout ran on the same workspace with a CSR of the
 * same structure (row pointers and columns) and out_cap, and the workspace was not used in
 * between. Workspace from snn_sparse_dw_workspace. Errors as snn_sparse_dw.
 */
snn_status snn_sparse_dw_layout(int T, int B, int N_in, int N_out, const int32_t* out_row_ptr,
                                const int32_t* out_col_idx, int64_t out_cap, void* workspace,
                                size_t workspace_bytes, void* stream);
snn_status snn_sparse_dw_prepared(const float* trace_in, int T, int B, int N_in, int N_out,
                                  const int32_t* out_row_ptr, const int32_t* out_col_idx, const float* out_g,
                                  const float* eps_out, int64_t out_cap, float* dW, void* workspace,
                                  size_t workspace_bytes, void* stream);
size_t snn_sparse_grad_in_workspace(int T, int B, int N_out);
snn_status snn_sparse_grad_in(const float* W, int T, int B, int N_in, int N_out, float alpha,
                              const int32_t* out_row_ptr, const int32_t* out_col_idx,
                              const float* out_g, const float* eps_out, int64_t out_cap,
                              const int32_t* in_row_ptr, const int32_t* in_col_idx, int64_t in_cap,
                              float* eps_in, int share_cu, void* workspace, size_t workspace_bytes,
                              void* stream);

/*
 * Trace recompute: dW without the stored input trace. The trace of Eq. (w_grad) obeys
 * trace[0] = 0, trace[t+1] = alpha trace[t] + S_in[t] (Sec. 2; float32, product and sum each
 * rounded, as the forward computes it), so it is determined by the input spikes and its values
 * at every K-th step.
 *
 * snn_trace_checkpoints: ck [ceil(T/K), B, N_in] float32 (written): ck[q] = trace[q K], from
 *   s_in [T,B,N_in] uint8 (read; nonzero = spike) with the forward's recurrence (bit-identical
 *   to the trace snn_lif_forward writes). snn_trace_checkpoint_count(T, K) = ceil(T/K).
 * snn_sparse_dw_spikes: the same dW as snn_sparse_dw (same CSR arguments), reading s_in and ck
 *   (with the K and alpha they were made with) instead of trace_in: each block rebuilds the trace
 *   values it needs in registers from the checkpoint at the start of its steps. The traces used
 *   are bit-identical to the stored ones; dW can differ from snn_sparse_dw's in the last bit only
 *   (float64 accumulation in another order). Memory: B N_in (ceil(T/K) floats + T bytes of
 *   spikes the forward keeps anyway) instead of T B N_in floats. Any N_out <= 4096 (narrow
 *   layers too, through the slab kernel). Errors: SNN_ERR_INVALID_ARG for NULL pointers, K < 1,
 *   alpha outside (0, 1], bad sizes or a short workspace; SNN_ERR_UNSUPPORTED for N_out > 4096.
 */
int64_t snn_trace_checkpoint_count(int T, int K);
snn_status snn_trace_checkpoints(const uint8_t* s_in, int T, int B, int N_in, float alpha, int K, float* ck,
                                 void* stream);
size_t snn_sparse_dw_spikes_workspace(int T, int B, int N_in, int N_out, int64_t out_cap, int K);
snn_status snn_sparse_dw_spikes(const uint8_t* s_in, const float* ck, int K, float alpha, int T, int B, int N_in,
                                int N_out, const int32_t* out_row_ptr, const int32_t* out_col_idx,
                                const float* out_g, const float* eps_out, int64_t out_cap, float* dW,
                                void* workspace, size_t workspace_bytes, void* stream);


/*
 * Dense surrogate BPTT of one layer on matrix cores: the baseline the sparse rule is
 * measured against (Table 1, "Original").
 *   W, trace_in as above; V [T,B,N_out] (read); eps_out [T,B,N_out] dense loss gradient
 *   w.r.t. this layer's spikes (read).
 *   G = eps_out * g(V) * 1[|V - theta| < b_th]; b_th = +INFINITY gives full surrogate BPTT;
 *   theta = +INFINITY marks the readout, whose factor is 1 (G = eps_out).
 *   grad_in [T,B,N_in] float32 (written unless NULL) = delta W^T, unmasked.
 *   dW [N_in,N_out] float32 (overwritten) = sum_t trace_in[t]^T G[t].
 */
size_t snn_dense_backward_workspace(int T, int B, int N_in, int N_out);
snn_status snn_dense_backward_ref(const float* W, const float* trace_in, const float* V,
                                  const float* eps_out, int T, int B, int N_in, int N_out, float alpha,
                                  float theta, float b_th, float beta, float* grad_in, float* dW,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Readout loss helper (App. E cross-entropy), outside the measured backward.
 *   V_out  [T,B,C] float32 readout membrane potential (read); labels int32 [B] device (read)
 *   mode 0 logits a[b,c] = max_t V_out[t,b,c] (first maximal t); mode 1 a = sum_t V_out.
 *   loss   float32 [1] device (written): mean over b of -log softmax(a)[b, label_b];
 *          NaN if a label is outside [0, C).
 *   CSR of the entries the loss reads, with eps = dL/da = (p - onehot)/B there:
 *   mode 0 nnz = B*C (the arg-max entries), mode 1 nnz = T*B*C (every entry);
 *   row_ptr int32 [T*B+1], col_idx int32 [nnz], eps float32 [nnz] (written).
 *   eps_dense [T,B,C] float32 (written unless NULL): dL/dV_out densely (zero where the loss
 *   does not read V_out), the input of the dense baseline's readout step.
 */
size_t snn_readout_ce_workspace(int T, int B, int C, int mode);
snn_status snn_readout_ce(const float* V_out, const int32_t* labels, int T, int B, int C, int mode,
                          int32_t* row_ptr, int32_t* col_idx, float* eps, float* loss, float* eps_dense,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * Activity penalties of App. E on one LIF layer's spikes (training step, outside the measured
 * backward). With zeta[b,i] = number of nonzero S[t,b,i] over t and, per sample,
 *   R_low[b] = (lam_low/N) sum_i max(0, nu_low - zeta[b,i])^2,
 *   R_up[b]  = lam_up max(0, (1/N) sum_i zeta[b,i] - nu_up)
 * (the appendix prints both negated, as terms to maximise; these are the penalties minimised),
 * the loss gains (1/B) sum_b (R_low[b] + R_up[b]).
 *   S        [T,B,N] uint8 spikes of the layer (read)
 *   zeta     int32 [B,N] (written unless NULL): the spike counts
 *   coef     float32 [B,N] (written): d loss / d zeta[b,i] =
 *            (-2 lam_low/N max(0, nu_low - zeta) + [mean_i zeta[b,i] > nu_up] lam_up/N) / B,
 *            which is also d loss / d S[t,b,i] at every t (slope 0 at the hinges)
 *   penalty  float32 [1] device (written unless NULL): (1/B) sum_b (R_low[b] + R_up[b])
 * lam_low, lam_up must be finite and >= 0, nu_low, nu_up finite; otherwise SNN_ERR_INVALID_ARG.
 * Sums are formed in float64 in a fixed order: outputs are deterministic.
 */
size_t snn_activity_reg_workspace(int T, int B, int N);
snn_status snn_activity_reg(const uint8_t* S, int T, int B, int N, float lam_low, float nu_low, float lam_up,
                            float nu_up, int32_t* zeta, float* coef, float* penalty, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Adds the penalties' gradient to a layer's spike gradient (App. E; the count is a sum over t,
 * so coef[b,i] joins the gradient w.r.t. S[t,b,i] at every t).
 *   coef     float32 [B,N] from snn_activity_reg (read)
 *   row_ptr, col_idx, capacity: the layer's active-set CSR (rows r = t*B + b); then eps is
 *            float32 [capacity], the spike gradient at those entries (snn_sparse_backward's
 *            eps_in), and eps[e] += coef[b, col_idx[e]] for e < min(row_ptr[T*B], capacity).
 *            Columns outside [0, N) are skipped.
 *   row_ptr NULL: eps is the dense [T,B,N] gradient and eps[t,b,i] += coef[b,i] everywhere.
 * No workspace; nothing is allocated.
 */
snn_status snn_activity_reg_grad(const float* coef, int T, int B, int N, const int32_t* row_ptr,
                                 const int32_t* col_idx, int64_t capacity, float* eps, void* stream);

/*
 * One Adam step on a float32 tensor of n elements (App. E's optimiser; Kingma and Ba,
 * Algorithm 1), in place:
 *   m = beta1 m + (1-beta1) grad;  v = beta2 v + (1-beta2) grad^2;
 *   W -= lr/(1-beta1^step) * m / (sqrt(v/(1-beta2^step)) + eps)
 * step counts from 1; m and v start at zero. The bias corrections are formed in float64 on
 * the host, the rest in float32. All four arrays are device float32 [n]; grad is read only.
 * SNN_ERR_INVALID_ARG for step < 1, n <= 0, lr < 0, betas outside [0, 1), eps <= 0, or
 * non-finite hyper-parameters.
 */
snn_status snn_adam_step(float* W, const float* grad, float* m, float* v, int64_t n, float lr, float beta1,
                         float beta2, float eps, int step, void* stream);

/*
 * Convolutional LIF layer, forward (the convolutional experiment of Sec. 3; App. E: 3x3 filters,
 * stride 1). Zero padding 1, channels last.
 *   s_in   [T,B,H,W,C] uint8 input spikes (read; nonzero = spike)
 *   Wc     [3,3,C,F] float32 filters (ky, kx, c, f); output (y, x) reads input (y+ky-1, x+kx-1)
 *   V      [T,B,H*W*F] float32 (written), neuron n = (y*W + x)*F + f
 *   s_out  [T,B,H*W*F] uint8 spikes (written)
 *   trace_in [T,B,H*W*C] float32 input trace (written unless NULL)
 *   active_bits (written unless NULL): the active set with band b_th, in the layout of
 *          snn_lif_forward_active with N = H*W*F (snn_active_bits_words(T, B, H*W*F) words)
 * The layer is a LIF layer whose weighted input is the convolution (its Toeplitz matrix): the
 * weighted input is summed over spiking inputs in ascending input index (y', x', c) in float32
 * from +0.0, then the recurrence of snn_lif_forward; results are bit-identical to
 * snn_lif_forward on that matrix.
 */
snn_status snn_conv_lif_forward(const uint8_t* s_in, const float* Wc, int T, int B, int H, int W, int C, int F,
                                float alpha, float theta, float b_th, float* V, uint8_t* s_out, float* trace_in,
                                uint64_t* active_bits, void* stream);

/*
 * 2x2 max pooling (stride 2) of a convolutional layer's spikes [T,B,H,W,F] (H, W even):
 *   P   [T,B,H/2,W/2,F] uint8 (written): OR of the window
 *   arg [T,B,H/2,W/2,F] uint8 (written): window position (0..3, row-major) of the first spike,
 *       0 when none; the window's gradient goes to that element (first maximal element).
 */
snn_status snn_maxpool_spikes(const uint8_t* S, int T, int B, int H, int W, int F, uint8_t* P, uint8_t* arg,
                              void* stream);

/*
 * The pooled layer's share of the active set: pooled neuron (t, b, np) is active iff the conv
 * neuron its pooling picked (arg) is active in conv_bits. Both bitsets in the layout of
 * snn_lif_forward_active (N = H*W*F for conv_bits, (H/2)*(W/2)*F for pool_bits, written).
 * snn_active_compact_bits(pool_bits, V = NULL, ..., g_act = NULL) gives its CSR, the input-side
 * CSR of the readout's snn_sparse_backward.
 */
snn_status snn_pool_route_bits(const uint64_t* conv_bits, const uint8_t* arg, int T, int B, int H, int W, int F,
                               uint64_t* pool_bits, void* stream);

/*
 * Routes the readout's spike gradient at the pooled entries (eps_pool, aligned with the pooled
 * CSR) to the conv layer's CSR: eps_conv[e] = eps_pool of the pooled entry whose pooling picked
 * conv entry e, else 0. eps_conv float32 [conv_cap] (written for e < conv_cap). Entries past the
 * capacities are ignored; columns are found by binary search (rows ascending, as compaction
 * writes them).
 */
snn_status snn_pool_scatter_eps(int T, int B, int H, int W, int F, const int32_t* pool_row_ptr,
                                const int32_t* pool_col_idx, int64_t pool_cap, const float* eps_pool,
                                const uint8_t* arg, const int32_t* conv_row_ptr, const int32_t* conv_col_idx,
                                int64_t conv_cap, float* eps_conv, void* stream);

/* Dense form: eps_conv [T,B,H*W*F] (written) from eps_pool [T,B,(H/2)*(W/2)*F] (read). */
snn_status snn_pool_scatter_eps_dense(const float* eps_pool, const uint8_t* arg, int T, int B, int H, int W, int F,
                                      float* eps_conv, void* stream);

/*
 * Sparse filter gradient of the convolutional layer (Eq. (w_grad) with the filter's shared
 * weights): dWc[ky,kx,c,f] = sum over its active entries (t,b,y,x,f) of eps*g times
 * trace_in[t,b,y+ky-1,x+kx-1,c]. conv CSR and g from snn_active_compact_bits; eps_conv from
 * snn_pool_scatter_eps; conv_g may be NULL (g = 1). dWc [3,3,C,F] float32 (overwritten).
 * SNN_ERR_UNSUPPORTED when C*F > 2048. Float64 accumulation.
 */
size_t snn_conv_sparse_dw_workspace(int T, int B, int H, int W, int C, int F);
snn_status snn_conv_sparse_dw(const float* trace_in, int T, int B, int H, int W, int C, int F,
                              const int32_t* conv_row_ptr, const int32_t* conv_col_idx, const float* conv_g,
                              const float* eps_conv, int64_t conv_cap, float* dWc, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * The same filter gradient from the pooled CSR alone, for a conv layer whose spikes reach the
 * loss only through the 2x2 pooling (no other term on the conv spikes, such as the activity
 * penalty): then an active conv neuron has a nonzero gradient only where its pooling picked it
 * for an active pooled entry, and those are exactly the pooled CSR's entries (snn_pool_route_bits
 * and compaction). Pooled entry (t,b,np) with gradient eps_pool stands for conv neuron
 * (t,b,2 py + arg/2, 2 px + arg%2, f) (np = (py (W/2) + px) F + f, arg from snn_maxpool_spikes),
 * G = eps_pool * g(V) there, g = 1/(beta |V - theta| + 1)^2 with the compaction's float32
 * operations and G = 0 outside |V - theta| < b_th. No conv-layer CSR and no routing call are
 * needed. V [T,B,H*W*F] float32, arg [T,B,(H/2)*(W/2)*F] uint8 (read). Workspace, dWc, errors
 * and accumulation as snn_conv_sparse_dw (SNN_ERR_INVALID_ARG also for a NaN theta, b_th or
 * beta, or a negative b_th or beta). Columns outside [0, (H/2)*(W/2)*F) are ignored.
 */
snn_status snn_conv_sparse_dw_pooled(const float* trace_in, const float* V, const uint8_t* arg, int T, int B, int H,
                                     int W, int C, int F, float theta, float b_th, float beta,
                                     const int32_t* pool_row_ptr, const int32_t* pool_col_idx, const float* eps_pool,
                                     int64_t pool_cap, float* dWc, void* workspace, size_t workspace_bytes,
                                     void* stream);

/*
 * Dense filter gradient (the baseline): every neuron's G = eps_conv * g(V) * [|V - theta| < b_th]
 * (b_th = +INFINITY: full surrogate) with eps_conv dense [T,B,H*W*F], then the same sum.
 * SNN_ERR_UNSUPPORTED when C*F > 2^20.
 */
size_t snn_conv_dense_dw_workspace(int T, int B, int H, int W, int C, int F);
snn_status snn_conv_dense_dw(const float* trace_in, const float* V, const float* eps_conv, int T, int B, int H, int W,
                             int C, int F, float theta, float b_th, float beta, float* dWc, void* workspace,
                             size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SNN_H */
