/*
 * zsa.h -- C interface of libzsa, the MI355X (gfx950) pruned layer-stack
 * forward of "Efficient Large Language Models with Zero-Shot Adjustable
 * Acceleration" (Kachuee & Sharifkhani).
 *
 * The method (Sec. 3.2-3.4): at a pruning layer every hidden activation (one
 * row of the hidden state per sequence position) is scored by the weight its
 * V row receives from the attention soft-score matrix softmax(QK^T/sqrt(d_k)
 * + M) (Eq. 1); only the N_l = max(alpha * N_{l-1}, tau) highest-scoring rows
 * (Eq. 2) are kept, and every later layer runs on the shorter sequence. The
 * keep rate alpha is an ordinary per-call argument (zero-shot: no retraining
 * is needed to change it, Sec. 3.4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Sequences are packed without padding: sequence b owns rows
 *    cu[b] .. cu[b+1]-1 of a [T, width] row-major array, cu[0] = 0,
 *    cu non-decreasing, cu[batch] = T. Functions take the offsets twice:
 *    `cu_host` (host memory, used for shapes and validation) and `cu_dev`
 *    (device memory, same values, read by kernels).
 *  - `dtype` is ZSA_F32 (float) or ZSA_BF16 (bfloat16 stored as uint16). It
 *    is the storage type of hidden rows, weights, Q/K/V and outputs;
 *    accumulation, softmax, log-sum-exp and scores are always fp32.
 *  - Device pointers are owned by the caller (e.g. torch tensors); the
 *    library never allocates device memory. Scratch memory comes from the
 *    caller's `ws` buffer of `ws_bytes`; the matching *_workspace_size call
 *    gives the minimum.
 *  - `stream` is a hipStream_t (NULL = the default stream). Work is only
 *    enqueued; nothing synchronises the host, so a call may be captured in a
 *    HIP graph. Calls on one stream are ordered; calls sharing a workspace
 *    must not run concurrently.
 *  - Hidden rows, weights and Q/K/V must be 16-byte aligned and rows must be
 *    a multiple of 16 bytes long.
 *  - Row indices are int32; pos[] holds each row's original sequence
 *    position (0 .. n_b-1 before any pruning) and travels with the row.
 *  - The rows one attention call reads for a sequence (its longest sequence,
 *    plus 256 rows, times the Q/K/V row stride) and the rows of one
 *    key/value cache slot must span less than 4 GiB: the kernels address
 *    them with 32-bit offsets. Larger calls return ZSA_EUNSUPPORTED.
 *  - Every entry point validates its arguments before it enqueues anything:
 *    on a validation error nothing is written and a negative status is
 *    returned; zsa_last_error() then describes it (thread-local). Faults in
 *    enqueued kernels surface at the caller's next synchronisation.
 */
#ifndef ZSA_H_
#define ZSA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
enum {
  ZSA_OK = 0,
  ZSA_EINVAL = -1,       /* bad value: NULL pointer, keep rate outside [0,1] or NaN, tau < 1 ... */
  ZSA_ESHAPE = -2,       /* inconsistent sizes (cu not monotone, k > n, T mismatch, ...) */
  ZSA_EALIGN = -3,       /* pointer or row length not a multiple of 16 bytes */
  ZSA_EUNSUPPORTED = -4, /* valid but unsupported configuration */
  ZSA_EWORKSPACE = -5,   /* workspace smaller than the *_workspace_size minimum */
  ZSA_EHIP = -6          /* a HIP runtime call or kernel launch failed */
};

enum { ZSA_F32 = 0, ZSA_BF16 = 1 };

/* block kinds (the two attention forms of Sec. 3.2 on the common pre-norm
 * backbone of Appendix A, Table 1) */
enum {
  ZSA_ENCODER = 0, /* LayerNorm, biases, exact GELU MLP, no positional rotation */
  ZSA_DECODER = 1  /* RMSNorm, rotary Q/K (rotate-half pairs (i, i+hd/2)), SwiGLU MLP */
};

enum { ZSA_NORM_LAYER = 0, ZSA_NORM_RMS = 1 };

/* epilogues of zsa_linear (applied to z = x W^T + bias, fp32) */
enum {
  ZSA_EPI_NONE = 0,     /* y = z */
  ZSA_EPI_GELU = 1,     /* y = z * Phi(z) (exact, erf-based GELU) */
  ZSA_EPI_SWIGLU = 2,   /* y[:, f] = silu(z[:, 2f]) * z[:, 2f+1]; y has n/2 columns */
  ZSA_EPI_RESIDUAL = 3, /* y = residual + z (residual may alias y) */
  ZSA_EPI_ROPE = 4      /* columns < rope_cols rotated per head by pos (as in the decoder) */
};

/* kernel classes for the optional timing hook */
enum {
  ZSA_K_GEMM = 0, ZSA_K_ATTENTION = 1, ZSA_K_SCORE = 2, ZSA_K_SELECT = 3,
  ZSA_K_GATHER = 4, ZSA_K_NORM = 5, ZSA_K_MISC = 6, ZSA_K_NCLASS = 7
};

/* One transformer block (pre-norm residual, Appendix A). */
typedef struct zsa_layer_cfg {
  int32_t kind;       /* ZSA_ENCODER or ZSA_DECODER */
  int32_t d_model;    /* hidden width d */
  int32_t n_heads;    /* H; head_dim * n_heads == d_model */
  int32_t head_dim;   /* hd = d_k of Eq. 1; even; attention scale 1/sqrt(hd) */
  int32_t d_ff;       /* MLP width F */
  int32_t causal;     /* 1: causal mask M (row i sees rows j <= i), 0: M = 0 (Eq. 1) */
  int32_t dtype;      /* ZSA_F32 or ZSA_BF16 */
  int32_t tau;        /* floor of Eq. 2 (the paper fixes it at 5, Sec. 4.2) */
  float norm_eps;     /* LayerNorm / RMSNorm epsilon */
  float rope_theta;   /* rotary base (decoder) */
  int32_t n_kv_heads; /* key/value heads, dividing n_heads (grouped-query
                         attention of the LLaMA 3 / Gemma 2 backbones, Table 1);
                         0 means n_heads, 1 is multi-query attention */
  int32_t force_keep_last; /* nonzero: every pruning point keeps the last row
                              of each sequence (the row the first generated
                              token is predicted from) and chooses the other
                              k - 1 rows by score */
  int32_t mark_only;  /* nonzero: the visualisation mode of Appendix B --
                         pruning points mark their kept rows (kept_rows_out,
                         pos_dbg) but remove none, so every row continues
                         and the outputs are those of the unpruned stack;
                         each point ranks all rows and marks the Eq. 2 count
                         of the previous point's marked count (a row can be
                         marked again after being passed over) */
} zsa_layer_cfg;

/* Weights of one block, device pointers in the storage dtype, PyTorch
 * Linear layout [out, in] (row-major, the input dimension contiguous).
 *   w_qkv  [d + 2*kv*hd, d]  rows q (d) | k (kv*hd) | v (kv*hd), head h at
 *          rows h*hd .. h*hd+hd-1 of its block (kv = key/value heads)
 *   w_o    [d, d]
 *   w_up   encoder [F, d]; decoder [2F, d] with row 2f = gate f, 2f+1 = up f
 *   w_down [d, F]
 *   norm*_w [d] gains; norm*_b [d] LayerNorm shifts (encoder only)
 * Any bias may be NULL (no bias); the decoder ignores norm*_b. */
typedef struct zsa_layer_weights {
  const void *norm1_w, *norm1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  const void *norm2_w, *norm2_b, *w_up, *b_up, *w_down, *b_down;
} zsa_layer_weights;

/* Thread-local text of the last non-OK status ("" if none). */
const char* zsa_last_error(void);
const char* zsa_version(void);

/* ---------------------------------------------------------------------
 * Eq. 2 (Sec. 3.3): rows kept at a pruning layer, N_l = max(alpha N_{l-1}, tau).
 * k = min(n, max(floor(keep_rate * n + 1e-9), tau)), the product and sum in
 * IEEE double without contraction. Host only.
 * Errors: ZSA_EINVAL if keep_rate is NaN or outside [0,1], tau < 1, n < 0 or
 * k_out is NULL.
 */
int zsa_keep_count(int32_t n, double keep_rate, int32_t tau, int32_t* k_out);

/* Eq. 2 compounded over n_points pruning points for a batch: counts_out
 * [n_points * batch] (host), entry p*batch+b = rows of sequence b after
 * point p. lengths[batch], keep_rate[batch] host arrays. Host only. */
int zsa_keep_schedule(int32_t batch, const int32_t* lengths, const double* keep_rate,
                      int32_t tau, int32_t n_points, int32_t* counts_out);

/* ---------------------------------------------------------------------
 * Row normalisation of the pre-norm block (Appendix A): y = LN(x) * gain +
 * shift (kind ZSA_NORM_LAYER; biased variance) or y = x / sqrt(mean(x^2) +
 * eps) * gain (ZSA_NORM_RMS; shift ignored, may be NULL).
 * x, y [rows, d] device, dtype; gain, shift [d]. y must not overlap x.
 * rows = 0 launches nothing; x and y may then be NULL.
 */
int zsa_norm(void* stream, int32_t dtype, int32_t kind, const void* x, const void* gain,
             const void* shift, int32_t rows, int32_t d, float eps, void* y);

/* ---------------------------------------------------------------------
 * Projection y = epilogue(x W^T + bias) for the Q/K/V, output and MLP
 * projections of the block (Appendix A; Eq. 1 inputs). x [m, k], w [n, k],
 * bias [n] or NULL, all dtype, device. y is [m, n] (row stride n), or
 * [m, n/2] for ZSA_EPI_SWIGLU (n even). residual [m, n] for
 * ZSA_EPI_RESIDUAL. ZSA_EPI_ROPE rotates the columns below rope_cols
 * (a multiple of head_dim) in head_dim blocks: channels i and i + hd/2
 * rotate by pos[row] * rope_theta^(-2i/hd); pos [m] int32 device.
 * bf16 uses MFMA tiles; fp32 uses vector ALU tiles.
 * ws (device, 16-byte aligned, caller-owned) or NULL: room for split-K
 * partial sums. When the output tiles of a bf16 product are too few to
 * fill the GPU, K is split into slices whose fp32 partials are summed in a
 * fixed slice order before the epilogue (results are reproducible; they
 * may differ from the unsplit sum in the last bits). A short bf16 product
 * (at most 64 rows, or 256 rows with n and k at most 1024; k a multiple of
 * 32) streams w into the matrix cores, one workgroup per 16 output columns
 * and 16 rows whose waves split K and add their sums in a fixed order (no
 * workspace). With ws NULL the product is never split.
 * ws_bytes below zsa_linear_workspace_size() returns ZSA_EWORKSPACE.
 * ZSA_EPI_ROPE in bf16: a workspace with m * head_dim * 4 more bytes than
 * that (past its 256-byte rounded size) lets the call first tabulate each
 * row's rotary (cos, sin) pairs there, which long products then read
 * instead of forming the angles themselves (same values).
 * m = 0 reads and writes nothing and launches nothing; x, y, residual and
 * pos may then be NULL (the other arguments are still checked).
 */
int zsa_linear(void* stream, int32_t dtype, const void* x, int32_t m, int32_t k, const void* w,
               int32_t n, const void* bias, int32_t epilogue, const void* residual,
               const int32_t* pos, int32_t head_dim, int32_t rope_cols, float rope_theta,
               void* y, void* ws, size_t ws_bytes);

/* Bytes of split-K workspace zsa_linear uses for this shape (0: none). */
size_t zsa_linear_workspace_size(int32_t dtype, int32_t m, int32_t n, int32_t k);

/* ---------------------------------------------------------------------
 * Attention of Eq. 1, per sequence and head, over packed varlen rows, and
 * optionally the contribution score of every row (Sec. 3.2-3.3):
 *     scores[j] = sum over heads h, query rows i of P_h[i, j],
 * P_h = softmax(Q_h K_h^T * scale + M) the normalised soft-score matrix.
 * P is never written to memory.
 *   q, k, v  device, dtype; row r of query head h starts at
 *            q + r*row_stride + h*hd, row r of key/value head g at
 *            k + r*row_stride + g*hd (and v); row_stride in elements
 *   n_kv_heads  key/value heads (divides n_heads; 0 means n_heads): query
 *            head h reads key/value head h / (n_heads / n_kv_heads)
 *   out      [T, n_heads*hd] dtype, row stride out_stride (elements)
 *   lse      [n_heads, T] fp32: natural-log log-sum-exp of each scaled,
 *            masked score row; NULL if not wanted
 *   scores   [T] fp32 or NULL (then no scoring pass runs)
 *   causal   mask by row order within the sequence (rows must be in
 *            ascending original position, as compaction keeps them)
 *   ws       >= zsa_attention_workspace_size(n_heads, T, want_scores)
 * bf16 with head_dim 64 or 128 runs the MFMA kernels; other shapes and fp32
 * run vector-ALU kernels. Sequences may be empty; with T = 0 (all of them)
 * nothing is launched and q, k, v, out may be NULL.
 */
int zsa_attention_with_scores(void* stream, int32_t dtype, const void* q, const void* k,
                              const void* v, int64_t row_stride, int32_t n_heads,
                              int32_t n_kv_heads, int32_t head_dim, int32_t causal, float scale,
                              int32_t batch, const int32_t* cu_host, const int32_t* cu_dev,
                              void* out, int64_t out_stride, float* lse, float* scores, void* ws,
                              size_t ws_bytes);
size_t zsa_attention_workspace_size(int32_t n_heads, int32_t total_rows, int32_t want_scores);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * call and result as zsa_attention_with_scores, with its scratch (the
 * score partials and, when lse is NULL, the log-sum-exp rows) in a static
 * device buffer of zsa_static_scratch_bytes() bytes (32 MiB) that the
 * library holds on every GPU it runs on until the process ends. It
 * allocates nothing and needs no workspace. A call whose scratch would not
 * fit (zsa_attention_workspace_size above the buffer; with scores about
 * n_heads * T <= 4 Mi) returns ZSA_EUNSUPPORTED before any launch. Every
 * call on one GPU shares that GPU's buffer: calls that may overlap on one
 * GPU (other streams, other threads) race and must not be issued. Nothing
 * in the buffer needs to start at zero: a call reads only what it wrote. */
int zsa_attention_with_scores_static(void* stream, int32_t dtype, const void* q, const void* k,
                                     const void* v, int64_t row_stride, int32_t n_heads,
                                     int32_t n_kv_heads, int32_t head_dim, int32_t causal,
                                     float scale, int32_t batch, const int32_t* cu_host,
                                     const int32_t* cu_dev, void* out, int64_t out_stride,
                                     float* lse, float* scores);
size_t zsa_static_scratch_bytes(void);

/* Contribution scores alone, from Q, K and the attention's log-sum-exp
 * (Sec. 3.2-3.3): scores[j] = sum_h sum_i exp(q_i . k_j * scale - lse[h, i]),
 * the sum over the rows i allowed by the mask. Deterministic (fixed
 * reduction order, no atomics). Arguments as in zsa_attention_with_scores;
 * lse [n_heads, T] fp32 device. ws >= zsa_score_workspace_size(n_heads, T).
 * With T = 0 nothing is launched and q, k, lse, scores may be NULL. */
int zsa_score_positions(void* stream, int32_t dtype, const void* q, const void* k,
                        int64_t row_stride, const float* lse, int32_t n_heads,
                        int32_t n_kv_heads, int32_t head_dim, int32_t causal, float scale,
                        int32_t batch, const int32_t* cu_host, const int32_t* cu_dev,
                        float* scores, void* ws, size_t ws_bytes);
size_t zsa_score_workspace_size(int32_t n_heads, int32_t total_rows);

/* ---------------------------------------------------------------------
 * Keep the k_host[b] highest-scoring rows of every sequence (Sec. 3.3).
 * Order: score descending, ties to the lower row; -0.0 equals +0.0; NaN
 * scores give an unspecified (but in-bounds) result. Output: kept_rows
 * [sum k] device int32, the global row ids (into the packed input) of the
 * kept rows, sequence by sequence, ascending within each sequence.
 *   scores [T] fp32 device; k_host [batch] host, 0 <= k_host[b] <= n_b
 *   force_keep_last  nonzero: the last row of every sequence is kept
 *            (when k_host[b] >= 1) and the other k - 1 are chosen by score
 *   ws >= zsa_select_workspace_size(batch)
 */
int zsa_select_topk(void* stream, const float* scores, int32_t batch, const int32_t* cu_host,
                    const int32_t* cu_dev, const int32_t* k_host, int32_t force_keep_last,
                    int32_t* kept_rows, void* ws, size_t ws_bytes);
size_t zsa_select_workspace_size(int32_t batch);

/* Compaction after pruning (Sec. 3.3: pruned rows take no part in later
 * layers): hidden_out[r] = hidden[kept_rows[r]], pos_out[r] =
 * pos[kept_rows[r]] for r < t_out. hidden [t_in, d] dtype, pos [t_in] int32
 * (or NULL together with pos_out), kept_rows [t_out], outputs must not
 * overlap inputs. An index outside [0, t_in) yields a zero row and pos -1. */
int zsa_compact_gather(void* stream, int32_t dtype, const void* hidden, int32_t d,
                       const int32_t* pos, int32_t t_in, const int32_t* kept_rows, int32_t t_out,
                       void* hidden_out, int32_t* pos_out);

/* ---------------------------------------------------------------------
 * One pre-norm block over a packed batch, optionally pruning its output.
 *   x1 = x + Attn(Norm1(x)) W_o^T + b_o;  out = x1 + MLP(Norm2(x1))
 * With keep_rate (host [batch]) non-NULL the block is a pruning layer: its
 * attention also yields the contribution scores, the Eq. 2 count of rows
 * (tau from cfg) with the highest scores is kept per sequence, and only
 * those rows are written, in their original order (Sec. 3.3). The rows a
 * pruning layer drops are not carried through the row-wise part of the
 * block (output projection and MLP); the kept rows' values are those of
 * running the whole block and then compacting.
 *   hidden_in [T, d], pos_in [T] int32, cu_host/cu_dev [batch+1]
 *   hidden_out [T', d], pos_out [T'], T' = sum of the kept counts
 *   (zsa_keep_schedule with one point) or T when keep_rate is NULL or
 *   cfg->mark_only is set (then kept_rows_out lists the marked rows)
 *   cu_out_host [batch+1] host, cu_out_dev [batch+1] device: written
 *   scores_out [T] fp32 / kept_rows_out [T'] int32 device, may be NULL
 *   ws >= zsa_layer_workspace_size(cfg, T, batch)
 * hidden_out must not overlap hidden_in.
 */
int zsa_layer_forward(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                      const void* hidden_in, const int32_t* pos_in, int32_t batch,
                      const int32_t* cu_host, const int32_t* cu_dev, const double* keep_rate,
                      void* hidden_out, int32_t* pos_out, int32_t* cu_out_host,
                      int32_t* cu_out_dev, float* scores_out, int32_t* kept_rows_out,
                      void* ws, size_t ws_bytes);
size_t zsa_layer_workspace_size(const zsa_layer_cfg* cfg, int32_t total_rows, int32_t batch);

/* The layer stack: blocks 1..n_layers, w[n_layers]; after every block listed
 * in prune_after (1-based, strictly ascending, n_prune entries) the output is
 * pruned at keep_rate[b] (host [batch]) as in zsa_layer_forward, each count
 * relative to the rows entering that block (Eq. 2 compounded).
 *   hidden_out [T_final, d], pos_out [T_final], cu_out_host/dev [batch+1]
 *   (T_final = T with cfg->mark_only: the rows are marked, not removed;
 *   pos_dbg then lists the positions each point marks)
 *   counts_out_host [n_prune * batch] host or NULL: rows kept per point
 *   scores_dbg fp32 device or NULL: the scores at each pruning point,
 *     concatenated (point p occupies the rows entering that block)
 *   pos_dbg int32 device or NULL: pos after each pruning point, concatenated
 *   hidden_dbg device or NULL: every block's output rows, dtype, concatenated
 *     in block order; block l occupies the rows leaving it (after its pruning
 *     point if it prunes, all current rows otherwise), so the whole buffer
 *     holds sum over blocks of those row counts times d_model elements
 *   kv_cache device or NULL (causal stacks only): the key/value cache a
 *     decode step attends to (see zsa_decode_step). Block l writes the k
 *     (after RoPE) and v of the rows that entered it, sequence b's row r at
 *     ((l * batch + b) * kv_capacity + r) * 2*kvd elements, k in the first
 *     kvd = kv_heads*head_dim and v in the next kvd, dtype. kv_capacity >=
 *     the longest input sequence. The rows a sequence has at block l are
 *     its count after the last pruning point before l.
 *   ws >= zsa_stack_workspace_size(cfg, T, batch, n_prune)
 * No host synchronisation: every shape follows from cu_host and keep_rate.
 * A pruning point at which Eq. 2 keeps every row of every sequence (each at
 * its floor tau, say) keeps them all in order: unless scores_dbg is given,
 * that block then runs unpruned, without the scores, the selection and the
 * gather, which would leave its output unchanged.
 */
int zsa_stack_forward(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                      int32_t n_layers, const int32_t* prune_after, int32_t n_prune,
                      const double* keep_rate, const void* hidden_in, const int32_t* pos_in,
                      int32_t batch, const int32_t* cu_host, const int32_t* cu_dev,
                      void* hidden_out, int32_t* pos_out, int32_t* cu_out_host,
                      int32_t* cu_out_dev, int32_t* counts_out_host, float* scores_dbg,
                      int32_t* pos_dbg, void* hidden_dbg, void* kv_cache, int32_t kv_capacity,
                      void* ws, size_t ws_bytes);
size_t zsa_stack_workspace_size(const zsa_layer_cfg* cfg, int32_t total_rows, int32_t batch,
                                int32_t n_prune);

/* ---------------------------------------------------------------------
 * Gradients of one block's weights: fp32 device pointers, the shapes of
 * zsa_layer_weights. norm*_b and the biases may be NULL (not wanted or not
 * present); the others are required.
 */
typedef struct zsa_layer_grads {
  float *norm1_w, *norm1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  float *norm2_w, *norm2_b, *w_up, *b_up, *w_down, *b_down;
} zsa_layer_grads;

/* Backward pass through the pruned stack (the step the fine-tuning of Eq. 3
 * trains with): for the loss sum(hidden_out * dy), with hidden_out the
 * output of zsa_stack_forward under the same arguments, writes dx [T, d]
 * (the gradient of hidden_in, dtype) and every weight gradient (fp32,
 * overwritten). Every pruning point's kept rows are taken as constants
 * (the selection is not differentiable): rows it drops still receive
 * gradient through that layer's keys and values and the layers before it.
 * The forward is recomputed inside (it is deterministic), layer by layer.
 *   dy [T_final, d] dtype device; grads[n_layers];
 *   ws >= zsa_stack_backward_workspace_size(cfg, T, batch, n_layers, n_prune)
 * bf16 with head_dim 64 or 128, compacting mode; otherwise ZSA_EUNSUPPORTED.
 */
int zsa_stack_backward(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                       const zsa_layer_grads* grads, int32_t n_layers, const int32_t* prune_after,
                       int32_t n_prune, const double* keep_rate, const void* hidden_in,
                       const int32_t* pos_in, int32_t batch, const int32_t* cu_host,
                       const int32_t* cu_dev, const void* dy, void* dx, void* ws,
                       size_t ws_bytes);
size_t zsa_stack_backward_workspace_size(const zsa_layer_cfg* cfg, int32_t total_rows,
                                         int32_t batch, int32_t n_layers, int32_t n_prune);

/* ---------------------------------------------------------------------
 * One generated row per sequence through the stack, after a prefill that
 * filled kv_cache (zsa_stack_forward). Generated rows are never pruned: at
 * block l the new row of sequence b attends (Eq. 1) to the kv_len_host[l *
 * batch + b] rows already in that block's cache (the rows that entered
 * block l in the pruned prefill, then earlier generated rows) and to
 * itself; its own k / v are appended at that row of the cache. The caller
 * adds 1 to every kv_len after the call.
 *   kv_cache [n_layers, batch, kv_capacity, 2 kvd] dtype device, 256-byte
 *   aligned; x_in, x_out [batch, d] dtype device (may alias); pos_host [batch] the
 *   original position of each new row (RoPE); kv_len_host [n_layers*batch]
 *   host, each < kv_capacity; ws >= zsa_decode_workspace_size(cfg,
 *   n_layers, batch, kv_capacity), device, owned by the caller, contents
 *   need not be preserved between calls. Causal stacks, bf16, head_dim 64
 *   or 128, 1/2/4/8 query heads per key/value head; otherwise
 *   ZSA_EUNSUPPORTED. Calls that share a workspace must not overlap.
 */
int zsa_decode_step(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                    int32_t n_layers, int32_t batch, const void* x_in, const int32_t* pos_host,
                    void* kv_cache, int32_t kv_capacity, const int32_t* kv_len_host, void* x_out,
                    void* ws, size_t ws_bytes);
size_t zsa_decode_workspace_size(const zsa_layer_cfg* cfg, int32_t n_layers, int32_t batch,
                                 int32_t kv_capacity);

/* ---------------------------------------------------------------------
 * Timing hook (profiling aid, not thread-safe): while armed, the next
 * `capacity` kernel launches of class `kclass` are bracketed by HIP
 * start/stop events on their own stream. zsa_timing_read synchronises
 * those events and returns the number of launches timed and their summed
 * duration in milliseconds, then disarms. Must not be armed during HIP
 * graph capture.
 */
int zsa_timing_arm(int32_t kclass, int32_t capacity);
int zsa_timing_read(int32_t kclass, int32_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* ZSA_H_ */
