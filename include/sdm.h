/*
 * sdm.h — C ABI of the Sparse Delta Memory (SDM) hot path on MI355X (gfx950).
 *
 * Paper: "Sparse Delta Memory", arXiv 2607.07386.  The layer keeps, per
 * (batch, head) stream, an explicit memory table M of N slots x d_v values.
 * Each token selects W write slots and R read slots by product-key
 * addressing, applies a gated delta-rule write to the W rows only, and reads
 * a weighted sum of the R rows (Sec. 3.1, Eqs. sdm-decay, sdm-write,
 * sdm-read).
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers, contiguous row-major with the
 *     innermost dimension last, at least 16-byte aligned.  Offsets are 64-bit.
 *   - The caller owns every buffer.  The library allocates no device memory;
 *     buffers it needs beyond inputs and outputs come in as `workspace`, sized
 *     by the matching *_workspace_bytes() call.
 *   - `stream` is a hipStream_t (NULL = the default stream).  A return of
 *     SDM_OK means the work was enqueued on it; completion is asynchronous.
 *   - Arguments are validated on the host before anything is launched.  On
 *     any error nothing is launched, no output is touched, the call returns a
 *     negative status and sdm_last_error() (thread-local) describes it.  No
 *     entry point prints, throws or aborts.
 *   - Process-wide state: four geometry switches (sdm_set_scan_slice_width,
 *     sdm_set_scan_line_io, sdm_set_scan_prefetch, sdm_set_chunk_scan_cols)
 *     choose which scan kernel
 *     a later launch runs and so the rounding order of its sums over rows;
 *     the event profiler (sdm_profile_*); and, per device, a second stream
 *     created on first use by the pipelined calls (sdm_forward with more than
 *     one stage, sdm_scan_fwd_chunked with 32 or more chunks, sdm_scan_bwd
 *     with more than one stage), whose enqueueing is serialised by a lock.
 *     Apart from these, calls keep no state between them and are thread safe:
 *     calls on different streams may run concurrently if their buffers do not
 *     overlap (pipelined calls on one device then share its second stream).
 *   - SDM_DEBUG=1 in the environment makes sdm_scan_fwd, sdm_scan_fwd_chunked
 *     and sdm_scan_bwd check every token's slot lists on the device first (ids
 *     in [0, N) and distinct within a list, the condition Sec. 3.1 step 2's
 *     sets imply and the backward's replace step needs) and return
 *     SDM_ERR_INVALID_ARG before any output is touched.  The check uses word 1
 *     of the workspace and synchronises the stream; without it a repeated id
 *     is undefined behaviour and an id out of range is clamped and flagged.
 *   - dtype codes: SDM_F32 (IEEE fp32) or SDM_BF16 (bfloat16).  Memory
 *     tables, outputs and gradients are always fp32.
 */
#ifndef SDM_H_
#define SDM_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum sdm_dtype { SDM_F32 = 0, SDM_BF16 = 1 };

enum sdm_status {
    SDM_OK = 0,
    SDM_ERR_INVALID_ARG = -1,   /* a size, pointer or alignment rule is violated */
    SDM_ERR_UNSUPPORTED = -2,   /* legal, but outside what the kernels implement */
    SDM_ERR_WORKSPACE = -3,     /* workspace / saved buffer too small */
    SDM_ERR_HIP = -4,           /* a HIP runtime call failed (launch, attribute) */
    SDM_ERR_DEVICE_CHECK = -5   /* a device-side index check found a bad slot id */
};

/* ------------------------------------------------------------------------
 * sdm_address — product-key addressing of one side (write keys or read
 * queries).  Sec. 2 "Product Key Memory" and Sec. 3.1 step 1: the projected
 * vector is split into two halves that give two score vectors s0, s1 of
 * length sqrt(N); slot (a, b) scores s0[a] + s1[b] and has flat id
 * a*sqrt(N) + b; the top-k slots are found through
 * top_k(s0 (+) s1) = top_k(top_k(s0) (+) top_k(s1)).  The weights are the
 * softmax of the selected scores (Sec. 4 "SDM Configuration") and the
 * selected ids are returned sorted ascending (App. A.2).
 *
 *   x         [B, H, T, d_k] in x_dtype: the projected keys (write side) or
 *             queries (read side).
 *   codebook  [H, 2, sqrt(N), d_k/2] in x_dtype: per-head sub-key codebooks;
 *             s_h[j] = <x[h*d_k/2 : (h+1)*d_k/2], codebook[head][h][j]>.
 *             NULL selects direct mode, which needs d_k == 2*sqrt(N) and takes
 *             s0 = x[0:sqrt(N)], s1 = x[sqrt(N):2*sqrt(N)] as the scores.
 *   N         slots per head; must be a perfect square, sqrt(N) <= 1024.
 *   topk      slots selected per token, 1 <= topk <= min(sqrt(N), 128).
 *   idx       out [B, H, T, topk] int32: selected slot ids, ascending.
 *   val       out [B, H, T, topk] fp32: softmax weights, in idx order.
 *   score     optional out [B, H, T, topk] fp32: the raw selected scores.
 * Ranking: score descending, ties to the lower flat id.  Scores are formed
 * in fp32 (bf16 products accumulated in fp32 on the matrix cores).
 * Codebook mode needs d_k even and d_k/2 <= 256.
 * ---------------------------------------------------------------------- */
int sdm_address(const void* x, int x_dtype, const void* codebook,
                int B, int H, int T, int d_k, int64_t N, int topk,
                int32_t* idx, float* val, float* score, void* stream);

/* ------------------------------------------------------------------------
 * sdm_scan_fwd — the sparse gated delta recurrence, in place on the memory
 * table.  For every (b, h) stream and t = 0 .. T-1 (Sec. 3.1 steps 2-3):
 *   P_n = M[i_n]                  the W write rows as left by step t-1
 *   D_n = alpha_t P_n             Eq. (sdm-decay), written rows only
 *   u   = sum_n kappa_n D_n       read-back of the decayed rows (Fig. 2)
 *   e   = beta_t (v_t - u)
 *   M[i_n] = D_n + kappa_n e      Eq. (sdm-write)
 *   y_t = sum_m rho_m M[j_m]      Eq. (sdm-read) on the post-write memory
 * Slots outside the write set are left bit-for-bit unchanged.
 *
 *   w_idx, w_val  [B, H, T, W] int32 / fp32: write slots i_n, weights kappa_n.
 *   r_idx, r_val  [B, H, T, R] int32 / fp32: read slots j_m, weights rho_m.
 *                 Any weights are accepted (not only softmax outputs).  Slot
 *                 ids must lie in [0, N) and be distinct within a token; out of
 *                 range ids are clamped on the device (never dereferenced out
 *                 of bounds) and reported by sdm_check_device_errors().
 *   v             [B, H, T, d_v] in in_dtype.
 *   alpha, beta   [B, H, T] in in_dtype: forget and input gates.
 *   mem           [B, H, N, d_v] fp32, in: M_0, out: M_T.
 *   y             out [B, H, T, d_v] fp32.
 *   saved         NULL for inference.  For training, out
 *                 [B, H, T, W, d_v] fp32: the pre-write rows P of every token
 *                 (the undo log of App. A.3); saved_bytes must be at least
 *                 sdm_scan_saved_bytes().
 *   workspace     at least sdm_scan_fwd_workspace_bytes() bytes, 256-B aligned.
 * Limits: 1 <= W, R <= 128; d_v % 4 == 0; d_v <= 4096; T == 0 is a no-op.
 * ---------------------------------------------------------------------- */
int sdm_scan_fwd(const int32_t* w_idx, const float* w_val, int W,
                 const int32_t* r_idx, const float* r_val, int R,
                 const void* v, const void* alpha, const void* beta, int in_dtype,
                 float* mem, int B, int H, int T, int d_v, int64_t N,
                 float* y, float* saved, size_t saved_bytes,
                 void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * sdm_forward — the whole forward of the layer's memory (Sec. 3.1 steps 1-3):
 * sdm_address on q (read side, codebook cb_q) and on k (write side, cb_k),
 * then sdm_scan_fwd with W = R = topk, with the same results bit for bit.
 * The addressing of a chunk of `chunk` tokens overlaps the scan of the
 * previous chunk: chunk c's addressing and records run on a library-owned
 * second stream of the device (created on first use, default priority,
 * synchronised with `stream` through events), its scan on `stream`.  When the
 * call returns, all of its work is ordered before later work on `stream`.
 *   q, k          [B, H, T, d_k] in x_dtype.
 *   cb_q, cb_k    codebooks as for sdm_address (may be the same pointer or
 *                 both NULL for direct mode).
 *   r_idx, r_val  out [B, H, T, topk]: read slots and weights.
 *   w_idx, w_val  out [B, H, T, topk]: write slots and weights.
 *   v, alpha, beta, in_dtype, mem, y, saved, saved_bytes, workspace, ws_bytes:
 *                 as for sdm_scan_fwd (workspace of
 *                 sdm_scan_fwd_workspace_bytes(B, H, T, topk, topk)).
 *   chunk         tokens per pipeline stage, rounded up to a multiple of 64
 *                 and to at most 64 stages (the last stage takes what is
 *                 left).  0 picks T/4 for T >= 2048 and a single stage
 *                 otherwise.
 * One token (T = 1, the decode step) without an undo log, both codebooks
 * given or both NULL: a single launch on `stream` does the addressing of both
 * sides and the scan step, one workgroup per (b, h) stream.  Slots and
 * weights are those of sdm_address bit for bit; y and mem agree with
 * sdm_scan_fwd to the rounding of the sums over rows (taken in another
 * order); `chunk` is ignored.
 * Outputs must not alias inputs or each other.  Validation as for the three
 * calls; on a HIP launch error part of the work may already be enqueued.
 * Concurrent calls on one device share its second stream, so they serialise
 * their addressing.
 * ---------------------------------------------------------------------- */
int sdm_forward(const void* q, const void* k, int x_dtype,
                const void* cb_q, const void* cb_k, int d_k, int topk,
                const void* v, const void* alpha, const void* beta, int in_dtype,
                float* mem, int B, int H, int T, int d_v, int64_t N,
                int32_t* r_idx, float* r_val, int32_t* w_idx, float* w_val,
                float* y, float* saved, size_t saved_bytes, int chunk,
                void* workspace, size_t ws_bytes, void* stream);

size_t sdm_scan_fwd_workspace_bytes(int B, int H, int T, int W, int R);
size_t sdm_scan_saved_bytes(int B, int H, int T, int W, int d_v);

/* ------------------------------------------------------------------------
 * sdm_forward_noalloc — sdm_forward for callers that cannot allocate device
 * memory or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, results and
 * validation as sdm_forward without `chunk`, `workspace` and `ws_bytes`: the
 * per-token records and device-error words live in a fixed device array of
 * SDM_NOALLOC_SCRATCH_BYTES (64 MiB) that each GPU the library runs on holds
 * until the process ends.  Sizes whose sdm_scan_fwd_workspace_bytes(B, H, T,
 * topk, topk) exceeds it return SDM_ERR_UNSUPPORTED before any device call
 * (at W = R = 32 that is about 102,000 token-heads, e.g. 16 x 16 streams of
 * 400 tokens; any single-token step of up to 65,535 streams fits).
 *   - Every step runs on `stream`, in one stage: no second stream, no events
 *     (with the event profiler off), no hipMalloc, hipFree or other allocating
 *     call.  The first call on a device looks up the array's address there.
 *   - All calls on one GPU share its array, which keeps the last call's
 *     contents (each call rewrites what it reads).  Calls that overlap in time
 *     on one GPU race: serialise them (one stream, or events).
 * ---------------------------------------------------------------------- */
#define SDM_NOALLOC_SCRATCH_BYTES (64u << 20)
int sdm_forward_noalloc(const void* q, const void* k, int x_dtype,
                        const void* cb_q, const void* cb_k, int d_k, int topk,
                        const void* v, const void* alpha, const void* beta, int in_dtype,
                        float* mem, int B, int H, int T, int d_v, int64_t N,
                        int32_t* r_idx, float* r_val, int32_t* w_idx, float* w_val,
                        float* y, float* saved, size_t saved_bytes, void* stream);
size_t sdm_forward_noalloc_max_bytes(void);

/* ------------------------------------------------------------------------
 * sdm_scan_fwd_chunked — the recurrence of sdm_scan_fwd by the chunk-parallel
 * form of App. A.1-A.2, for inference.  Tokens are taken 64 at a time.  Within
 * a chunk starting from the table M0, with lambda_{t,i} the sum of log alpha_s
 * over the chunk's tokens s <= t that write slot i, the innovations
 * x_t = beta_t (v_t - u_t) solve the unit lower-triangular system
 * (I + diag(beta) A) x = diag(beta) (V - retrieved) with the gated sparse inner
 * products A of App. A.2 (Eq. sparse-ip); the reads are the decayed M0 rows plus
 * a triangular product QK x; each slot written in the chunk is then stored
 * once.  The first kernel (all chunks in parallel) builds per-chunk
 * coefficients from the slot lists and gates alone; the second walks the
 * chunks of each stream in order, one workgroup per 8 or 32 columns (see
 * sdm_set_chunk_scan_cols).  With 32 or more chunks both run over 8 chunk
 * ranges, the coefficients of the next range on the library's second stream
 * (as sdm_forward's) beside the scan of the current one; all work is ordered
 * before later work on `stream` when the call returns.  Results equal
 * sdm_scan_fwd's up to the rounding of the reassociated sums and of the
 * triangular solve (and may vary in the last bits between runs: see
 * sdm_set_chunk_scan_cols).
 *   Arguments as for sdm_scan_fwd, without the undo log; workspace of at least
 *   sdm_scan_fwd_chunked_workspace_bytes() bytes (256-B aligned), which holds
 *   about (8 C^2 + 4 C (W + R) + 40 C W) bytes per stream and chunk (C = 64).
 * Limits: W, R <= 64 (SDM_ERR_UNSUPPORTED beyond); forget gates must be > 0
 * (the decays are taken in log form): a gate <= 0 is treated as 1e-30 and
 * flagged for sdm_check_device_errors, as are out-of-range slot ids (clamped).
 * ---------------------------------------------------------------------- */
int sdm_scan_fwd_chunked(const int32_t* w_idx, const float* w_val, int W,
                         const int32_t* r_idx, const float* r_val, int R,
                         const void* v, const void* alpha, const void* beta, int in_dtype,
                         float* mem, int B, int H, int T, int d_v, int64_t N,
                         float* y, void* workspace, size_t ws_bytes, void* stream);
size_t sdm_scan_fwd_chunked_workspace_bytes(int B, int H, int T, int W, int R);
/* Columns per workgroup of sdm_scan_fwd_chunked's scan kernel: 8 (the narrow
 * kernel: 16 workgroups per 128-column stream, which fill the chip at few
 * streams; needs d_v % 8 == 0), 16 or 32 (a 128-byte piece of every row), or
 * 0 (the default): 8 when d_v % 8 == 0, W <= 32 and the narrow workgroups
 * (B H d_v / 8) fit the device at one per compute unit, else 32.
 * Process-wide; any other value returns SDM_ERR_INVALID_ARG and keeps the
 * setting.  The coefficient kernel adds the pair terms of its triangular
 * system with LDS atomics, so results may differ from run to run in the last
 * bits (a GPU test bounds the spread at 1e-6 relative). */
int sdm_set_chunk_scan_cols(int cols);

/* ------------------------------------------------------------------------
 * sdm_scan_bwd — reverse mode of sdm_scan_fwd plus the addressing gradient.
 * Past memory states are recovered by undoing the in-place writes from the
 * saved pre-write rows (App. A.3); per token the forward intermediates
 * (D_n, u, e) are recomputed from those rows.  Per stream, t = T-1 .. 0,
 * with G the adjoint of the memory (initialised from dmem_T):
 *   read    rbar_m = <dy_t, M_t[j_m]>;  G[j_m] += rho_m dy_t
 *   write   g_n = G[i_n]; ebar = sum_n kappa_n g_n; dv_t = beta ebar;
 *           dbeta_t = <ebar, v_t - u>; kbar_n = <g_n, e> - beta <ebar, D_n>;
 *           Dbar_n = g_n - beta kappa_n ebar; dalpha_t = sum_n <Dbar_n, P_n>;
 *           G[i_n] = alpha Dbar_n
 *   undo    M[i_n] = P_n
 * The weight gradients then pass through the softmax and the product-key
 * scores to the projected vectors (the selection itself has no gradient):
 *   sbar_n = w_n (wbar_n - sum_m w_m wbar_m); s0bar[a] += sbar_n,
 *   s1bar[b] += sbar_n; xbar_h = sum_j shbar[j] codebook[h][j]
 *   (direct mode: xbar = [s0bar, s1bar]).
 *
 *   cb_q, cb_k    codebooks of the read / write side ([H,2,sqrt(N),d_k/2]
 *                 in cb_dtype) or NULL for direct mode; may be the same pointer.
 *   w_idx .. beta, in_dtype, W, R, N, d_v: exactly as given to sdm_scan_fwd.
 *   mem           in: M_T (as left by sdm_scan_fwd), out: M_0, bit-exact.
 *   saved         the buffer filled by sdm_scan_fwd.
 *   dy            [B, H, T, d_v] fp32: gradient of y.
 *   dmem_T        optional [B, H, N, d_v] fp32 gradient of M_T (NULL = 0).
 *                 May alias dmem0.
 *   chunk         (> 0) sets the pipeline stages of the backward: with
 *                 L = max(chunk, T/4) rounded up to 64 (and at least T/63), the
 *                 first stage (the end of the sequence) and the last are a
 *                 quarter of L, the tokens between them even stages of at most
 *                 L (multiples of 64); chunk >= T runs one stage.  Each stage's scan runs
 *                 on `stream`; the records of the next stage and the weight
 *                 and addressing gradients of the previous one run meanwhile on
 *                 the library's second stream (the one sdm_forward uses, with
 *                 the same event ordering: when the call returns, all of its
 *                 work is ordered before later work on `stream`).  Results do
 *                 not depend on chunk, bit for bit.
 *   dq, dk        optional out [B, H, T, d_k] fp32 (NULL = not computed).
 *   dv            out [B, H, T, d_v] fp32.
 *   dalpha, dbeta out [B, H, T] fp32.
 *   dmem0         out [B, H, N, d_v] fp32: gradient of M_0.
 *   dw_val, dr_val optional out [B, H, T, W] / [B, H, T, R] fp32.
 *   workspace     at least sdm_scan_bwd_workspace_bytes() bytes, 256-B aligned.
 * ---------------------------------------------------------------------- */
int sdm_scan_bwd(const void* cb_q, const void* cb_k, int cb_dtype, int d_k,
                 const int32_t* w_idx, const float* w_val, int W,
                 const int32_t* r_idx, const float* r_val, int R,
                 const void* v, const void* alpha, const void* beta, int in_dtype,
                 float* mem, const float* saved, size_t saved_bytes,
                 const float* dy, const float* dmem_T, int chunk,
                 int B, int H, int T, int d_v, int64_t N,
                 float* dq, float* dk, float* dv, float* dalpha, float* dbeta,
                 float* dmem0, float* dw_val, float* dr_val,
                 void* workspace, size_t ws_bytes, void* stream);

size_t sdm_scan_bwd_workspace_bytes(int B, int H, int T, int W, int R, int d_v);

/* ------------------------------------------------------------------------
 * The steps either side of the recurrence.
 *
 * sdm_gates — the gate producers of Sec. 3.1 step 2, per head and token:
 *   alpha = exp(-A[h] softplus(a + b_dt[h]))   (forget gate)
 *   beta  = sigma(b)                           (input gate)
 * from the pre-activations a = W_a x and b = W_b x, which the caller's input
 * projection GEMM produces.  A is the learnable decay (Sec. 4 initialises it
 * in [0, 16]), b_dt the time-step bias (inverse softplus of [0.001, 0.1]).
 *   a_pre, b_pre  [B, H, T] in dtype;  A, b_dt [H] fp32;
 *   alpha, beta   out [B, H, T] fp32.
 * sdm_gates_bwd — its reverse mode: with z = a + b_dt,
 *   da = dalpha (-A alpha sigma(z)),  db = dbeta beta (1 - beta),
 *   dA[h] = sum over (b, t) of dalpha (-softplus(z) alpha),  db_dt[h] = sum of da,
 * the sums over a head's tokens taken in a fixed order (reproducible).
 *   dalpha, dbeta [B, H, T] fp32;  da, db out [B, H, T];  dA, db_dt out [H].
 * ---------------------------------------------------------------------- */
int sdm_gates(const void* a_pre, const void* b_pre, int dtype, const float* A, const float* b_dt,
              int B, int H, int T, float* alpha, float* beta, void* stream);
int sdm_gates_bwd(const void* a_pre, const void* b_pre, int dtype, const float* A, const float* b_dt,
                  const float* dalpha, const float* dbeta, int B, int H, int T,
                  float* da, float* db, float* dA, float* db_dt, void* stream);

/* ------------------------------------------------------------------------
 * sdm_norm_gate — the output epilogue of Sec. 3.1 step 4 ("Norm, Gating, and
 * Head Mixing") and Fig. 2's g (.) Norm(y): per (b, h, t) row of d_v values
 *   rstd = 1 / sqrt(mean_c y[c]^2 + eps),  o[c] = y[c] rstd gamma[c] phi(g[c]),
 * phi = identity (act = 0, the element-wise gate as the text states it) or
 * SiLU g sigma(g) (act = 1).  W_o, which mixes the heads afterwards, is a
 * plain GEMM outside this library.
 *   y      [B, H, T, d_v] fp32 (the read of Eq. sdm-read);
 *   g      [B, H, T, d_v] in g_dtype: the output gate W_g x;
 *   gamma  [d_v] fp32 norm scale shared by the heads, or NULL (ones);
 *   o      out [B, H, T, d_v] fp32;  rstd  optional out [B, H, T] fp32.
 *   d_v % 4 == 0, d_v <= 4096, eps >= 0.
 * sdm_norm_gate_bwd — its reverse mode, with n = y rstd:
 *   dg = dout gamma n phi'(g);  dn = dout phi(g) gamma;
 *   dy = rstd (dn - n mean_c(dn n));  dgamma = sum over rows of dout phi(g) n
 * (dgamma summed per workgroup, then across workgroups in a fixed order;
 * NULL skips it).  Workspace: sdm_norm_gate_bwd_workspace_bytes(), 256-B
 * aligned.
 * ---------------------------------------------------------------------- */
int sdm_norm_gate(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act,
                  int B, int H, int T, int d_v, float* o, float* rstd, void* stream);
size_t sdm_norm_gate_bwd_workspace_bytes(int B, int H, int T, int d_v);
int sdm_norm_gate_bwd(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act,
                      const float* dout, int B, int H, int T, int d_v,
                      float* dy, float* dg, float* dgamma, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * sdm_layer_fwd — the layer from its projections to the input of W_o
 * (Sec. 3.1 steps 1-4): addressing of q (top-R) and k (top-W), the gates
 * formed from their pre-activations inside the scan's per-token records (no
 * alpha / beta arrays), the recurrence, and the norm-gate epilogue of each
 * pipeline stage right after that stage's scan.  Pipelined as sdm_forward
 * (addressing of the next stage on the library's second stream).
 *   q, k, cb_q, cb_k, x_dtype, d_k, N, chunk: as for sdm_forward; W, R the
 *     write and read list lengths (may differ).
 *   v, a_pre, b_pre, g    [B, H, T, d_v] / [B, H, T] / [B, H, T] /
 *                         [B, H, T, d_v] in in_dtype.
 *   A, b_dt, gamma, eps, act: as for sdm_gates / sdm_norm_gate.
 *   mem, saved, saved_bytes: as for sdm_scan_fwd (saved holds W rows per token).
 *   r_idx, r_val [B,H,T,R], w_idx, w_val [B,H,T,W]: out, as sdm_address.
 *   y  out [B, H, T, d_v] fp32 (kept for the backward);  o  out, as sdm_norm_gate;
 *   rstd optional out.
 *   workspace  at least sdm_scan_fwd_workspace_bytes(B, H, T, W, R) bytes.
 * A single token (T = 1, no undo log, W = R) takes the one-launch step of
 * sdm_forward, then the epilogue.
 * ---------------------------------------------------------------------- */
int sdm_layer_fwd(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int d_k,
                  int W, int R, const void* v, const void* a_pre, const void* b_pre, const void* g, int in_dtype,
                  const float* A, const float* b_dt, const float* gamma, float eps, int act,
                  float* mem, int B, int H, int T, int d_v, int64_t N,
                  int32_t* r_idx, float* r_val, int32_t* w_idx, float* w_val,
                  float* y, float* o, float* rstd, float* saved, size_t saved_bytes, int chunk,
                  void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * sdm_layer_bwd — reverse mode of sdm_layer_fwd: the epilogue's backward over
 * the whole sequence (dy, dg, dgamma), then sdm_scan_bwd's path with the gates
 * formed from the pre-activations in its records (dq, dk, dv, dM0; M_T -> M_0
 * bit-exact), then the gates' backward (da, db, dA, db_dt).
 *   Inputs as given to sdm_layer_fwd (slot lists and weights as it returned
 *   them), y as it returned it, dout [B, H, T, d_v] fp32 the gradient of o,
 *   dmem_T optional (NULL = 0), chunk as for sdm_scan_bwd.
 *   dq, dk optional; dv; da, db [B,H,T]; dA, db_dt [H]; dg [B,H,T,d_v];
 *   dgamma [d_v] optional; dmem0 [B,H,N,d_v].
 *   workspace  at least sdm_layer_bwd_workspace_bytes() bytes, 256-B aligned.
 * ---------------------------------------------------------------------- */
size_t sdm_layer_bwd_workspace_bytes(int B, int H, int T, int W, int R, int d_v);
int sdm_layer_bwd(const void* cb_q, const void* cb_k, int cb_dtype, int d_k,
                  const int32_t* w_idx, const float* w_val, int W,
                  const int32_t* r_idx, const float* r_val, int R,
                  const void* v, const void* a_pre, const void* b_pre, const void* g, int in_dtype,
                  const float* A, const float* b_dt, const float* gamma, float eps, int act,
                  float* mem, const float* saved, size_t saved_bytes, const float* y, const float* dout,
                  const float* dmem_T, int chunk, int B, int H, int T, int d_v, int64_t N,
                  float* dq, float* dk, float* dv, float* da, float* db, float* dA, float* db_dt,
                  float* dg, float* dgamma, float* dmem0, void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * sdm_mem_init — initial memory per call.  The learned initial state M_0 of
 * Sec. 3.1 ("Learned Initial State") is one [H, N, d_v] parameter shared by
 * all sequences; every sequence starts from its own copy:
 *   dst[b, h] = m0[h] for every b   (m0 != NULL)
 *   dst = 0                         (m0 == NULL)
 *   dst  out [B, H, N, d_v] fp32;  m0  [H, N, d_v] fp32 or NULL.
 * d_v % 4 == 0, B*H <= 65535, pointers 16-B aligned.
 * ---------------------------------------------------------------------- */
int sdm_mem_init(float* dst, const float* m0, int B, int H, int64_t N, int d_v, void* stream);

/* ------------------------------------------------------------------------
 * Scan geometry.  Every column of the state is an independent recurrence
 * (Eq. 3-5 mix rows only within a column), so the scans give each wave a slice
 * of columns of one (b, h) stream.  sdm_set_scan_slice_width(sw):
 *   0   automatic (default): 8 columns per wave, unless B*H*ceil(d_v/8)
 *       waves would put 1.5 or more on every SIMD of the device: then 16 (half
 *       as many waves); 8 as well where 16 columns cannot hold W or R (> 64),
 *       and for the forward's line-cooperative kernel at W = R = 64 (whose
 *       16-column form holds most of a CU's LDS);
 *   8, 16  force that width.
 * Process-wide; applies to launches that start after the call.  Results of
 * the two widths agree to the rounding of the sums over rows.  Any other
 * value returns SDM_ERR_INVALID_ARG and keeps the setting.
 * ---------------------------------------------------------------------- */
int sdm_set_scan_slice_width(int sw);

/* ------------------------------------------------------------------------
 * Scan prefetch depth: tokens whose table rows are in flight while one is
 * computed (the prep kernels link rows written within that window to LDS
 * rings).  sdm_set_scan_prefetch(pd):
 *   0   automatic (default): 4, except 16 (8 where LDS does not allow 16) for
 *       the line-cooperative forward kernel when its launch has fewer waves
 *       than the device has SIMDs (few streams: each stream's step time is
 *       then set by the row loads' latency over the tokens in flight);
 *   4, 8, 16  force that depth for the line-cooperative forward kernel (the
 *       per-wave kernels always take 4, or 2 for four-pass backward shapes);
 *       8 and 16 also give the line-cooperative backward kernel at 32 rows a
 *       depth of 8 (its default, and its depth at 64 rows, is 4).
 * Results do not depend on it.  Process-wide; applies to launches that start
 * after the call.  Any other value returns SDM_ERR_INVALID_ARG.
 * ---------------------------------------------------------------------- */
int sdm_set_scan_prefetch(int pd);

/* ------------------------------------------------------------------------
 * Table I/O of the scans.  By default each scan runs a four-wave
 * line-cooperative kernel where the shape allows it: the waves of four
 * adjacent column slices (4 x 8 or 4 x 16 columns: one or two 128-byte lines
 * of every table row) move table rows between HBM and LDS as whole lines and
 * exchange their pieces in LDS.  Forward: W = R = 32 or 64 and d_v a
 * multiple of 4 times the slice width; backward: 8-column slices, W = R = 32
 * (where the per-wave plan takes 8-column slices) or 64, and d_v a multiple of
 * 32.  Each stream's table and saved rows must stay below 2 GiB (32-bit
 * offsets), else the per-wave kernels run.  sdm_set_scan_line_io(0) always
 * uses the per-wave kernels
 * (each wave moves its own pieces of the rows), 1 restores the default.  The
 * two do the same arithmetic per slice; results agree to rounding (the sums
 * over rows are taken in a different order, and the compiler may fuse a
 * product into an fma in one and not the other).  Process-wide; applies to
 * launches that start after the call.  Any other value returns
 * SDM_ERR_INVALID_ARG and keeps the setting.
 * ---------------------------------------------------------------------- */
int sdm_set_scan_line_io(int on);

/* ------------------------------------------------------------------------
 * Per-kernel timing with HIP events, off by default.  While enabled, every
 * kernel the library launches is bracketed by two HIP events recorded on the
 * stream it is launched on; sdm_profile_read() waits for the recorded events
 * and returns the summed elapsed time and launch count of one kernel kind
 * since the last sdm_profile_enable(1).  Events come from a pool that is
 * grown on first use and reused afterwards.  Not meant for concurrent use
 * from several host threads.
 * ---------------------------------------------------------------------- */
enum sdm_kernel {
    SDM_K_ADDRESS = 0, SDM_K_FWD_PREP = 1, SDM_K_FWD_SCAN = 2, SDM_K_BWD_PREP = 3,
    SDM_K_BWD_SCAN = 4, SDM_K_BWD_REDUCE = 5, SDM_K_ADDRESS_BWD = 6, SDM_K_MEM_INIT = 7,
    SDM_K_DECODE = 8, SDM_K_CHUNK_COEF = 9, SDM_K_CHUNK_SCAN = 10, SDM_K_NORM_GATE = 11, SDM_K_GATES = 12,
    SDM_K_COUNT = 13
};
int sdm_profile_enable(int on);
/* Which kernel kinds the events bracket while profiling is enabled: bit k for
 * enum sdm_kernel k (all by default).  Fewer events disturb a pipelined call
 * less.  Bits past SDM_K_COUNT return SDM_ERR_INVALID_ARG. */
int sdm_profile_select(unsigned int mask);
int sdm_profile_read(int kernel, double* total_ms, int64_t* launches);

/* ------------------------------------------------------------------------
 * Diagnostics.
 *   sdm_check_device_errors  synchronises `stream`, then reports whether
 *       any scan since the last check clamped an out-of-range slot id, or
 *       the chunked scan met a forget gate <= 0 (SDM_ERR_DEVICE_CHECK), and
 *       clears the flag held in `workspace`.
 *   sdm_status_string        static text for a status code.
 *   sdm_last_error           thread-local text of the last failure.
 *   sdm_version              library version string.
 * ---------------------------------------------------------------------- */
int sdm_check_device_errors(void* workspace, void* stream);
const char* sdm_status_string(int status);
const char* sdm_last_error(void);
const char* sdm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SDM_H_ */
