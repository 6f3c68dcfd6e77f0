// Host-side launchers shared between the kernel files and the C ABI layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#define SDM_DT_F32 0
#define SDM_DT_BF16 1

// Prefetch depth (tokens in flight per wave) of the forward and backward scans;
// the prep kernels compute read-after-write links for exactly this window.
#define SDM_FWD_PD 4
#define SDM_BWD_PD 4
// Deeper forward window for launches with fewer waves than SIMDs (latency-bound).
#define SDM_FWD_PD_DEEP 16

// Per-token record of the forward scan (written by the prep kernel, staged in
// LDS by the scan): slots and weights of both sides (a read row whose slot the
// token writes weighted rho alpha), forwarding links, gates and yc, the sum of
// rho kappa over those rows.
struct FwdRec {
    int W, R;
    int off_wval, off_rslot, off_rval, off_link, off_ab, bytes;
};

__host__ __device__ inline FwdRec fwd_rec_layout(int W, int R) {
    FwdRec r;
    r.W = W;
    r.R = R;
    r.off_wval = 4 * W;
    r.off_rslot = 8 * W;
    r.off_rval = 8 * W + 4 * R;
    r.off_link = 8 * W + 8 * R;
    r.off_ab = (r.off_link + 2 * (W + R) + 3) & ~3;   // alpha, beta, yc
    r.bytes = (r.off_ab + 12 + 15) & ~15;
    return r;
}

// Backward record: slots/weights as forward, plus links for the rows the
// reverse step reads (M[j_m], G[j_m], G[i_n]).
struct BwdRec {
    int W, R;
    int off_wval, off_rslot, off_rval, off_lm, off_lgr, off_lgw, off_ab, bytes;
};

__host__ __device__ inline BwdRec bwd_rec_layout(int W, int R) {
    BwdRec r;
    r.W = W;
    r.R = R;
    r.off_wval = 4 * W;
    r.off_rslot = 8 * W;
    r.off_rval = 8 * W + 4 * R;
    r.off_lm = 8 * W + 8 * R;          // int16 [R]: source of M_t[j_m]
    r.off_lgr = r.off_lm + 2 * R;      // int16 [R]: source of G[j_m]
    r.off_lgw = r.off_lgr + 2 * R;     // int16 [W]: source of G[i_n]
    r.off_ab = (r.off_lgw + 2 * W + 3) & ~3;
    r.bytes = (r.off_ab + 8 + 15) & ~15;
    return r;
}

// Workspace header: device-side error flag(s) at offset 0.
#define SDM_WS_HEADER 256

// Tokens [tb, tb + tn) of every stream (layout strides use T).
// lds_free > 0: the launch shares every CU with work that holds the rest of its
// LDS (the pipelined forward's scan), and keeps to the workgroups that fit
// beside it (when two or more do), each looping over tiles (0: one workgroup
// per tile).
hipError_t sdm_launch_address(const void* x, int x_dtype, const void* cb, int B, int H, int T,
                              int tb, int tn, int dk, int s, int k, int32_t* idx, float* val,
                              float* score, hipStream_t st, size_t lds_free = 0);
// token-sides (b, h, t) for t in [tb, tb + tn)
// One token per stream (T = 1, no undo log): addressing of both sides and the
// scan step in one launch, one workgroup per stream.  cb_q and cb_k are both
// codebooks or both NULL (direct mode).
hipError_t sdm_launch_decode(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int B,
                             int H, int dk, int s, int topk, const void* v, const void* alpha, const void* beta,
                             int in_dtype, float* mem, int64_t N, int dv, int32_t* r_idx, float* r_val,
                             int32_t* w_idx, float* w_val, float* y, unsigned int* flags, hipStream_t st,
                             const float* gate_A = nullptr, const float* gate_bdt = nullptr);
hipError_t sdm_launch_address_bwd(const void* cb, int cb_dtype, int B, int H, int T, int tb, int tn, int dk,
                                  int s, int k, const int32_t* idx, const float* val, const float* dval,
                                  float* dx, hipStream_t st);

struct ScanFwdArgs {
    const int32_t* w_idx;
    const float* w_val;
    const int32_t* r_idx;
    const float* r_val;
    const void* v;
    const void* alpha;
    const void* beta;
    int in_dtype;
    float* mem;
    int B, H, T, dv, W, R;
    int64_t N;
    float* y;
    float* saved;
    unsigned char* ws;   // workspace base (header + records)
    int tb = 0, te = 0;  // tokens processed: [tb, te) (layout strides use T); tb a multiple of 16
    // Gate producers fused into the records: with gate_A set, alpha and beta hold the
    // gates' pre-activations and alpha = exp(-A softplus(a + b_dt)), beta = sigma(b)
    // are formed per token (A, b_dt per head, fp32).
    const float* gate_A = nullptr;
    const float* gate_bdt = nullptr;
};
hipError_t sdm_launch_scan_fwd(const ScanFwdArgs& a, hipStream_t st);   // prep + scan
size_t sdm_fwd_scan_lds(const ScanFwdArgs& a);   // LDS of one workgroup of that scan
// the two halves separately (records of [tb, te), then the scan of [tb, te))
hipError_t sdm_launch_fwd_prep_range(const ScanFwdArgs& a, hipStream_t st);
hipError_t sdm_launch_fwd_scan_range(const ScanFwdArgs& a, hipStream_t st);
// SIMDs (4 per compute unit) of the current device; 1024 if it cannot be queried.
int sdm_device_simds();
// Forced scan slice width (8 or 16), or 0 for the automatic choice.
int sdm_scan_slice_width();
// Forced forward prefetch depth (4, 8 or 16), or 0 for the automatic choice.
int sdm_scan_prefetch();
// Prefetch depth (tokens in flight) of the forward scan for these arguments;
// the prep kernel links over the same window.
int sdm_fwd_pd(const ScanFwdArgs& a);
// Whether the scans may use their line-cooperative kernels (default: yes).
bool sdm_line_io_enabled();
// true if the forward scan has a launch plan for this shape (registers, LDS)
bool sdm_fwd_plan_ok(int W, int R, int dv, int in_dtype);
size_t sdm_fwd_ws_bytes(int B, int H, int T, int W, int R);

template <int PD>
hipError_t sdm_launch_fwd_prep(const ScanFwdArgs& a, hipStream_t st);

// Chunk-parallel forward scan: tokens in chunks of SDM_CHUNK, W and R at most
// SDM_CHUNK_MAX_LIST.  The coefficient kernel writes one record per (stream,
// chunk) after the workspace header; the scan kernel reads them (a.saved unused).
// Both take the chunks of tokens [a.tb, a.te) (tb a multiple of SDM_CHUNK).
#define SDM_CHUNK 64
#define SDM_CHUNK_MAX_LIST 64
bool sdm_chunk_shape_ok(int W, int R);
// Forced columns per workgroup of the chunked scan (16 or 32), or 0 for automatic.
int sdm_chunk_cols();
size_t sdm_chunk_ws_bytes(int B, int H, int T, int W, int R);
hipError_t sdm_launch_chunk_coef(const ScanFwdArgs& a, hipStream_t st);
hipError_t sdm_launch_chunk_scan(const ScanFwdArgs& a, hipStream_t st);

struct ScanBwdArgs {
    const int32_t* w_idx;
    const float* w_val;
    const int32_t* r_idx;
    const float* r_val;
    const void* v;
    const void* alpha;
    const void* beta;
    int in_dtype;
    float* mem;
    const float* saved;
    const float* dy;
    int chunk;
    int B, H, T, dv, W, R;
    int64_t N;
    float* dv_out;
    float* dalpha;
    float* dbeta;
    float* G;         // dmem0 buffer, holds dM_T on entry
    float* dw_val;    // [B,H,T,W] (workspace if the caller passed NULL)
    float* dr_val;    // [B,H,T,R]
    unsigned char* ws;
    int tb = 0, te = 0;  // tokens processed, te-1 down to tb (layout strides use T)
    int line = -1;       // line-cooperative kernel: 1 / 0, or -1 to decide from the shape
    const float* gate_A = nullptr;     // as in ScanFwdArgs: alpha, beta are pre-activations
    const float* gate_bdt = nullptr;
};
// Backward of tokens a.te-1 down to a.tb, in three steps: records (with links
// inside the range), the scan, the sum of the partial scalars.  Ranges are run
// from the end of the sequence down; tables carry the state between them.
hipError_t sdm_launch_bwd_prep_range(const ScanBwdArgs& a, hipStream_t st);
hipError_t sdm_launch_bwd_scan_range(const ScanBwdArgs& a, hipStream_t st);
hipError_t sdm_launch_bwd_reduce_range(const ScanBwdArgs& a, hipStream_t st);
// whether the backward of this shape runs the line-cooperative kernel now
bool sdm_bwd_line_io(const ScanBwdArgs& a);
template <int PD>
hipError_t sdm_launch_bwd_prep(const ScanBwdArgs& a, hipStream_t st);
bool sdm_bwd_plan_ok(int W, int R, int dv, int in_dtype);
size_t sdm_bwd_ws_bytes(int B, int H, int T, int W, int R, int dv);

// Gate producers (Sec. 3.1 step 2) and their reverse mode; dA, db_dt are per-head sums.
hipError_t sdm_launch_gates(const void* a, const void* b, int dtype, const float* A, const float* bdt, int B, int H,
                            int T, float* alpha, float* beta, hipStream_t st);
hipError_t sdm_launch_gates_bwd(const void* a, const void* b, int dtype, const float* A, const float* bdt,
                                const float* dalpha, const float* dbeta, int B, int H, int T, float* da, float* db,
                                float* dA, float* db_dt, hipStream_t st);
// Output epilogue (Sec. 3.1 step 4) on tokens [tb, tb + tn) of S streams of T tokens.
hipError_t sdm_launch_norm_gate(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act,
                                int64_t S, int T, int tb, int tn, int dv, float* o, float* rstd, hipStream_t st);
// Its reverse mode on `rows` contiguous rows; `part` holds sdm_norm_gate_bwd_ws() bytes
// of per-workgroup dgamma sums.
size_t sdm_norm_gate_bwd_ws(int64_t rows, int dv);
hipError_t sdm_launch_norm_gate_bwd(const float* y, const void* g, int g_dtype, const float* gamma, float eps,
                                    int act, const float* dout, int64_t rows, int dv, float* dy, float* dg,
                                    float* dgamma, float* part, hipStream_t st);

// Debug check of slot lists (range and distinctness within each token's list):
// ORs bit 0 (out of range) and bit 1 (repeated id) into *flag.
hipError_t sdm_launch_check_ids(const int32_t* w_idx, int W, const int32_t* r_idx, int R, int64_t ntok,
                                int64_t N, unsigned int* flag, hipStream_t st);

hipError_t sdm_launch_mem_init(float* dst, const float* m0, int B, int H, int64_t N, int dv,
                               hipStream_t st);
hipError_t sdm_launch_copy(float* dst, const float* src, size_t n, hipStream_t st);
hipError_t sdm_launch_zero_words(void* p, int n, hipStream_t st);

// Optional steps either side of the forward scan: the gates formed from their
// pre-activations (gate_A set: alpha and beta hold a = W_a x, b = W_b x) and the
// norm-gate epilogue o = norm(y) gamma phi(g) after each stage's scan (o set).
struct SdmFwdExtras {
    const float* gate_A = nullptr;
    const float* gate_bdt = nullptr;
    const void* g = nullptr;      // [B, H, T, d_v] in the input dtype
    const float* gamma = nullptr; // [d_v] or NULL (ones)
    float eps = 0.f;
    int act = 0;                  // 0 identity, 1 SiLU
    float* o = nullptr;           // [B, H, T, d_v] fp32
    float* rstd = nullptr;        // [B, H, T] fp32 or NULL
};
// The body of sdm_forward, with separate write and read list lengths.
// pipelined = false runs every step on `stream` in one stage (no second
// stream, no events): the path of the allocation-free entry point.
int sdm_forward_impl(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int d_k,
                     int W, int R, const void* v, const void* alpha, const void* beta, int in_dtype, float* mem,
                     int B, int H, int T, int d_v, int64_t N, int32_t* r_idx, float* r_val, int32_t* w_idx,
                     float* w_val, float* y, float* saved, size_t saved_bytes, int chunk, void* workspace,
                     size_t ws_bytes, void* stream, bool pipelined, const SdmFwdExtras* ex);
// Sets the thread's sdm_last_error() text and returns status.
int sdm_set_error(int status, const char* msg);

// Event bracketing of kernel launches (active only while profiling is enabled).
void sdm_prof_begin(int kernel, hipStream_t st);
void sdm_prof_end(int kernel, hipStream_t st);
struct SdmProfScope {
    int k;
    hipStream_t st;
    SdmProfScope(int kk, hipStream_t s) : k(kk), st(s) { sdm_prof_begin(k, st); }
    ~SdmProfScope() { sdm_prof_end(k, st); }
};
