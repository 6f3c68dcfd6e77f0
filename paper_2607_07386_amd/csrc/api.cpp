// C ABI of the SDM hot path: host-side validation, workspace sizing and
// launch on the caller's stream.  Declarations and contracts: include/sdm.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

#include "sdm.h"
#include "sdm_internal.h"

namespace {
std::atomic<int> g_slice_width{0};
std::atomic<int> g_line_io{1};
std::atomic<int> g_prefetch{0};
}

int sdm_scan_slice_width() { return g_slice_width.load(std::memory_order_relaxed); }
int sdm_scan_prefetch() { return g_prefetch.load(std::memory_order_relaxed); }
std::atomic<int> g_chunk_cols{0};
int sdm_chunk_cols() { return g_chunk_cols.load(std::memory_order_relaxed); }
bool sdm_line_io_enabled() { return g_line_io.load(std::memory_order_relaxed) != 0; }

int sdm_device_simds() {
    constexpr int MAXDEV = 64;
    static int cache[MAXDEV] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAXDEV) return 1024;
    if (cache[dev] == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
        cache[dev] = 4 * cus;
    }
    return cache[dev];
}

namespace {

thread_local char g_err[512] = "";

int fail(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char* where) {
    return fail(SDM_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int isqrt64(int64_t n) {
    if (n <= 0) return -1;
    int64_t s = (int64_t)std::llround(std::sqrt((double)n));
    while (s * s > n) --s;
    while ((s + 1) * (s + 1) <= n) ++s;
    return s * s == n ? (int)s : -1;
}

bool valid_dtype(int d) { return d == SDM_F32 || d == SDM_BF16; }

constexpr int kMaxStreams = 65535;

int check_scan_common(const int32_t* w_idx, const float* w_val, int W, const int32_t* r_idx,
                      const float* r_val, int R, const void* v, const void* alpha,
                      const void* beta, int in_dtype, const float* mem, int B, int H, int T,
                      int d_v, int64_t N) {
    if (B < 0 || H < 0 || T < 0) return fail(SDM_ERR_INVALID_ARG, "B, H, T must be >= 0");
    if ((int64_t)B * H > kMaxStreams) return fail(SDM_ERR_UNSUPPORTED, "B*H must be <= %d", kMaxStreams);
    if (W < 1 || R < 1) return fail(SDM_ERR_INVALID_ARG, "W and R must be >= 1");
    if (W > 128 || R > 128) return fail(SDM_ERR_UNSUPPORTED, "W and R must be <= 128");
    if (d_v < 4 || d_v % 4 != 0) return fail(SDM_ERR_INVALID_ARG, "d_v must be a positive multiple of 4");
    if (d_v > 4096) return fail(SDM_ERR_UNSUPPORTED, "d_v must be <= 4096");
    if (N < 1 || N > (int64_t)1 << 31) return fail(SDM_ERR_INVALID_ARG, "N must be in [1, 2^31]");
    if (!valid_dtype(in_dtype)) return fail(SDM_ERR_INVALID_ARG, "in_dtype must be SDM_F32 or SDM_BF16");
    // arrays of zero size may come as NULL (empty tensors have no storage)
    const bool tok = (int64_t)B * H * T > 0;
    if ((tok && (!w_idx || !w_val || !r_idx || !r_val || !v || !alpha || !beta)) ||
        ((int64_t)B * H > 0 && !mem))
        return fail(SDM_ERR_INVALID_ARG, "null input pointer");
    if (!aligned(w_idx, 16) || !aligned(w_val, 16) || !aligned(r_idx, 16) || !aligned(r_val, 16) ||
        !aligned(v, 16) || !aligned(alpha, 4) || !aligned(beta, 4) || !aligned(mem, 16))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer (16-byte alignment required)");
    return SDM_OK;
}

// SDM_DEBUG=1 in the environment: the scans first check every token's slot
// lists on the device (ids in [0, N), distinct within a list) and return
// SDM_ERR_INVALID_ARG before touching any output.  The check synchronises the
// stream and uses word 1 of the workspace header.
bool debug_checks() {
    const char* e = std::getenv("SDM_DEBUG");
    return e && e[0] == '1' && e[1] == 0;
}

int debug_check_ids(const int32_t* w_idx, int W, const int32_t* r_idx, int R, int64_t ntok, int64_t N,
                    void* workspace, hipStream_t st) {
    unsigned int* flag = static_cast<unsigned int*>(workspace) + 1;
    hipError_t e = sdm_launch_zero_words(workspace, 4, st);
    if (e == hipSuccess) e = sdm_launch_check_ids(w_idx, W, r_idx, R, ntok, N, flag, st);
    unsigned int h = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&h, flag, sizeof(h), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "SDM_DEBUG slot-list check");
    if (h & 2u) return fail(SDM_ERR_INVALID_ARG, "SDM_DEBUG: a token's slot list repeats an id");
    if (h & 1u) return fail(SDM_ERR_INVALID_ARG, "SDM_DEBUG: a slot id lies outside [0, N)");
    return SDM_OK;
}

// ---- event profiler ----
struct ProfState {
    std::mutex mu;
    bool on = false;
    unsigned int mask = (1u << SDM_K_COUNT) - 1;   // kernel kinds timed while on
    std::vector<hipEvent_t> pool;                 // free events
    std::vector<std::pair<hipEvent_t, hipEvent_t>> done[SDM_K_COUNT];
    hipEvent_t open_ev[SDM_K_COUNT] = {};
};
ProfState& prof() {
    static ProfState p;
    return p;
}
hipEvent_t take_event(ProfState& p) {
    if (!p.pool.empty()) {
        hipEvent_t e = p.pool.back();
        p.pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

void sdm_prof_begin(int k, hipStream_t st) {
    ProfState& p = prof();
    if (!p.on || !(p.mask >> k & 1u)) return;
    std::lock_guard<std::mutex> g(p.mu);
    hipEvent_t e = take_event(p);
    if (e && hipEventRecord(e, st) == hipSuccess) p.open_ev[k] = e;
}

void sdm_prof_end(int k, hipStream_t st) {
    ProfState& p = prof();
    if (!p.on || !(p.mask >> k & 1u)) return;
    std::lock_guard<std::mutex> g(p.mu);
    hipEvent_t b = p.open_ev[k];
    p.open_ev[k] = nullptr;
    if (!b) return;
    hipEvent_t e = take_event(p);
    if (e && hipEventRecord(e, st) == hipSuccess) p.done[k].push_back({b, e});
}

namespace {

// Validation shared by sdm_address and sdm_forward; *s_out = sqrt(N).
int check_address(const void* x, int x_dtype, const void* codebook, int B, int H, int T, int d_k,
                  int64_t N, int topk, const int32_t* idx, const float* val, const float* score,
                  int* s_out) {
    if (B < 0 || H < 0 || T < 0) return fail(SDM_ERR_INVALID_ARG, "B, H, T must be >= 0");
    if ((int64_t)B * H > kMaxStreams) return fail(SDM_ERR_UNSUPPORTED, "B*H must be <= %d", kMaxStreams);
    if (!valid_dtype(x_dtype)) return fail(SDM_ERR_INVALID_ARG, "x_dtype must be SDM_F32 or SDM_BF16");
    const int s = isqrt64(N);
    if (s < 0) return fail(SDM_ERR_INVALID_ARG, "N=%lld is not a perfect square", (long long)N);
    if (s > 1024) return fail(SDM_ERR_UNSUPPORTED, "sqrt(N) must be <= 1024");
    if (topk < 1 || topk > s) return fail(SDM_ERR_INVALID_ARG, "topk must be in [1, sqrt(N)]");
    if (topk > 128) return fail(SDM_ERR_UNSUPPORTED, "topk must be <= 128");
    if (d_k < 1) return fail(SDM_ERR_INVALID_ARG, "d_k must be >= 1");
    if (codebook) {
        if (d_k % 2) return fail(SDM_ERR_INVALID_ARG, "codebook mode needs an even d_k");
        if (d_k / 2 > 256) return fail(SDM_ERR_UNSUPPORTED, "codebook mode needs d_k/2 <= 256");
        if (!aligned(codebook, 16)) return fail(SDM_ERR_INVALID_ARG, "misaligned codebook");
    } else if (d_k != 2 * s) {
        return fail(SDM_ERR_INVALID_ARG, "direct mode needs d_k == 2*sqrt(N)");
    }
    *s_out = s;
    if ((int64_t)B * H * T == 0) return SDM_OK;   // nothing is read or written
    if (!x || !idx || !val) return fail(SDM_ERR_INVALID_ARG, "null pointer");
    if (!aligned(x, 16) || !aligned(idx, 4) || !aligned(val, 4) || (score && !aligned(score, 4)))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer");
    return SDM_OK;
}

// Outputs, plan and workspace of a forward scan (after check_scan_common, T > 0).
int check_scan_fwd_rest(int W, int R, int in_dtype, int B, int H, int T, int d_v, const float* y,
                        const float* saved, size_t saved_bytes, const void* workspace, size_t ws_bytes) {
    if (!y || !aligned(y, 16)) return fail(SDM_ERR_INVALID_ARG, "y must be a 16-byte aligned pointer");
    if (saved) {
        if (!aligned(saved, 16)) return fail(SDM_ERR_INVALID_ARG, "misaligned saved buffer");
        if (saved_bytes < sdm_scan_saved_bytes(B, H, T, W, d_v))
            return fail(SDM_ERR_WORKSPACE, "saved buffer too small: %zu < %zu", saved_bytes,
                        sdm_scan_saved_bytes(B, H, T, W, d_v));
    }
    if (!sdm_fwd_plan_ok(W, R, d_v, in_dtype))
        return fail(SDM_ERR_UNSUPPORTED, "no forward launch plan for W=%d R=%d d_v=%d", W, R, d_v);
    const size_t need = sdm_fwd_ws_bytes(B, H, T, W, R);
    if (!workspace || !aligned(workspace, 256))
        return fail(SDM_ERR_INVALID_ARG, "workspace must be a 256-byte aligned pointer");
    if (ws_bytes < need) return fail(SDM_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);
    return SDM_OK;
}

}  // namespace

// ---- state of the fused forward's pipeline ----
namespace {
constexpr int kMaxChunks = 64;
constexpr size_t kCuLds = 160 * 1024;   // LDS per CU (gfx950)
constexpr int kMaxDevices = 64;
struct SidePipe {
    std::mutex mu;
    hipStream_t side[kMaxDevices] = {};
    std::vector<hipEvent_t> ev[kMaxDevices];
};
SidePipe& side_pipe() {
    static SidePipe p;
    return p;
}
// The current device's second stream (created on first use, default priority)
// and at least nev events; the caller holds sp.mu while it enqueues.
hipError_t side_get(SidePipe& sp, int nev, hipStream_t* side, std::vector<hipEvent_t>** ev, int* dev_out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    if (!sp.side[dev]) {
        if ((e = hipStreamCreateWithFlags(&sp.side[dev], hipStreamNonBlocking)) != hipSuccess) {
            sp.side[dev] = nullptr;
            return e;
        }
    }
    std::vector<hipEvent_t>& v = sp.ev[dev];
    while ((int)v.size() < nev) {
        hipEvent_t x;
        if ((e = hipEventCreateWithFlags(&x, hipEventDisableTiming)) != hipSuccess) return e;
        v.push_back(x);
    }
    *side = sp.side[dev];
    *ev = &v;
    *dev_out = dev;
    return hipSuccess;
}
int round_up(int x, int m) { return (x + m - 1) / m * m; }
}  // namespace

extern "C" {

int sdm_set_scan_slice_width(int sw) {
    g_err[0] = 0;
    if (sw != 0 && sw != 8 && sw != 16)
        return fail(SDM_ERR_INVALID_ARG, "sdm_set_scan_slice_width: width must be 0 (automatic), 8 or 16, got %d", sw);
    g_slice_width.store(sw, std::memory_order_relaxed);
    return SDM_OK;
}

int sdm_set_scan_prefetch(int pd) {
    g_err[0] = 0;
    if (pd != 0 && pd != 4 && pd != 8 && pd != 16)
        return fail(SDM_ERR_INVALID_ARG, "sdm_set_scan_prefetch: depth must be 0 (automatic), 4, 8 or 16, got %d", pd);
    g_prefetch.store(pd, std::memory_order_relaxed);
    return SDM_OK;
}

int sdm_set_chunk_scan_cols(int cols) {
    g_err[0] = 0;
    if (cols != 0 && cols != 8 && cols != 16 && cols != 32)
        return fail(SDM_ERR_INVALID_ARG, "sdm_set_chunk_scan_cols: expected 0 (automatic), 8, 16 or 32, got %d", cols);
    g_chunk_cols.store(cols, std::memory_order_relaxed);
    return SDM_OK;
}

int sdm_set_scan_line_io(int on) {
    g_err[0] = 0;
    if (on != 0 && on != 1)
        return fail(SDM_ERR_INVALID_ARG, "sdm_set_scan_line_io: expected 0 or 1, got %d", on);
    g_line_io.store(on, std::memory_order_relaxed);
    return SDM_OK;
}

int sdm_profile_enable(int on) {
    ProfState& p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    for (int k = 0; k < SDM_K_COUNT; ++k) {
        for (auto& pr : p.done[k]) {
            (void)hipEventSynchronize(pr.second);
            p.pool.push_back(pr.first);
            p.pool.push_back(pr.second);
        }
        p.done[k].clear();
    }
    p.on = on != 0;
    return SDM_OK;
}

int sdm_profile_select(unsigned int mask) {
    g_err[0] = 0;
    if (mask >> SDM_K_COUNT) return fail(SDM_ERR_INVALID_ARG, "sdm_profile_select: unknown kernel kinds in 0x%x", mask);
    ProfState& p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    p.mask = mask;
    return SDM_OK;
}

int sdm_profile_read(int kernel, double* total_ms, int64_t* launches) {
    g_err[0] = 0;
    if (kernel < 0 || kernel >= SDM_K_COUNT || !total_ms || !launches)
        return fail(SDM_ERR_INVALID_ARG, "bad kernel id or null output");
    ProfState& p = prof();
    std::lock_guard<std::mutex> g(p.mu);
    double tot = 0.0;
    for (auto& pr : p.done[kernel]) {
        hipError_t e = hipEventSynchronize(pr.second);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, pr.first, pr.second);
        if (e != hipSuccess) return hip_fail(e, "sdm_profile_read");
        tot += ms;
    }
    *total_ms = tot;
    *launches = (int64_t)p.done[kernel].size();
    return SDM_OK;
}


const char* sdm_version(void) { return "sdm-mi355x 0.1 (gfx950)"; }

const char* sdm_last_error(void) { return g_err; }

const char* sdm_status_string(int status) {
    switch (status) {
        case SDM_OK: return "ok";
        case SDM_ERR_INVALID_ARG: return "invalid argument";
        case SDM_ERR_UNSUPPORTED: return "unsupported configuration";
        case SDM_ERR_WORKSPACE: return "workspace or saved buffer too small";
        case SDM_ERR_HIP: return "HIP runtime error";
        case SDM_ERR_DEVICE_CHECK: return "device-side index check failed";
        default: return "unknown status";
    }
}


int sdm_address(const void* x, int x_dtype, const void* codebook, int B, int H, int T, int d_k,
                int64_t N, int topk, int32_t* idx, float* val, float* score, void* stream) {
    g_err[0] = 0;
    int s = 0;
    const int rc = check_address(x, x_dtype, codebook, B, H, T, d_k, N, topk, idx, val, score, &s);
    if (rc != SDM_OK || (int64_t)B * H * T == 0) return rc;
    hipError_t e;
    {
        SdmProfScope ps(SDM_K_ADDRESS, (hipStream_t)stream);
        e = sdm_launch_address(x, x_dtype, codebook, B, H, T, 0, T, d_k, s, topk, idx, val, score,
                               (hipStream_t)stream);
    }
    if (e != hipSuccess) return hip_fail(e, "sdm_address launch");
    return SDM_OK;
}

size_t sdm_scan_fwd_workspace_bytes(int B, int H, int T, int W, int R) {
    if (B < 0 || H < 0 || T < 0 || W < 1 || R < 1) return 0;
    return sdm_fwd_ws_bytes(B, H, T, W, R);
}

size_t sdm_scan_saved_bytes(int B, int H, int T, int W, int d_v) {
    if (B < 0 || H < 0 || T < 0 || W < 0 || d_v < 0) return 0;
    return (size_t)B * H * T * W * d_v * sizeof(float);
}

size_t sdm_scan_bwd_workspace_bytes(int B, int H, int T, int W, int R, int d_v) {
    if (B < 0 || H < 0 || T < 0 || W < 1 || R < 1 || d_v < 1) return 0;
    return sdm_bwd_ws_bytes(B, H, T, W, R, d_v);
}

int sdm_scan_fwd(const int32_t* w_idx, const float* w_val, int W, const int32_t* r_idx,
                 const float* r_val, int R, const void* v, const void* alpha, const void* beta,
                 int in_dtype, float* mem, int B, int H, int T, int d_v, int64_t N, float* y,
                 float* saved, size_t saved_bytes, void* workspace, size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    int rc = check_scan_common(w_idx, w_val, W, r_idx, r_val, R, v, alpha, beta, in_dtype, mem, B,
                               H, T, d_v, N);
    if (rc != SDM_OK) return rc;
    if ((int64_t)B * H * T == 0) return SDM_OK;   // nothing is read or written
    rc = check_scan_fwd_rest(W, R, in_dtype, B, H, T, d_v, y, saved, saved_bytes, workspace, ws_bytes);
    if (rc != SDM_OK) return rc;
    hipStream_t st = (hipStream_t)stream;
    if (debug_checks() &&
        (rc = debug_check_ids(w_idx, W, r_idx, R, (int64_t)B * H * T, N, workspace, st)) != SDM_OK)
        return rc;
    hipError_t e = sdm_launch_zero_words(workspace, 4, st);
    if (e != hipSuccess) return hip_fail(e, "sdm_scan_fwd flag reset");
    ScanFwdArgs a;
    a.w_idx = w_idx; a.w_val = w_val; a.r_idx = r_idx; a.r_val = r_val;
    a.v = v; a.alpha = alpha; a.beta = beta; a.in_dtype = in_dtype;
    a.mem = mem; a.B = B; a.H = H; a.T = T; a.dv = d_v; a.W = W; a.R = R; a.N = N;
    a.y = y; a.saved = saved; a.ws = static_cast<unsigned char*>(workspace);
    a.tb = 0; a.te = T;
    e = sdm_launch_scan_fwd(a, st);
    if (e != hipSuccess) return hip_fail(e, "sdm_scan_fwd launch");
    return SDM_OK;
}

size_t sdm_scan_fwd_chunked_workspace_bytes(int B, int H, int T, int W, int R) {
    if (B < 0 || H < 0 || T < 0 || W < 1 || R < 1) return 0;
    return sdm_chunk_ws_bytes(B, H, T, W, R);
}

int sdm_scan_fwd_chunked(const int32_t* w_idx, const float* w_val, int W, const int32_t* r_idx,
                         const float* r_val, int R, const void* v, const void* alpha, const void* beta,
                         int in_dtype, float* mem, int B, int H, int T, int d_v, int64_t N, float* y,
                         void* workspace, size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    int rc = check_scan_common(w_idx, w_val, W, r_idx, r_val, R, v, alpha, beta, in_dtype, mem, B,
                               H, T, d_v, N);
    if (rc != SDM_OK) return rc;
    if ((int64_t)B * H * T == 0) return SDM_OK;
    if (!y || !aligned(y, 16)) return fail(SDM_ERR_INVALID_ARG, "y must be a 16-byte aligned pointer");
    if (!sdm_chunk_shape_ok(W, R))
        return fail(SDM_ERR_UNSUPPORTED, "the chunked scan takes W, R <= %d (got W=%d R=%d)",
                    SDM_CHUNK_MAX_LIST, W, R);
    const size_t need = sdm_chunk_ws_bytes(B, H, T, W, R);
    if (!workspace || !aligned(workspace, 256))
        return fail(SDM_ERR_INVALID_ARG, "workspace must be a 256-byte aligned pointer");
    if (ws_bytes < need) return fail(SDM_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);
    hipStream_t st = (hipStream_t)stream;
    if (debug_checks() &&
        (rc = debug_check_ids(w_idx, W, r_idx, R, (int64_t)B * H * T, N, workspace, st)) != SDM_OK)
        return rc;
    hipError_t e = sdm_launch_zero_words(workspace, 4, st);
    if (e != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked flag reset");
    ScanFwdArgs a;
    a.w_idx = w_idx; a.w_val = w_val; a.r_idx = r_idx; a.r_val = r_val;
    a.v = v; a.alpha = alpha; a.beta = beta; a.in_dtype = in_dtype;
    a.mem = mem; a.B = B; a.H = H; a.T = T; a.dv = d_v; a.W = W; a.R = R; a.N = N;
    a.y = y; a.saved = nullptr; a.ws = static_cast<unsigned char*>(workspace);
    // Chunk ranges: the coefficients of range r + 1 (all chunks independent)
    // run on the second stream beside the scan of range r, which holds a
    // workgroup per (stream, slice) only.
    const int nch = (T + SDM_CHUNK - 1) / SDM_CHUNK;
    const int nr = nch >= 32 ? 8 : 1;
    // the first range is a quarter of the others: its coefficients overlap nothing
    auto bound = [&](int r) {
        return r == 0 ? 0 : r == nr ? nch : (int)((int64_t)nch * (4 * r - 3) / (4 * nr - 3));
    };
    auto range = [&](int r) {
        ScanFwdArgs b = a;
        b.tb = bound(r) * SDM_CHUNK;
        b.te = std::min(T, bound(r + 1) * SDM_CHUNK);
        return b;
    };
    auto coef = [&](const ScanFwdArgs& b, hipStream_t s) {
        SdmProfScope ps(SDM_K_CHUNK_COEF, s);
        return sdm_launch_chunk_coef(b, s);
    };
    auto scan = [&](const ScanFwdArgs& b) {
        SdmProfScope ps(SDM_K_CHUNK_SCAN, st);
        return sdm_launch_chunk_scan(b, st);
    };
    if (nr == 1) {
        a.tb = 0; a.te = T;
        if ((e = coef(a, st)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked coefficient launch");
        if ((e = scan(a)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked scan launch");
        return SDM_OK;
    }
    SidePipe& sp = side_pipe();
    std::lock_guard<std::mutex> lk(sp.mu);
    hipStream_t side;
    std::vector<hipEvent_t>* evp;
    int dev;
    if ((e = side_get(sp, nr + 1, &side, &evp, &dev)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked streams");
    std::vector<hipEvent_t>& ev = *evp;
    if ((e = hipEventRecord(ev[0], st)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked record");
    if ((e = hipStreamWaitEvent(side, ev[0], 0)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked wait");
    if ((e = coef(range(0), st)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked coefficient launch");
    for (int r = 0; r < nr; ++r) {
        if (r + 1 < nr) {
            if ((e = coef(range(r + 1), side)) != hipSuccess)
                return hip_fail(e, "sdm_scan_fwd_chunked coefficient launch");
            if ((e = hipEventRecord(ev[r + 1], side)) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked record");
        }
        if ((e = scan(range(r))) != hipSuccess) return hip_fail(e, "sdm_scan_fwd_chunked scan launch");
        if (r + 1 < nr && (e = hipStreamWaitEvent(st, ev[r + 1], 0)) != hipSuccess)
            return hip_fail(e, "sdm_scan_fwd_chunked wait");
    }
    return SDM_OK;
}

}  // extern "C"

// ---- fused forward: addressing pipelined with the scan over chunks of tokens ----

namespace {
// Validation of the optional steps either side of the scan (gates from
// pre-activations, the norm-gate epilogue).
int check_extras(const SdmFwdExtras* ex, int in_dtype, bool tok) {
    if (!ex) return SDM_OK;
    if (ex->gate_A || ex->gate_bdt) {
        if (!ex->gate_A || !ex->gate_bdt) return fail(SDM_ERR_INVALID_ARG, "A and b_dt go together");
        if (!aligned(ex->gate_A, 4) || !aligned(ex->gate_bdt, 4))
            return fail(SDM_ERR_INVALID_ARG, "misaligned A or b_dt");
    }
    if (ex->o) {
        if (ex->act != 0 && ex->act != 1) return fail(SDM_ERR_INVALID_ARG, "act must be 0 (identity) or 1 (SiLU)");
        if (!(ex->eps >= 0.f) || !std::isfinite(ex->eps)) return fail(SDM_ERR_INVALID_ARG, "eps must be finite and >= 0");
        if (tok && !ex->g) return fail(SDM_ERR_INVALID_ARG, "null output gate g");
        if (!aligned(ex->o, 16) || !aligned(ex->g, 16) || (ex->gamma && !aligned(ex->gamma, 16)) ||
            (ex->rstd && !aligned(ex->rstd, 4)))
            return fail(SDM_ERR_INVALID_ARG, "misaligned epilogue pointer (16-byte alignment required)");
    }
    (void)in_dtype;
    return SDM_OK;
}
}  // namespace

int sdm_forward_impl(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int d_k,
                     int W, int R, const void* v, const void* alpha, const void* beta, int in_dtype, float* mem,
                     int B, int H, int T, int d_v, int64_t N, int32_t* r_idx, float* r_val, int32_t* w_idx,
                     float* w_val, float* y, float* saved, size_t saved_bytes, int chunk, void* workspace,
                     size_t ws_bytes, void* stream, bool pipelined, const SdmFwdExtras* ex) {
    g_err[0] = 0;
    int s = 0;
    int rc = check_address(q, x_dtype, cb_q, B, H, T, d_k, N, R, r_idx, r_val, nullptr, &s);
    if (rc != SDM_OK) return rc;
    rc = check_address(k, x_dtype, cb_k, B, H, T, d_k, N, W, w_idx, w_val, nullptr, &s);
    if (rc != SDM_OK) return rc;
    rc = check_scan_common(w_idx, w_val, W, r_idx, r_val, R, v, alpha, beta, in_dtype, mem, B, H,
                           T, d_v, N);
    if (rc != SDM_OK) return rc;
    if (chunk < 0) return fail(SDM_ERR_INVALID_ARG, "chunk must be >= 0");
    if ((rc = check_extras(ex, in_dtype, (int64_t)B * H * T > 0)) != SDM_OK) return rc;
    if ((int64_t)B * H * T == 0) return SDM_OK;
    rc = check_scan_fwd_rest(W, R, in_dtype, B, H, T, d_v, y, saved, saved_bytes, workspace,
                             ws_bytes);
    if (rc != SDM_OK) return rc;

    hipStream_t st = (hipStream_t)stream;
    const float* gA = ex ? ex->gate_A : nullptr;
    const float* gbdt = ex ? ex->gate_bdt : nullptr;
    const bool epi = ex && ex->o;
    const int S = B * H;
    // the epilogue of tokens [tb, te), after their scan on the same stream
    auto epilogue = [&](int tb, int te, hipStream_t sx) -> hipError_t {
        if (!epi) return hipSuccess;
        SdmProfScope ps(SDM_K_NORM_GATE, sx);
        return sdm_launch_norm_gate(y, ex->g, in_dtype, ex->gamma, ex->eps, ex->act, S, T, tb, te - tb, d_v, ex->o,
                                    ex->rstd, sx);
    };
    // one token without an undo log, both sides in the same addressing mode and
    // W = R: addressing and the scan step in one launch
    if (T == 1 && !saved && W == R && (cb_q == nullptr) == (cb_k == nullptr)) {
        hipError_t e;
        {
            SdmProfScope ps(SDM_K_DECODE, st);
            e = sdm_launch_decode(q, k, x_dtype, cb_q, cb_k, B, H, d_k, s, W, v, alpha, beta, in_dtype, mem, N,
                                  d_v, r_idx, r_val, w_idx, w_val, y, static_cast<unsigned int*>(workspace), st,
                                  gA, gbdt);
        }
        if (e == hipSuccess) e = epilogue(0, 1, st);
        return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_forward single-token launch");
    }

    // pipeline stages of len tokens (multiples of 64 tokens, at most kMaxChunks
    // of them), the last one shorter.  The first stage's addressing overlaps
    // nothing; a shorter first stage (a quarter of len) left the scan idle
    // while the second stage's addressing ran beside the short first scan:
    // 1.4B-shaped step 6.27 against 6.15 ms, learned-M0 5.54 against 5.38.
    int len = T, first = T, nchunks = 1;
    if (pipelined && (chunk > 0 || T >= 2048)) {
        len = chunk > 0 ? round_up(chunk, 64) : round_up((T + 3) / 4, 64);
        len = std::max(len, round_up((T + kMaxChunks - 1) / kMaxChunks, 64));
        first = std::min(T, len);
        nchunks = (T + len - 1) / len;
    }
    auto stage_begin = [&](int c) { return c == 0 ? 0 : std::min(T, first + (c - 1) * len); };

    hipError_t e = sdm_launch_zero_words(workspace, 4, st);
    if (e != hipSuccess) return hip_fail(e, "sdm_forward flag reset");
    ScanFwdArgs a;
    a.w_idx = w_idx; a.w_val = w_val; a.r_idx = r_idx; a.r_val = r_val;
    a.v = v; a.alpha = alpha; a.beta = beta; a.in_dtype = in_dtype;
    a.mem = mem; a.B = B; a.H = H; a.T = T; a.dv = d_v; a.W = W; a.R = R; a.N = N;
    a.y = y; a.saved = saved; a.ws = static_cast<unsigned char*>(workspace);
    a.gate_A = gA; a.gate_bdt = gbdt;

    // lds_free > 0: the stage's addressing runs beside a scan stage, which holds
    // the rest of every CU's LDS
    auto stage_front = [&](int tb, int te, hipStream_t sx, size_t lds_free) -> hipError_t {
        hipError_t ee;
        {
            SdmProfScope ps(SDM_K_ADDRESS, sx);
            ee = sdm_launch_address(q, x_dtype, cb_q, B, H, T, tb, te - tb, d_k, s, R, r_idx, r_val,
                                    nullptr, sx, lds_free);
        }
        if (ee != hipSuccess) return ee;
        {
            SdmProfScope ps(SDM_K_ADDRESS, sx);
            ee = sdm_launch_address(k, x_dtype, cb_k, B, H, T, tb, te - tb, d_k, s, W, w_idx, w_val,
                                    nullptr, sx, lds_free);
        }
        if (ee != hipSuccess) return ee;
        ScanFwdArgs ac = a;
        ac.tb = tb;
        ac.te = te;
        return sdm_launch_fwd_prep_range(ac, sx);
    };

    if (nchunks == 1) {
        e = stage_front(0, T, st, 0);
        if (e == hipSuccess) {
            a.tb = 0;
            a.te = T;
            e = sdm_launch_fwd_scan_range(a, st);
        }
        if (e == hipSuccess) e = epilogue(0, T, st);
        return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_forward launch");
    }

    SidePipe& sp = side_pipe();
    std::lock_guard<std::mutex> lk(sp.mu);
    hipStream_t side = nullptr;
    std::vector<hipEvent_t>* evp = nullptr;
    int dev = 0;
    if ((e = side_get(sp, nchunks + 1, &side, &evp, &dev)) != hipSuccess) return hip_fail(e, "sdm_forward side stream");
    std::vector<hipEvent_t>& ev = *evp;
    // the side stream starts after the caller's earlier work; chunk c's scan waits for its front
    if ((e = hipEventRecord(ev[0], st)) != hipSuccess) return hip_fail(e, "sdm_forward record");
    if ((e = hipStreamWaitEvent(side, ev[0], 0)) != hipSuccess) return hip_fail(e, "sdm_forward wait");
    const size_t scan_lds = sdm_fwd_scan_lds(a);
    const size_t lds_beside = scan_lds < kCuLds ? kCuLds - scan_lds : 0;
    for (int c = 0; c < nchunks; ++c) {
        const int tb = stage_begin(c), te = stage_begin(c + 1) > tb ? stage_begin(c + 1) : T;
        // stage 0's addressing has the device to itself; later stages' run beside the previous scan
        if ((e = stage_front(tb, te, side, c == 0 ? 0 : lds_beside)) != hipSuccess)
            return hip_fail(e, "sdm_forward launch");
        if ((e = hipEventRecord(ev[c + 1], side)) != hipSuccess) return hip_fail(e, "sdm_forward record");
        if ((e = hipStreamWaitEvent(st, ev[c + 1], 0)) != hipSuccess) return hip_fail(e, "sdm_forward wait");
        a.tb = tb;
        a.te = te;
        if ((e = sdm_launch_fwd_scan_range(a, st)) != hipSuccess) return hip_fail(e, "sdm_forward launch");
        if ((e = epilogue(tb, te, st)) != hipSuccess) return hip_fail(e, "sdm_forward epilogue launch");
    }
    return SDM_OK;
}

int sdm_set_error(int status, const char* msg) { return fail(status, "%s", msg); }

extern "C" {

int sdm_forward(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int d_k,
                int topk, const void* v, const void* alpha, const void* beta, int in_dtype, float* mem,
                int B, int H, int T, int d_v, int64_t N, int32_t* r_idx, float* r_val, int32_t* w_idx,
                float* w_val, float* y, float* saved, size_t saved_bytes, int chunk, void* workspace,
                size_t ws_bytes, void* stream) {
    return sdm_forward_impl(q, k, x_dtype, cb_q, cb_k, d_k, topk, topk, v, alpha, beta, in_dtype, mem, B, H, T,
                            d_v, N, r_idx, r_val, w_idx, w_val, y, saved, saved_bytes, chunk, workspace, ws_bytes,
                            stream, true, nullptr);
}

}  // extern "C"

namespace {
// The body of sdm_scan_bwd; gA, gbdt set: alpha and beta hold the gates'
// pre-activations and the records take the gates formed from them.
int scan_bwd_impl(const void* cb_q, const void* cb_k, int cb_dtype, int d_k, const int32_t* w_idx,
                  const float* w_val, int W, const int32_t* r_idx, const float* r_val, int R,
                  const void* v, const void* alpha, const void* beta, int in_dtype, float* mem,
                  const float* saved, size_t saved_bytes, const float* dy, const float* dmem_T,
                  int chunk, int B, int H, int T, int d_v, int64_t N, float* dq, float* dk,
                  float* dv, float* dalpha, float* dbeta, float* dmem0, float* dw_val,
                  float* dr_val, void* workspace, size_t ws_bytes, void* stream, const float* gA,
                  const float* gbdt) {
    int rc = check_scan_common(w_idx, w_val, W, r_idx, r_val, R, v, alpha, beta, in_dtype, mem, B,
                               H, T, d_v, N);
    if (rc != SDM_OK) return rc;
    if (chunk < 1) return fail(SDM_ERR_INVALID_ARG, "chunk must be >= 1");
    const bool tok = (int64_t)B * H * T > 0;
    if ((tok && (!saved || !dy || !dv || !dalpha || !dbeta)) || ((int64_t)B * H > 0 && !dmem0))
        return fail(SDM_ERR_INVALID_ARG, "null pointer (saved, dy, dv, dalpha, dbeta, dmem0 are required)");
    if (!aligned(saved, 16) || !aligned(dy, 16) || !aligned(dv, 16) || !aligned(dmem0, 16) ||
        (dmem_T && !aligned(dmem_T, 16)))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer (16-byte alignment required)");
    if (saved_bytes < sdm_scan_saved_bytes(B, H, T, W, d_v))
        return fail(SDM_ERR_WORKSPACE, "saved buffer too small");
    const int s = isqrt64(N);
    if (dq || dk) {
        if (!valid_dtype(cb_dtype)) return fail(SDM_ERR_INVALID_ARG, "cb_dtype must be SDM_F32 or SDM_BF16");
        if (s < 0) return fail(SDM_ERR_INVALID_ARG, "addressing gradients need a perfect-square N");
        if (W > s || R > s) return fail(SDM_ERR_INVALID_ARG, "W, R must be <= sqrt(N) for addressing gradients");
        if (dq && !cb_q && d_k != 2 * s) return fail(SDM_ERR_INVALID_ARG, "direct mode needs d_k == 2*sqrt(N)");
        if (dk && !cb_k && d_k != 2 * s) return fail(SDM_ERR_INVALID_ARG, "direct mode needs d_k == 2*sqrt(N)");
        if ((cb_q || cb_k) && (d_k % 2 || d_k < 2)) return fail(SDM_ERR_INVALID_ARG, "codebook mode needs an even d_k");
    }
    if (!sdm_bwd_plan_ok(W, R, d_v, in_dtype))
        return fail(SDM_ERR_UNSUPPORTED, "no backward launch plan for W=%d R=%d d_v=%d", W, R, d_v);
    const size_t need = sdm_bwd_ws_bytes(B, H, T, W, R, d_v);
    if (!workspace || !aligned(workspace, 256))
        return fail(SDM_ERR_INVALID_ARG, "workspace must be a 256-byte aligned pointer");
    if (ws_bytes < need) return fail(SDM_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);
    hipStream_t st = (hipStream_t)stream;
    if (debug_checks() && (int64_t)B * H * T > 0 &&
        (rc = debug_check_ids(w_idx, W, r_idx, R, (int64_t)B * H * T, N, workspace, st)) != SDM_OK)
        return rc;
    hipError_t e = sdm_launch_zero_words(workspace, 4, st);
    if (e != hipSuccess) return hip_fail(e, "sdm_scan_bwd flag reset");
    // adjoint of the memory starts as dL/dM_T (on `stream`, before the first scan;
    // the records do not need it, so the pipelined path overlaps the two)
    const size_t memel = (size_t)B * H * N * d_v;
    auto init_adjoint = [&]() -> hipError_t {
        SdmProfScope ps(SDM_K_MEM_INIT, st);
        if (dmem_T == nullptr) return sdm_launch_mem_init(dmem0, nullptr, B, H, N, d_v, st);
        if (dmem_T != dmem0) return sdm_launch_copy(dmem0, dmem_T, memel, st);
        return hipSuccess;
    };
    if ((int64_t)B * H * T == 0) {
        if ((e = init_adjoint()) != hipSuccess) return hip_fail(e, "sdm_scan_bwd adjoint init");
        return SDM_OK;
    }
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    const size_t ST = (size_t)B * H * T;
    float* spare = reinterpret_cast<float*>(ws + need - ST * (W + R) * sizeof(float));
    ScanBwdArgs a;
    a.w_idx = w_idx; a.w_val = w_val; a.r_idx = r_idx; a.r_val = r_val;
    a.v = v; a.alpha = alpha; a.beta = beta; a.in_dtype = in_dtype;
    a.mem = mem; a.saved = saved; a.dy = dy; a.chunk = chunk;
    a.B = B; a.H = H; a.T = T; a.dv = d_v; a.W = W; a.R = R; a.N = N;
    a.dv_out = dv; a.dalpha = dalpha; a.dbeta = dbeta; a.G = dmem0;
    a.dw_val = dw_val ? dw_val : spare;
    a.dr_val = dr_val ? dr_val : spare + ST * W;
    a.ws = ws;
    a.gate_A = gA;
    a.gate_bdt = gbdt;
    a.line = sdm_bwd_line_io(a) ? 1 : 0;   // one decision for every stage and the reduce

    // Stages of tokens from the end of the sequence down: a short first stage,
    // then stages of len = max(chunk, T/4) tokens (multiples of 64, at most
    // about kMaxChunks of them); chunk >= T runs one stage.  Stage c's scan
    // runs on `stream`; its records, and the sums and addressing gradients of
    // the stage before, run on the library's second stream meanwhile.
    int len = T, first = T;
    if (chunk < T) {
        len = round_up(std::max(chunk, (T + 3) / 4), 64);
        len = std::max(len, round_up((T + kMaxChunks - 2) / (kMaxChunks - 1), 64));
        first = std::min(T, round_up(std::max(len / 4, 64), 64));
    }
    // first and last stages short (nothing overlaps the first stage's records or
    // the last stage's gradient tails); the tokens between them in even stages of
    // at most len (multiples of 64)
    int nmid = 0, mid = 0, last = 0;
    if (first < T) {
        last = std::min(first, T - first);
        const int rest = T - first - last;
        nmid = rest > 0 ? (rest + len - 1) / len : 0;
        mid = nmid > 0 ? round_up((rest + nmid - 1) / nmid, 64) : 0;
    }
    const int nchunks = first >= T ? 1 : 1 + nmid + 1;
    auto stage_end = [&](int c) {
        if (c == 0) return T;
        if (c <= nmid + 1) return std::max(last, T - first - (c - 1) * mid);
        return 0;
    };
    auto ranged = [&](int c) {
        ScanBwdArgs ac = a;
        ac.te = stage_end(c);
        ac.tb = stage_end(c + 1);
        return ac;
    };
    auto post = [&](const ScanBwdArgs& ac, hipStream_t sx) -> hipError_t {
        hipError_t ee = sdm_launch_bwd_reduce_range(ac, sx);
        if (ee != hipSuccess) return ee;
        if (dq) {
            SdmProfScope ps(SDM_K_ADDRESS_BWD, sx);
            ee = sdm_launch_address_bwd(cb_q, cb_dtype, B, H, T, ac.tb, ac.te - ac.tb, d_k, s, R, r_idx, r_val,
                                        a.dr_val, dq, sx);
            if (ee != hipSuccess) return ee;
        }
        if (dk) {
            SdmProfScope ps(SDM_K_ADDRESS_BWD, sx);
            ee = sdm_launch_address_bwd(cb_k, cb_dtype, B, H, T, ac.tb, ac.te - ac.tb, d_k, s, W, w_idx, w_val,
                                        a.dw_val, dk, sx);
        }
        return ee;
    };
    if (nchunks == 1) {
        ScanBwdArgs ac = ranged(0);
        if ((e = init_adjoint()) != hipSuccess) return hip_fail(e, "sdm_scan_bwd adjoint init");
        if ((e = sdm_launch_bwd_prep_range(ac, st)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd launch");
        if ((e = sdm_launch_bwd_scan_range(ac, st)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd launch");
        if ((e = post(ac, st)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd launch");
        return SDM_OK;
    }
    SidePipe& sp = side_pipe();
    std::lock_guard<std::mutex> lk(sp.mu);
    hipStream_t side = nullptr;
    std::vector<hipEvent_t>* evp = nullptr;
    int dev = 0;
    // events: [0] start, [1 + c] records of stage c ready, [1 + nchunks + c] scan of stage c done, last: side done
    if ((e = side_get(sp, 2 * nchunks + 2, &side, &evp, &dev)) != hipSuccess)
        return hip_fail(e, "sdm_scan_bwd side stream");
    std::vector<hipEvent_t>& ev = *evp;
    hipEvent_t ev_start = ev[0], ev_end = ev[2 * nchunks + 1];
    auto ev_prep = [&](int c) { return ev[1 + c]; };
    auto ev_scan = [&](int c) { return ev[1 + nchunks + c]; };
    // the flag reset above (and the caller's earlier work) precede the side stream;
    // the adjoint init follows on `stream`, beside the first stages' records
    if ((e = hipEventRecord(ev_start, st)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd record");
    if ((e = hipStreamWaitEvent(side, ev_start, 0)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd wait");
    if ((e = init_adjoint()) != hipSuccess) return hip_fail(e, "sdm_scan_bwd adjoint init");
    // side: prep 0, prep 1, then for each c: [scan c done] post c, prep c + 2
    for (int c = 0; c < std::min(2, nchunks); ++c) {
        if ((e = sdm_launch_bwd_prep_range(ranged(c), side)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd launch");
        if ((e = hipEventRecord(ev_prep(c), side)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd record");
    }
    for (int c = 0; c < nchunks; ++c) {
        const ScanBwdArgs ac = ranged(c);
        if ((e = hipStreamWaitEvent(st, ev_prep(c), 0)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd wait");
        if ((e = sdm_launch_bwd_scan_range(ac, st)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd launch");
        if ((e = hipEventRecord(ev_scan(c), st)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd record");
        if ((e = hipStreamWaitEvent(side, ev_scan(c), 0)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd wait");
        if ((e = post(ac, side)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd launch");
        if (c + 2 < nchunks) {
            if ((e = sdm_launch_bwd_prep_range(ranged(c + 2), side)) != hipSuccess)
                return hip_fail(e, "sdm_scan_bwd launch");
            if ((e = hipEventRecord(ev_prep(c + 2), side)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd record");
        }
    }
    // everything the call enqueued is ordered before later work on `stream`
    if ((e = hipEventRecord(ev_end, side)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd record");
    if ((e = hipStreamWaitEvent(st, ev_end, 0)) != hipSuccess) return hip_fail(e, "sdm_scan_bwd wait");
    return SDM_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Regions of sdm_layer_bwd's workspace: the scan's, dy, dalpha and dbeta, the
// epilogue's dgamma partial sums.
struct LayerBwdWs {
    size_t scan, dy, dab, part, total;
};
LayerBwdWs layer_bwd_ws(int B, int H, int T, int W, int R, int d_v) {
    LayerBwdWs w;
    const size_t ST = (size_t)B * H * T;
    w.scan = 0;
    w.dy = align256(sdm_bwd_ws_bytes(B, H, T, W, R, d_v));
    w.dab = w.dy + align256(ST * d_v * sizeof(float));
    w.part = w.dab + align256(2 * ST * sizeof(float));
    w.total = w.part + align256(sdm_norm_gate_bwd_ws((int64_t)ST, d_v));
    return w;
}

int check_gate_args(const void* a_pre, const void* b_pre, int dtype, const float* A, const float* b_dt, int B,
                    int H, int T) {
    if (B < 0 || H < 0 || T < 0) return fail(SDM_ERR_INVALID_ARG, "B, H, T must be >= 0");
    if ((int64_t)B * H > kMaxStreams) return fail(SDM_ERR_UNSUPPORTED, "B*H must be <= %d", kMaxStreams);
    if (!valid_dtype(dtype)) return fail(SDM_ERR_INVALID_ARG, "dtype must be SDM_F32 or SDM_BF16");
    if (H > 0 && (!A || !b_dt)) return fail(SDM_ERR_INVALID_ARG, "null A or b_dt");
    if ((int64_t)B * H * T > 0 && (!a_pre || !b_pre)) return fail(SDM_ERR_INVALID_ARG, "null pre-activation");
    if (!aligned(A, 4) || !aligned(b_dt, 4) || !aligned(a_pre, 4) || !aligned(b_pre, 4))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer");
    return SDM_OK;
}

int check_norm_gate_args(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act, int B,
                         int H, int T, int d_v) {
    if (B < 0 || H < 0 || T < 0) return fail(SDM_ERR_INVALID_ARG, "B, H, T must be >= 0");
    if (d_v < 4 || d_v % 4) return fail(SDM_ERR_INVALID_ARG, "d_v must be a positive multiple of 4");
    if (d_v > 4096) return fail(SDM_ERR_UNSUPPORTED, "d_v must be <= 4096");
    if (!valid_dtype(g_dtype)) return fail(SDM_ERR_INVALID_ARG, "g_dtype must be SDM_F32 or SDM_BF16");
    if (act != 0 && act != 1) return fail(SDM_ERR_INVALID_ARG, "act must be 0 (identity) or 1 (SiLU)");
    if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(SDM_ERR_INVALID_ARG, "eps must be finite and >= 0");
    if ((int64_t)B * H * T > 0 && (!y || !g)) return fail(SDM_ERR_INVALID_ARG, "null y or g");
    if (!aligned(y, 16) || !aligned(g, 16) || (gamma && !aligned(gamma, 16)))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer (16-byte alignment required)");
    return SDM_OK;
}
}  // namespace

extern "C" {

int sdm_scan_bwd(const void* cb_q, const void* cb_k, int cb_dtype, int d_k, const int32_t* w_idx,
                 const float* w_val, int W, const int32_t* r_idx, const float* r_val, int R,
                 const void* v, const void* alpha, const void* beta, int in_dtype, float* mem,
                 const float* saved, size_t saved_bytes, const float* dy, const float* dmem_T,
                 int chunk, int B, int H, int T, int d_v, int64_t N, float* dq, float* dk,
                 float* dv, float* dalpha, float* dbeta, float* dmem0, float* dw_val,
                 float* dr_val, void* workspace, size_t ws_bytes, void* stream) {
    return scan_bwd_impl(cb_q, cb_k, cb_dtype, d_k, w_idx, w_val, W, r_idx, r_val, R, v, alpha, beta, in_dtype, mem,
                         saved, saved_bytes, dy, dmem_T, chunk, B, H, T, d_v, N, dq, dk, dv, dalpha, dbeta, dmem0,
                         dw_val, dr_val, workspace, ws_bytes, stream, nullptr, nullptr);
}

// ---- the steps either side of the recurrence (Sec. 3.1 steps 2 and 4) ----

int sdm_gates(const void* a_pre, const void* b_pre, int dtype, const float* A, const float* b_dt, int B, int H,
              int T, float* alpha, float* beta, void* stream) {
    g_err[0] = 0;
    int rc = check_gate_args(a_pre, b_pre, dtype, A, b_dt, B, H, T);
    if (rc != SDM_OK) return rc;
    if ((int64_t)B * H * T == 0) return SDM_OK;
    if (!alpha || !beta || !aligned(alpha, 4) || !aligned(beta, 4))
        return fail(SDM_ERR_INVALID_ARG, "null or misaligned alpha / beta output");
    hipError_t e;
    {
        SdmProfScope ps(SDM_K_GATES, (hipStream_t)stream);
        e = sdm_launch_gates(a_pre, b_pre, dtype, A, b_dt, B, H, T, alpha, beta, (hipStream_t)stream);
    }
    return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_gates launch");
}

int sdm_gates_bwd(const void* a_pre, const void* b_pre, int dtype, const float* A, const float* b_dt,
                  const float* dalpha, const float* dbeta, int B, int H, int T, float* da, float* db, float* dA,
                  float* db_dt, void* stream) {
    g_err[0] = 0;
    int rc = check_gate_args(a_pre, b_pre, dtype, A, b_dt, B, H, T);
    if (rc != SDM_OK) return rc;
    if (H == 0) return SDM_OK;
    if (!dA || !db_dt || !aligned(dA, 4) || !aligned(db_dt, 4))
        return fail(SDM_ERR_INVALID_ARG, "null or misaligned dA / db_dt");
    if ((int64_t)B * T > 0 && (!dalpha || !dbeta || !da || !db || !aligned(dalpha, 4) || !aligned(dbeta, 4) ||
                               !aligned(da, 4) || !aligned(db, 4)))
        return fail(SDM_ERR_INVALID_ARG, "null or misaligned gradient pointer");
    hipError_t e;
    {
        SdmProfScope ps(SDM_K_GATES, (hipStream_t)stream);
        e = sdm_launch_gates_bwd(a_pre, b_pre, dtype, A, b_dt, dalpha, dbeta, B, H, T, da, db, dA, db_dt,
                                 (hipStream_t)stream);
    }
    return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_gates_bwd launch");
}

int sdm_norm_gate(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act, int B, int H,
                  int T, int d_v, float* o, float* rstd, void* stream) {
    g_err[0] = 0;
    int rc = check_norm_gate_args(y, g, g_dtype, gamma, eps, act, B, H, T, d_v);
    if (rc != SDM_OK) return rc;
    if ((int64_t)B * H * T == 0) return SDM_OK;
    if (!o || !aligned(o, 16) || (rstd && !aligned(rstd, 4)))
        return fail(SDM_ERR_INVALID_ARG, "null or misaligned output");
    hipError_t e;
    {
        SdmProfScope ps(SDM_K_NORM_GATE, (hipStream_t)stream);
        e = sdm_launch_norm_gate(y, g, g_dtype, gamma, eps, act, (int64_t)B * H, T, 0, T, d_v, o, rstd,
                                 (hipStream_t)stream);
    }
    return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_norm_gate launch");
}

size_t sdm_norm_gate_bwd_workspace_bytes(int B, int H, int T, int d_v) {
    if (B < 0 || H < 0 || T < 0 || d_v < 4) return 0;
    return align256(sdm_norm_gate_bwd_ws((int64_t)B * H * T, d_v));
}

int sdm_norm_gate_bwd(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act,
                      const float* dout, int B, int H, int T, int d_v, float* dy, float* dg, float* dgamma,
                      void* workspace, size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    int rc = check_norm_gate_args(y, g, g_dtype, gamma, eps, act, B, H, T, d_v);
    if (rc != SDM_OK) return rc;
    const bool tok = (int64_t)B * H * T > 0;
    if (tok && (!dout || !dy || !dg)) return fail(SDM_ERR_INVALID_ARG, "null dout, dy or dg");
    if (!aligned(dout, 16) || !aligned(dy, 16) || !aligned(dg, 16) || (dgamma && !aligned(dgamma, 4)))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer (16-byte alignment required)");
    const size_t need = sdm_norm_gate_bwd_workspace_bytes(B, H, T, d_v);
    if (!workspace || !aligned(workspace, 256))
        return fail(SDM_ERR_INVALID_ARG, "workspace must be a 256-byte aligned pointer");
    if (ws_bytes < need) return fail(SDM_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, need);
    hipError_t e;
    {
        SdmProfScope ps(SDM_K_NORM_GATE, (hipStream_t)stream);
        e = sdm_launch_norm_gate_bwd(y, g, g_dtype, gamma, eps, act, dout, (int64_t)B * H * T, d_v, dy, dg, dgamma,
                                     static_cast<float*>(workspace), (hipStream_t)stream);
    }
    return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_norm_gate_bwd launch");
}

int sdm_layer_fwd(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int d_k, int W,
                  int R, const void* v, const void* a_pre, const void* b_pre, const void* g, int in_dtype,
                  const float* A, const float* b_dt, const float* gamma, float eps, int act, float* mem, int B,
                  int H, int T, int d_v, int64_t N, int32_t* r_idx, float* r_val, int32_t* w_idx, float* w_val,
                  float* y, float* o, float* rstd, float* saved, size_t saved_bytes, int chunk, void* workspace,
                  size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    int rc = check_gate_args(a_pre, b_pre, in_dtype, A, b_dt, B, H, T);
    if (rc != SDM_OK) return rc;
    rc = check_norm_gate_args(y, g, in_dtype, gamma, eps, act, B, H, T, d_v);
    if (rc != SDM_OK) return rc;
    if ((int64_t)B * H * T > 0 && !o) return fail(SDM_ERR_INVALID_ARG, "null output o");
    SdmFwdExtras ex;
    ex.gate_A = A;
    ex.gate_bdt = b_dt;
    ex.g = g;
    ex.gamma = gamma;
    ex.eps = eps;
    ex.act = act;
    ex.o = o;
    ex.rstd = rstd;
    return sdm_forward_impl(q, k, x_dtype, cb_q, cb_k, d_k, W, R, v, a_pre, b_pre, in_dtype, mem, B, H, T, d_v, N,
                            r_idx, r_val, w_idx, w_val, y, saved, saved_bytes, chunk, workspace, ws_bytes, stream,
                            true, &ex);
}

size_t sdm_layer_bwd_workspace_bytes(int B, int H, int T, int W, int R, int d_v) {
    if (B < 0 || H < 0 || T < 0 || W < 1 || R < 1 || d_v < 4) return 0;
    return layer_bwd_ws(B, H, T, W, R, d_v).total;
}

int sdm_layer_bwd(const void* cb_q, const void* cb_k, int cb_dtype, int d_k, const int32_t* w_idx,
                  const float* w_val, int W, const int32_t* r_idx, const float* r_val, int R, const void* v,
                  const void* a_pre, const void* b_pre, const void* g, int in_dtype, const float* A,
                  const float* b_dt, const float* gamma, float eps, int act, float* mem, const float* saved,
                  size_t saved_bytes, const float* y, const float* dout, const float* dmem_T, int chunk, int B,
                  int H, int T, int d_v, int64_t N, float* dq, float* dk, float* dv, float* da, float* db,
                  float* dA, float* db_dt, float* dg, float* dgamma, float* dmem0, void* workspace,
                  size_t ws_bytes, void* stream) {
    g_err[0] = 0;
    int rc = check_gate_args(a_pre, b_pre, in_dtype, A, b_dt, B, H, T);
    if (rc != SDM_OK) return rc;
    rc = check_norm_gate_args(y, g, in_dtype, gamma, eps, act, B, H, T, d_v);
    if (rc != SDM_OK) return rc;
    rc = check_scan_common(w_idx, w_val, W, r_idx, r_val, R, v, a_pre, b_pre, in_dtype, mem, B, H, T, d_v, N);
    if (rc != SDM_OK) return rc;
    const bool tok = (int64_t)B * H * T > 0;
    if (tok && (!dout || !da || !db || !dg)) return fail(SDM_ERR_INVALID_ARG, "null dout, da, db or dg");
    if (H > 0 && (!dA || !db_dt)) return fail(SDM_ERR_INVALID_ARG, "null dA or db_dt");
    if (!aligned(dout, 16) || !aligned(dg, 16) || !aligned(da, 4) || !aligned(db, 4) || !aligned(dA, 4) ||
        !aligned(db_dt, 4) || (dgamma && !aligned(dgamma, 4)))
        return fail(SDM_ERR_INVALID_ARG, "misaligned pointer");
    const LayerBwdWs L = layer_bwd_ws(B, H, T, W, R, d_v);
    if (!workspace || !aligned(workspace, 256))
        return fail(SDM_ERR_INVALID_ARG, "workspace must be a 256-byte aligned pointer");
    if (ws_bytes < L.total) return fail(SDM_ERR_WORKSPACE, "workspace too small: %zu < %zu", ws_bytes, L.total);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    float* dy = reinterpret_cast<float*>(ws + L.dy);
    float* dal = reinterpret_cast<float*>(ws + L.dab);
    float* dbe = dal + (size_t)B * H * T;
    float* part = reinterpret_cast<float*>(ws + L.part);
    hipStream_t st = (hipStream_t)stream;
    hipError_t e;
    // 1. epilogue backward over the whole sequence: dy (the scan's upstream gradient), dg, dgamma
    {
        SdmProfScope ps(SDM_K_NORM_GATE, st);
        e = sdm_launch_norm_gate_bwd(y, g, in_dtype, gamma, eps, act, dout, (int64_t)B * H * T, d_v, dy, dg, dgamma,
                                     part, st);
    }
    if (e != hipSuccess) return hip_fail(e, "sdm_layer_bwd epilogue launch");
    // 2. the recurrence's backward, its records taking the gates formed from the pre-activations
    rc = scan_bwd_impl(cb_q, cb_k, cb_dtype, d_k, w_idx, w_val, W, r_idx, r_val, R, v, a_pre, b_pre, in_dtype, mem,
                       saved, saved_bytes, dy, dmem_T, chunk, B, H, T, d_v, N, dq, dk, dv, dal, dbe, dmem0, nullptr,
                       nullptr, ws, L.dy, stream, A, b_dt);
    if (rc != SDM_OK) return rc;
    // 3. the gates' backward: da, db and the per-head sums dA, db_dt
    {
        SdmProfScope ps(SDM_K_GATES, st);
        e = sdm_launch_gates_bwd(a_pre, b_pre, in_dtype, A, b_dt, dal, dbe, B, H, T, da, db, dA, db_dt, st);
    }
    return e == hipSuccess ? SDM_OK : hip_fail(e, "sdm_layer_bwd gates launch");
}

int sdm_mem_init(float* dst, const float* m0, int B, int H, int64_t N, int d_v, void* stream) {
    g_err[0] = 0;
    if (B < 0 || H < 0 || N < 0 || d_v < 0) return fail(SDM_ERR_INVALID_ARG, "negative size");
    if (d_v % 4) return fail(SDM_ERR_INVALID_ARG, "d_v must be a multiple of 4");
    if ((int64_t)B * H > kMaxStreams) return fail(SDM_ERR_UNSUPPORTED, "B*H must be <= %d", kMaxStreams);
    if (!dst || !aligned(dst, 16) || (m0 && !aligned(m0, 16)))
        return fail(SDM_ERR_INVALID_ARG, "null or misaligned pointer");
    hipError_t e;
    {
        SdmProfScope ps(SDM_K_MEM_INIT, (hipStream_t)stream);
        e = sdm_launch_mem_init(dst, m0, B, H, N, d_v, (hipStream_t)stream);
    }
    if (e != hipSuccess) return hip_fail(e, "sdm_mem_init launch");
    return SDM_OK;
}

int sdm_check_device_errors(void* workspace, void* stream) {
    g_err[0] = 0;
    if (!workspace) return fail(SDM_ERR_INVALID_ARG, "null workspace");
    hipStream_t st = (hipStream_t)stream;
    unsigned int flag = 0;
    hipError_t e = hipMemcpyAsync(&flag, workspace, sizeof(flag), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "sdm_check_device_errors");
    if (flag) {
        e = sdm_launch_zero_words(workspace, 1, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "sdm_check_device_errors clear");
        if (flag & 1u) return fail(SDM_ERR_DEVICE_CHECK, "a slot id outside [0, N) was clamped");
        return fail(SDM_ERR_DEVICE_CHECK, "the chunked scan met a forget gate alpha <= 0");
    }
    return SDM_OK;
}

}  // extern "C"
