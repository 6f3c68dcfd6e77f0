// Forward sparse gated-delta scan (Sec. 3.1 steps 2-3: Eqs. sdm-decay,
// sdm-write in the read-back form of Fig. 2, sdm-read on M_t) for gfx950.
//
// Given the addressing, the recurrence is independent per value column, so
// one wave owns one (stream, column slice) pair for the whole sequence and
// no two waves ever touch the same bytes of the memory table.
//
// Per wave:
//  * a PD-token software pipeline: the rows of token t+PD are loaded (HBM,
//    one 16-byte piece per lane, CQ lanes per row slice) while token t is
//    computed;
//  * a row loaded for token u before tokens u-PD+1 .. u-1 have written it
//    would be stale.  The prep kernel records, per row, the latest writer
//    within that window (or the token itself, for reads); such rows are
//    taken from an LDS ring holding the last PD tokens' written rows.  Older
//    writers stored before the load was issued, in program order of the same
//    wave, so the load returns their value;
//  * per-token records (slots, weights, links, gates) are staged in LDS in
//    blocks of G tokens, loaded L tokens ahead with 16-byte loads.
#include <algorithm>

#include "sdm_common.h"
#include "sdm_internal.h"
#include "sdm.h"

namespace {

constexpr int G = 4;            // tokens per staging block
constexpr int MAX_WPB = 4;      // waves (column slices) per workgroup, at most
constexpr int LDS_LIMIT = 160 * 1024;

template <int PD>
__host__ __device__ constexpr int stage_lead() {   // L: records of token u are staged by step u-PD
    return ((G + PD + G - 1) / G) * G;
}
template <int PD>
__host__ __device__ constexpr int stage_slots() {
    return stage_lead<PD>() <= 8 ? 8 : (stage_lead<PD>() <= 16 ? 16 : 32);
}

// Staging of the G records (and v slices) of tokens [u0, u0 + G): global -> registers.
// Every lane always loads: indices at or past te are clamped to valid data (the
// surplus is never read), so the loads carry no control flow.
template <typename VT, int SW, int NR>
__device__ __forceinline__ void stage_load(u4v (&st)[NR], u2v& stv, const unsigned char* srec,
                                           const VT* sv, int u0, int te, int dv, int slice,
                                           int rec_bytes, int lane) {
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;   // 8-byte pieces per token
    const int ub = min(u0, te - 1);
    const int cnt = min(G, te - ub);
    const u4v* src = reinterpret_cast<const u4v*>(srec + (size_t)ub * rec_bytes);
    const int last = cnt * rec_bytes / 16 - 1;
#pragma unroll
    for (int r = 0; r < NR; ++r) st[r] = src[min(r * SDM_WAVE + lane, last)];
    const int tk = min(lane / ppt, cnt - 1);
    const int pc = min(lane % ppt, (dv - slice * SW) * (int)sizeof(VT) / 8 - 1);
    stv = *reinterpret_cast<const u2v*>(
        reinterpret_cast<const unsigned char*>(sv + (size_t)(ub + tk) * dv) + pc * 8);
}

// Registers -> LDS rings (slot = token mod NS; a block never wraps: u0 % G == 0).
template <typename VT, int SW, int NS, int NR>
__device__ __forceinline__ void stage_store(const u4v (&st)[NR], u2v stv, unsigned char* rring,
                                            unsigned char* vring, int u0, int rec_bytes, int lane) {
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
    u4v* dst = reinterpret_cast<u4v*>(rring + (u0 & (NS - 1)) * rec_bytes);
    const int nchunk = G * rec_bytes / 16;   // <= NR * 64 (checked by the host plan)
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int c = r * SDM_WAVE + lane;
        if (c < nchunk) dst[c] = st[r];
    }
    const int tk = lane / ppt, pc = lane % ppt;
    if (tk < G) *reinterpret_cast<u2v*>(vring + ((u0 + tk) & (NS - 1)) * VB + pc * 8) = stv;
}

// Rows of token u (state as of its load) for this lane: write rows i_n, read rows j_m.
template <int K, int RG, int NS>
__device__ __forceinline__ void issue_rows(v4f (&Pw)[K], v4f (&Pr)[K], const unsigned char* rring,
                                           const FwdRec& L, const float* tab, int u, int dv,
                                           int rg) {
    const unsigned char* rec = rring + (u & (NS - 1)) * L.bytes;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = min(rg + RG * k, L.W - 1);
        const int m = min(rg + RG * k, L.R - 1);
        Pw[k] = ld4(tab + (size_t)reinterpret_cast<const int*>(rec)[n] * dv);
        Pr[k] = ld4(tab + (size_t)reinterpret_cast<const int*>(rec + L.off_rslot)[m] * dv);
    }
}

template <typename VT, int SW, int PD, int K, bool SAVE>
struct FwdCtx {
    const unsigned char* rring;
    const unsigned char* vring;
    float* fring;
    float* tab;       // this lane's columns of row 0 of the stream's table
    float* ystream;   // y of the stream, this lane's columns
    float* sstream;   // saved of the stream, this lane's columns
    FwdRec L;
    int dv, W, R, rg, cq;
    bool colok;
};

// One token of the recurrence for this lane's rows and columns.
template <typename VT, int SW, int PD, int K, bool SAVE, int NS>
__device__ __forceinline__ void fwd_token(const FwdCtx<VT, SW, PD, K, SAVE>& c, const v4f (&Pw)[K],
                                          const v4f (&Pr)[K], int t) {
    constexpr int CQ = SW / 4;
    constexpr int RG = SDM_WAVE / CQ;
    constexpr int VB = SW * (int)sizeof(VT);
    const FwdRec& L = c.L;
    const unsigned char* rec = c.rring + (t & (NS - 1)) * L.bytes;
    const float al = reinterpret_cast<const float*>(rec + L.off_ab)[0];
    const float be = reinterpret_cast<const float*>(rec + L.off_ab)[1];
    const short* lk = reinterpret_cast<const short*>(rec + L.off_link);

    // write rows: pre-write row (from the ring if a token still in flight wrote
    // it), decay, read-back sum
    v4f D[K];
    float kap[K];
    v4f up = v4zero();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = c.rg + RG * k;
        const bool rok = n < c.W;
        const int nn = rok ? n : 0;
        const int l = lk[nn];
        const int fidx = l >= 0 ? (((t - (l >> 8)) & (PD - 1)) * c.W + min(l & 255, c.W - 1)) : 0;
        const v4f f = ld4(c.fring + fidx * SW + c.cq * 4);
        v4f P = v4sel(l >= 0, f, Pw[k]);
        P = v4sel(rok, P, v4zero());
        kap[k] = rok ? reinterpret_cast<const float*>(rec + L.off_wval)[nn] : 0.f;
        if (SAVE && rok && c.colok) st4(c.sstream + ((size_t)t * c.W + n) * c.dv, P);
        D[k] = al * P;
        up = v4fma(kap[k], D[k], up);
    }
#pragma unroll
    for (int m = CQ; m < SDM_WAVE; m <<= 1) up += v4shfl_xor(up, m);
    const v4f vv = ld4v(reinterpret_cast<const VT*>(c.vring + (t & (NS - 1)) * VB) + c.cq * 4);
    const v4f e = be * (vv - up);
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = c.rg + RG * k;
        if (n < c.W) {
            const v4f nw = v4fma(kap[k], e, D[k]);
            st4(c.fring + ((t & (PD - 1)) * c.W + n) * SW + c.cq * 4, nw);
            if (c.colok) st4(c.tab + (size_t)reinterpret_cast<const int*>(rec)[n] * c.dv, nw);
        }
    }
    // read rows on the post-write memory
    v4f yp = v4zero();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int m = c.rg + RG * k;
        const bool rok = m < c.R;
        const int mm = rok ? m : 0;
        const int l = lk[c.W + mm];
        const int fidx = l >= 0 ? (((t - (l >> 8)) & (PD - 1)) * c.W + min(l & 255, c.W - 1)) : 0;
        const v4f f = ld4(c.fring + fidx * SW + c.cq * 4);
        const v4f P = v4sel(l >= 0, f, Pr[k]);
        const float rho = rok ? reinterpret_cast<const float*>(rec + L.off_rval)[mm] : 0.f;
        yp = v4fma(rho, P, yp);
    }
#pragma unroll
    for (int m = CQ; m < SDM_WAVE; m <<= 1) yp += v4shfl_xor(yp, m);
    if (c.rg == 0 && c.colok) st4(c.ystream + (size_t)t * c.dv, yp);
}

template <typename VT, int SW, int PD, int K, int NR, bool SAVE>
__global__ __launch_bounds__(MAX_WPB * SDM_WAVE) void scan_fwd_kernel(
    const unsigned char* __restrict__ recs, const VT* __restrict__ v, float* __restrict__ mem,
    float* __restrict__ y, float* __restrict__ saved, int T, int tb, int te, int dv, int W, int R,
    int64_t N, int n_slices, int lds_per_wave) {
    // tokens [tb, te) of each stream (tb a multiple of PD); layout strides use T
    constexpr int CQ = SW / 4;           // lanes per row slice (16 bytes each)
    constexpr int RG = SDM_WAVE / CQ;    // rows per load instruction
    constexpr int LEAD = stage_lead<PD>();
    constexpr int NS = stage_slots<PD>();
    constexpr int VB = SW * (int)sizeof(VT);
    static_assert(PD % G == 0, "prefetch depth must be a multiple of the staging block");
    static_assert(NS > LEAD && NS > PD, "record ring too small");

    const int lane = lane_id();
    const int wave = threadIdx.x / SDM_WAVE;
    const int wpb = blockDim.x / SDM_WAVE;
    int group, stream;
    scan_wg_coords<false>((n_slices + wpb - 1) / wpb, group, stream);
    const int slice = group * wpb + wave;
    if (slice >= n_slices) return;

    FwdCtx<VT, SW, PD, K, SAVE> c;
    c.L = fwd_rec_layout(W, R);
    c.dv = dv;
    c.W = W;
    c.R = R;
    c.rg = lane / CQ;
    c.cq = lane % CQ;
    const int col_raw = slice * SW + c.cq * 4;
    c.colok = col_raw < dv;
    const int col = c.colok ? col_raw : dv - 4;   // loads stay in bounds; results unused

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* rring = smem + (size_t)wave * lds_per_wave;   // NS records
    unsigned char* vring = rring + NS * c.L.bytes;               // NS v slices
    c.rring = rring;
    c.vring = vring;
    c.fring = reinterpret_cast<float*>(vring + NS * VB);         // [PD][W][SW] written rows
    c.tab = mem + (size_t)stream * N * dv + col;
    c.ystream = y + (size_t)stream * T * dv + col;
    c.sstream = SAVE ? saved + (size_t)stream * T * W * dv + col : nullptr;

    const unsigned char* srec = recs + (size_t)stream * T * c.L.bytes;
    const VT* sv = v + (size_t)stream * T * dv + slice * SW;

    u4v st[NR];
    u2v stv;
    v4f Pw[PD][K], Pr[PD][K];

    // ---- prologue: records of tokens [tb, tb+LEAD-G) in LDS, the next block in
    //      registers, rows of tokens [tb, tb+PD) in flight ----
    for (int u0 = tb; u0 < tb + LEAD - G; u0 += G) {
        stage_load<VT, SW, NR>(st, stv, srec, sv, u0, te, dv, slice, c.L.bytes, lane);
        stage_store<VT, SW, NS, NR>(st, stv, rring, vring, u0, c.L.bytes, lane);
    }
    stage_load<VT, SW, NR>(st, stv, srec, sv, tb + LEAD - G, te, dv, slice, c.L.bytes, lane);
#pragma unroll
    for (int j = 0; j < PD; ++j)
        issue_rows<K, RG, NS>(Pw[j], Pr[j], rring, c.L, c.tab, min(tb + j, te - 1), dv, c.rg);

    // ---- main loop over whole blocks of PD tokens; buffer j holds token t0 + j ----
    const int Tfull = te - (te - tb) % PD;
    for (int t0 = tb; t0 < Tfull; t0 += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            const int t = t0 + j;
            if (j % G == 0) {
                stage_store<VT, SW, NS, NR>(st, stv, rring, vring, t + LEAD - G, c.L.bytes, lane);
                stage_load<VT, SW, NR>(st, stv, srec, sv, t + LEAD, te, dv, slice, c.L.bytes, lane);
            }
            fwd_token<VT, SW, PD, K, SAVE, NS>(c, Pw[j], Pr[j], t);
            issue_rows<K, RG, NS>(Pw[j], Pr[j], rring, c.L, c.tab, min(t + PD, te - 1), dv, c.rg);
        }
    }
    // ---- tail: fewer than PD tokens, all rows already in flight ----
#pragma unroll
    for (int j = 0; j < PD; ++j) {
        const int t = Tfull + j;
        if (t < te) fwd_token<VT, SW, PD, K, SAVE, NS>(c, Pw[j], Pr[j], t);
    }
}

constexpr int FWD_PD = SDM_FWD_PD;

// Staging registers per lane (16 bytes each) for a block of G records: enough
// for every record of a shape with max(W, R) <= K RG, whose record takes at
// most 20 K RG + 8 bytes rounded up to 16.
template <int SW>
constexpr int nr_for_k(int K) {
    constexpr int RG = SDM_WAVE / (SW / 4);
    return (G * ((20 * K * RG + 8 + 15) / 16 * 16) + SDM_WAVE * 16 - 1) / (SDM_WAVE * 16);
}

struct FwdPlan {
    int SW, K, NR, lds_per_wave, wpb, n_slices;
};

// Launch geometry of the forward scan with SW columns per wave; false if the
// shape cannot be run.
template <int SW>
bool fwd_plan_sw(int W, int R, int dv, int in_dtype, FwdPlan* p) {
    constexpr int RG = SDM_WAVE / (SW / 4);
    const int need = (std::max(W, R) + RG - 1) / RG;
    if (need > (SW == 16 ? 4 : 2)) return false;
    p->SW = SW;
    p->K = need <= 1 ? 1 : (need <= 2 ? 2 : 4);
    p->NR = nr_for_k<SW>(p->K);
    const FwdRec L = fwd_rec_layout(W, R);
    if (G * L.bytes > p->NR * SDM_WAVE * 16) return false;
    const int vbytes = in_dtype == SDM_DT_BF16 ? 2 : 4;
    constexpr int NS = stage_slots<FWD_PD>();
    p->lds_per_wave = NS * L.bytes + NS * SW * vbytes + FWD_PD * W * SW * 4;
    if (p->lds_per_wave > LDS_LIMIT) return false;
    p->n_slices = (dv + SW - 1) / SW;
    p->wpb = std::min(std::min(MAX_WPB, p->n_slices), LDS_LIMIT / p->lds_per_wave);
    return true;
}

// 16 columns per wave when that already gives every SIMD a wave, else 8
// (twice the waves, half the columns each), unless a width is forced.
bool fwd_plan(int S, int W, int R, int dv, int in_dtype, FwdPlan* p) {
    const int forced = sdm_scan_slice_width();
    if (forced == 16 || (forced == 0 && (int64_t)S * ((dv + 15) / 16) >= sdm_device_simds()))
        return fwd_plan_sw<16>(W, R, dv, in_dtype, p);
    return fwd_plan_sw<8>(W, R, dv, in_dtype, p);
}

template <typename VT, int SW, int K, bool SAVE>
hipError_t launch_fwd_k(const ScanFwdArgs& a, const FwdPlan& p, hipStream_t st) {
    constexpr int NR = nr_for_k<SW>(K);
    const int S = a.B * a.H;
    dim3 grid((p.n_slices + p.wpb - 1) / p.wpb * S);   // order: scan_wg_coords
    const size_t sm = (size_t)p.lds_per_wave * p.wpb;
    auto kfn = scan_fwd_kernel<VT, SW, FWD_PD, K, NR, SAVE>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, grid, dim3(p.wpb * SDM_WAVE), sm, st,
                       a.ws + SDM_WS_HEADER, static_cast<const VT*>(a.v), a.mem, a.y, a.saved, a.T,
                       a.tb, a.te, a.dv, a.W, a.R, a.N, p.n_slices, p.lds_per_wave);
    return hipGetLastError();
}

template <typename VT, bool SAVE>
hipError_t launch_fwd_kk(const ScanFwdArgs& a, const FwdPlan& p, hipStream_t st) {
    if (p.SW == 8) {
        if (p.K == 1) return launch_fwd_k<VT, 8, 1, SAVE>(a, p, st);
        return launch_fwd_k<VT, 8, 2, SAVE>(a, p, st);
    }
    if (p.K == 1) return launch_fwd_k<VT, 16, 1, SAVE>(a, p, st);
    if (p.K == 2) return launch_fwd_k<VT, 16, 2, SAVE>(a, p, st);
    return launch_fwd_k<VT, 16, 4, SAVE>(a, p, st);
}

}  // namespace

size_t sdm_fwd_ws_bytes(int B, int H, int T, int W, int R) {
    return SDM_WS_HEADER + (size_t)B * H * T * fwd_rec_layout(W, R).bytes;
}

bool sdm_fwd_plan_ok(int W, int R, int dv, int in_dtype) {
    FwdPlan p;   // the 16-column plan fits whenever the 8-column one does
    return fwd_plan_sw<16>(W, R, dv, in_dtype, &p) && fwd_plan_sw<8>(W, R, dv, in_dtype, &p);
}

hipError_t sdm_launch_fwd_prep_range(const ScanFwdArgs& a, hipStream_t st) {
    SdmProfScope ps(SDM_K_FWD_PREP, st);
    return sdm_launch_fwd_prep<FWD_PD>(a, st);
}

hipError_t sdm_launch_fwd_scan_range(const ScanFwdArgs& a, hipStream_t st) {
    FwdPlan p;
    if (!fwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &p)) return hipErrorInvalidConfiguration;
    const bool save = a.saved != nullptr;
    SdmProfScope ps(SDM_K_FWD_SCAN, st);
    if (a.in_dtype == SDM_DT_BF16)
        return save ? launch_fwd_kk<bf16_t, true>(a, p, st) : launch_fwd_kk<bf16_t, false>(a, p, st);
    return save ? launch_fwd_kk<float, true>(a, p, st) : launch_fwd_kk<float, false>(a, p, st);
}

hipError_t sdm_launch_scan_fwd(const ScanFwdArgs& a, hipStream_t st) {
    hipError_t e = sdm_launch_fwd_prep_range(a, st);
    if (e != hipSuccess) return e;
    return sdm_launch_fwd_scan_range(a, st);
}
