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
//    would be stale.  The prep kernel records, per row of either list, the
//    latest writer within that window; such rows are taken from an LDS ring
//    holding the last PD tokens' written rows.  Older writers stored before
//    the load was issued, in program order of the same wave, so the load
//    returns their value;
//  * read rows are taken at their value before the token, P: a read row the
//    token itself writes ends at alpha P + kappa_n e, so its record weight is
//    rho alpha and the token's record carries yc = sum of rho kappa_n over
//    such rows, and y = sum rho' P + yc e (Eqs. sdm-write, sdm-read);
//  * per-token records (slots, weights, links, gates) are staged in LDS in
//    blocks of G tokens, loaded L tokens ahead with 16-byte loads.
#include <algorithm>

#include "sdm_common.h"
#include "sdm_internal.h"
#include "sdm_reduce.h"
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
    // line kernel: y of the stream as a buffer (below 2 GiB), its row t at byte
    // offset t 4 d_v + 4 column
    __amdgpu_buffer_rsrc_t yrs;
    uint32_t dv4, ycol4;
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
        const int fidx = l >= 0 ? min(l, PD * c.W - 1) : 0;   // the writer's ring row
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
    // read rows on the post-write memory, y = sum rho' P + yc e: P the value
    // before the token (a row the token writes carries rho alpha as rho', and
    // its rho kappa in yc)
    v4f yp = v4zero();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int m = c.rg + RG * k;
        const bool rok = m < c.R;
        const int mm = rok ? m : 0;
        const int l = lk[c.W + mm];
        const int fidx = l >= 0 ? min(l, PD * c.W - 1) : 0;
        const v4f f = ld4(c.fring + fidx * SW + c.cq * 4);
        const v4f P = v4sel(l >= 0, f, Pr[k]);
        const float rho = rok ? reinterpret_cast<const float*>(rec + L.off_rval)[mm] : 0.f;
        yp = v4fma(rho, P, yp);
    }
#pragma unroll
    for (int m = CQ; m < SDM_WAVE; m <<= 1) yp += v4shfl_xor(yp, m);
    const float yc = reinterpret_cast<const float*>(rec + L.off_ab)[2];
    if (c.rg == 0 && c.colok) st4(c.ystream + (size_t)t * c.dv, v4fma(yc, e, yp));
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
    // the block staged at step t (tokens t+LEAD-G .. t+LEAD-1) reuses only slots of
    // tokens already done, while tokens t .. t+LEAD-G-1 stay: NS >= LEAD suffices
    static_assert(NS >= LEAD && NS >= PD, "record ring too small");

    __builtin_amdgcn_s_setprio(3);   // as in scan_fwd_line_kernel
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

// ---------------------------------------------------------------------------
// Line-cooperative variant (W = R = FR, 32 or 64; d_v a multiple of 4 SW).
//
// The four waves of a workgroup are four adjacent SW-column slices of one
// stream (4 SW columns: a 128-byte line of every table row at SW = 8, two at
// SW = 16).  Moving only its own SW columns of each row, a wave touches a
// line in pieces at times of its own and the rows are served more slowly
// than when whole lines move together, so table rows go through LDS: each
// wave loads and stores FR / 4 of a token's FR rows over all 4 SW columns, and the
// waves exchange their pieces in LDS, with two workgroup barriers per token.
// The recurrence (links, the written-row ring, the per-token arithmetic) is
// that of scan_fwd_kernel, per wave and slice.
//
// Per token t (B1, B2 workgroup barriers):
//   S1  this wave's rows of token t (loaded earlier) -> LDS row buffer
//   B1
//   S2  row loads of token t + PD - 1
//   S3  each wave computes its pieces; written rows (and, when saving, the
//       pre-write rows) -> LDS staging buffer; y of its columns -> HBM
//   B2
//   S4  each wave stores FR / 4 staged rows as whole lines
// A load issued in S2 sees the stores of tokens <= t - 1 (every wave stored
// those before B1); the tokens t .. t + PD - 2 it cannot see are the PD - 1
// writers the prep kernel links to the ring, as for the per-wave kernel.
// One ring of records serves the four waves (they read the same records),
// which keeps LDS low enough for an addressing workgroup to share the CU.
constexpr int FLW = 4;       // waves (slices) per workgroup
template <int SW>
__host__ __device__ constexpr int frow_bytes() { return 20 * SW; }   // 16 SW of line + 4 SW of padding
template <int SW, int FR>
constexpr int fline_shared_bytes(bool save, int ns, int rec_bytes) {
    return ns * rec_bytes + (2 + (save ? 2 : 1)) * FR * frow_bytes<SW>();
}

template <int SW, int FR>
__device__ __forceinline__ v4f fl_ld(const unsigned char* base, int a, int r, int q) {
    return *reinterpret_cast<const v4f*>(base + (a * FR + r) * frow_bytes<SW>() + q * 16);
}
template <int SW, int FR>
__device__ __forceinline__ void fl_st(unsigned char* base, int a, int r, int q, v4f v) {
    *reinterpret_cast<v4f*>(base + (a * FR + r) * frow_bytes<SW>() + q * 16) = v;
}

// Rows per wave in line layout: instruction i covers rows (FR / 4) w + LRI i + lane / LQ.
template <int SW, int FR>
struct FLine {
    static constexpr int LQ = SW;            // 16-byte quads per staged row (4 SW columns)
    static constexpr int LRI = SDM_WAVE / LQ;
    static constexpr int NLI = FR / FLW / LRI;
    v4f Pw[NLI], Pr[NLI];
};

template <int SW>
struct FLinePtrs {
    float* tab;        // the stream's table at this lane's line columns
    float* sv;         // the stream's saved rows, same columns
    int r0, lq;        // first line row of this lane, quad within the row
    // The table rows through buffer instructions: the stream's table (below
    // 2 GiB, checked on the host) as the descriptor's base, a row's byte
    // offset slot * 4 d_v + 4 column in one 32-bit register (one 24-bit
    // multiply-add per row instead of 64-bit address arithmetic).
    __amdgpu_buffer_rsrc_t trs;
    uint32_t dv4, lc4;
};

template <int SW>
__device__ __forceinline__ uint32_t fl_row_off(const FLinePtrs<SW>& p, int slot) {
    return __umul24((uint32_t)slot, p.dv4) + p.lc4;
}
template <int SW>
__device__ __forceinline__ v4f fl_tab_ld(const FLinePtrs<SW>& p, int slot) {
    return __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(p.trs, (int)fl_row_off(p, slot), 0, 0));
}
template <int SW>
__device__ __forceinline__ void fl_tab_st(const FLinePtrs<SW>& p, int slot, v4f v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), p.trs, (int)fl_row_off(p, slot), 0, 0);
}

// Staging of G records, shared by the workgroup: wave w moves 16-byte chunks
// w 64 + lane + 256 j, j < NC (NC chunks per lane cover G records up to NC 4
// KB); v slices per wave.
template <typename VT, int SW, int NC>
__device__ __forceinline__ void fl_stage_load(u4v (&st)[NC], u2v& stv, const unsigned char* srec, const VT* sv,
                                              int u0, int te, int dv, int slice, int rec_bytes, int w,
                                              int lane) {
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
    const int ub = min(u0, te - 1);
    const int cnt = min(G, te - ub);
    const u4v* src = reinterpret_cast<const u4v*>(srec + (size_t)ub * rec_bytes);
#pragma unroll
    for (int j = 0; j < NC; ++j)
        st[j] = src[min(w * SDM_WAVE + lane + j * FLW * SDM_WAVE, cnt * rec_bytes / 16 - 1)];
    const int tk = min(lane / ppt, cnt - 1);
    const int pc = min(lane % ppt, (dv - slice * SW) * (int)sizeof(VT) / 8 - 1);
    stv = *reinterpret_cast<const u2v*>(
        reinterpret_cast<const unsigned char*>(sv + (size_t)(ub + tk) * dv) + pc * 8);
}
template <typename VT, int SW, int NS, int NC>
__device__ __forceinline__ void fl_stage_store(const u4v (&st)[NC], u2v stv, unsigned char* rring,
                                               unsigned char* vring, int u0, int rec_bytes, int w, int lane) {
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
#pragma unroll
    for (int j = 0; j < NC; ++j) {
        const int c = w * SDM_WAVE + lane + j * FLW * SDM_WAVE;
        if (c < G * rec_bytes / 16) reinterpret_cast<u4v*>(rring + (u0 & (NS - 1)) * rec_bytes)[c] = st[j];
    }
    const int tk = lane / ppt, pc = lane % ppt;
    if (tk < G) *reinterpret_cast<u2v*>(vring + ((u0 + tk) & (NS - 1)) * VB + pc * 8) = stv;
}

template <int SW, int NS, int FR>
__device__ __forceinline__ void fl_issue(FLine<SW, FR>& b, const unsigned char* rring, const FwdRec& L,
                                         const FLinePtrs<SW>& p, int u, int dv) {
    const unsigned char* rec = rring + (u & (NS - 1)) * L.bytes;
#pragma unroll
    for (int i = 0; i < FLine<SW, FR>::NLI; ++i) {
        const int r = p.r0 + FLine<SW, FR>::LRI * i;
        b.Pw[i] = fl_tab_ld(p, reinterpret_cast<const int*>(rec)[r]);
        b.Pr[i] = fl_tab_ld(p, reinterpret_cast<const int*>(rec + L.off_rslot)[r]);
    }
}

// One token on this wave's pieces (rows rg + RG k, columns 4 cq.. of slice w).
template <typename VT, int SW, int PD, bool SAVE, int NS, int FR>
__device__ __forceinline__ void fwd_token_line(const FwdCtx<VT, SW, PD, 2, SAVE>& c, const unsigned char* lb,
                                               unsigned char* sb, int t, int w) {
    using namespace sdm_reduce;
    constexpr int CQ = SW / 4;
    constexpr int RG = SDM_WAVE / CQ;
    constexpr int K = FR / RG;
    constexpr int VB = SW * (int)sizeof(VT);
    const FwdRec& L = c.L;
    const int q = w * CQ + c.cq;
    const unsigned char* rec = c.rring + (t & (NS - 1)) * L.bytes;
    const float al = reinterpret_cast<const float*>(rec + L.off_ab)[0];
    const float be = reinterpret_cast<const float*>(rec + L.off_ab)[1];
    const short* lk = reinterpret_cast<const short*>(rec + L.off_link);

    // pre-write value of write entry n: a ring row if a token still in flight
    // wrote it, else the row loaded from HBM
    static_assert((PD * FR & (PD * FR - 1)) == 0, "ring rows a power of two");
    auto pre_write = [&](int n) -> v4f {
        const int l = lk[n];
        const int fidx = l & (PD * FR - 1);   // the writer's ring row (no link: any row, unused)
        return v4sel(l >= 0, ld4(c.fring + fidx * SW + c.cq * 4), fl_ld<SW, FR>(lb, 0, n, q));
    };
    v4f D[K];
    float kap[K];
    v4f up = v4zero();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = c.rg + RG * k;
        const v4f P = pre_write(n);
        kap[k] = reinterpret_cast<const float*>(rec + L.off_wval)[n];
        if (SAVE) fl_st<SW, FR>(sb, 1, n, q, P);
        D[k] = al * P;
        up = v4fma(kap[k], D[k], up);
    }
    // read rows on the post-write memory, before the write: y = sum rho' P +
    // yc e, P the row's value before the token (a row the token writes carries
    // rho alpha as rho', and its rho kappa in the record's yc)
    v4f yp = v4zero();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int m = c.rg + RG * k;
        const int l = lk[FR + m];
        const float rho = reinterpret_cast<const float*>(rec + L.off_rval)[m];
        const int fidx = l & (PD * FR - 1);
        yp = v4fma(rho, v4sel(l >= 0, ld4(c.fring + fidx * SW + c.cq * 4), fl_ld<SW, FR>(lb, 1, m, q)), yp);
    }
    rows_allreduce8<CQ>(up, yp);
    const float yc = reinterpret_cast<const float*>(rec + L.off_ab)[2];
    const v4f vv = ld4v(reinterpret_cast<const VT*>(c.vring + (t & (NS - 1)) * VB) + c.cq * 4);
    const v4f e = be * (vv - up);
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = c.rg + RG * k;
        const v4f nw = v4fma(kap[k], e, D[k]);
        st4(c.fring + ((t & (PD - 1)) * FR + n) * SW + c.cq * 4, nw);
        fl_st<SW, FR>(sb, 0, n, q, nw);
    }
    if (c.rg == 0) {
        typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v4fma(yc, e, yp)), c.yrs,
                                               (int)(__umul24((uint32_t)t, c.dv4) + c.ycol4), 0, 0);
    }
}

template <typename VT, int SW, int PD, bool SAVE, int NS, int FR>
__device__ __forceinline__ void fl_step(const FwdCtx<VT, SW, PD, 2, SAVE>& c, const FLinePtrs<SW>& p,
                                        unsigned char* lb, unsigned char* sb, const FLine<SW, FR>& cur,
                                        FLine<SW, FR>& nxt, int t, int te, int w, bool issue) {
    constexpr int NLI = FLine<SW, FR>::NLI, LRI = FLine<SW, FR>::LRI;
    const FwdRec& L = c.L;
    int wslot[NLI];
    const unsigned char* rec = c.rring + (t & (NS - 1)) * L.bytes;
#pragma unroll
    for (int i = 0; i < NLI; ++i) wslot[i] = reinterpret_cast<const int*>(rec)[p.r0 + LRI * i];
#pragma unroll
    for (int i = 0; i < NLI; ++i) {
        fl_st<SW, FR>(lb, 0, p.r0 + LRI * i, p.lq, cur.Pw[i]);
        fl_st<SW, FR>(lb, 1, p.r0 + LRI * i, p.lq, cur.Pr[i]);
    }
    __syncthreads();
    // every wave stored token t - 1 before the barrier: the loads may go now
    if (issue) fl_issue<SW, NS, FR>(nxt, c.rring, L, p, min(t + PD - 1, te - 1), c.dv);
    fwd_token_line<VT, SW, PD, SAVE, NS, FR>(c, lb, sb, t, w);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NLI; ++i) {
        const int r = p.r0 + LRI * i;
        fl_tab_st(p, wslot[i], fl_ld<SW, FR>(sb, 0, r, p.lq));
        if (SAVE) st4(p.sv + ((size_t)t * FR + r) * c.dv, fl_ld<SW, FR>(sb, 1, r, p.lq));
    }
}

template <typename VT, int SW, int PD, bool SAVE, int FR>
__global__ __launch_bounds__(FLW * SDM_WAVE) void scan_fwd_line_kernel(
    const unsigned char* __restrict__ recs, const VT* __restrict__ v, float* __restrict__ mem,
    float* __restrict__ y, float* __restrict__ saved, int T, int tb, int te, int dv, int64_t N,
    int n_slices, int per_wave_lds) {
    constexpr int CQ = SW / 4;
    constexpr int LEAD = stage_lead<PD>();
    constexpr int NS = stage_slots<PD>();
    constexpr int VB = SW * (int)sizeof(VT);
    static_assert(PD % G == 0, "prefetch depth must be a multiple of the staging block");
    // the block staged at step t (tokens t+LEAD-G .. t+LEAD-1) reuses only slots of
    // tokens already done, while tokens t .. t+LEAD-G-1 stay: NS >= LEAD suffices
    static_assert(NS >= LEAD && NS >= PD, "record ring too small");
    static_assert(FLine<SW, FR>::NLI * FLine<SW, FR>::LRI * FLW == FR, "FR / 4 rows per wave");
    // records of G tokens in NC 16-byte chunks per lane of the workgroup
    constexpr int NC = (G * ((20 * FR + 12 + 15) / 16 * 16) + FLW * SDM_WAVE * 16 - 1) / (FLW * SDM_WAVE * 16);

    // In the pipelined forward the next stage's addressing and records share the
    // CUs; the scan waves are latency-bound and go first at each issue slot
    // (wave priority, not a queue priority), the others fill the gaps.
    __builtin_amdgcn_s_setprio(3);
    const int lane = lane_id();
    const int w = threadIdx.x / SDM_WAVE;
    int group, stream;
    scan_wg_coords<false>(n_slices / FLW, group, stream);
    const int slice = group * FLW + w;   // n_slices is a multiple of FLW: every wave exists

    FwdCtx<VT, SW, PD, 2, SAVE> c;
    c.L = fwd_rec_layout(FR, FR);
    c.dv = dv;
    c.W = FR;
    c.R = FR;
    c.rg = lane / CQ;
    c.cq = lane % CQ;
    c.colok = true;
    const int col = slice * SW + c.cq * 4;

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* rring = smem;                                   // NS records, shared
    unsigned char* lb = rring + NS * c.L.bytes;                    // [2][32] rows
    unsigned char* sb = lb + 2 * FR * frow_bytes<SW>();         // [1 or 2][FR] rows
    unsigned char* own = sb + (SAVE ? 2 : 1) * FR * frow_bytes<SW>() + (size_t)w * per_wave_lds;
    unsigned char* vring = own;                                    // NS v slices of this wave
    c.rring = rring;
    c.vring = vring;
    c.fring = reinterpret_cast<float*>(vring + NS * VB);           // [PD][32][SW] written rows
    c.tab = mem + (size_t)stream * N * dv + col;
    c.ystream = y + (size_t)stream * T * dv + col;
    c.yrs = __builtin_amdgcn_make_buffer_rsrc(y + (size_t)stream * T * dv, 0, (int)((size_t)T * dv * 4), 0x00020000);
    c.dv4 = (uint32_t)dv * 4;
    c.ycol4 = (uint32_t)col * 4;
    c.sstream = nullptr;

    FLinePtrs<SW> p;
    p.r0 = FR / FLW * w + lane / FLine<SW, FR>::LQ;
    p.lq = lane % FLine<SW, FR>::LQ;
    const size_t lcol = (size_t)group * FLW * SW + p.lq * 4;
    p.tab = mem + (size_t)stream * N * dv + lcol;
    p.trs = __builtin_amdgcn_make_buffer_rsrc(mem + (size_t)stream * N * dv, 0, (int)((size_t)N * dv * 4),
                                              0x00020000);
    p.dv4 = (uint32_t)dv * 4;
    p.lc4 = (uint32_t)lcol * 4;
    p.sv = SAVE ? saved + (size_t)stream * T * FR * dv + lcol : nullptr;

    const unsigned char* srec = recs + (size_t)stream * T * c.L.bytes;
    const VT* sv = v + (size_t)stream * T * dv + slice * SW;
    u4v st[NC];
    u2v stv;
    FLine<SW, FR> buf[PD];

    for (int u0 = tb; u0 < tb + LEAD - G; u0 += G) {
        fl_stage_load<VT, SW, NC>(st, stv, srec, sv, u0, te, dv, slice, c.L.bytes, w, lane);
        fl_stage_store<VT, SW, NS, NC>(st, stv, rring, vring, u0, c.L.bytes, w, lane);
    }
    fl_stage_load<VT, SW, NC>(st, stv, srec, sv, tb + LEAD - G, te, dv, slice, c.L.bytes, w, lane);
    __syncthreads();   // records of the first tokens from every wave
#pragma unroll
    for (int j = 0; j < PD - 1; ++j) fl_issue<SW, NS, FR>(buf[j], rring, c.L, p, min(tb + j, te - 1), dv);

    // Token t = t0 + j uses buf[j]; its step loads token t + PD - 1 into
    // buf[(j + PD - 1) % PD], the buffer token t - 1 used.
    const int Tfull = te - (te - tb) % PD;
    for (int t0 = tb; t0 < Tfull; t0 += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            const int t = t0 + j;
            if (j % G == 0) {
                fl_stage_store<VT, SW, NS, NC>(st, stv, rring, vring, t + LEAD - G, c.L.bytes, w, lane);
                fl_stage_load<VT, SW, NC>(st, stv, srec, sv, t + LEAD, te, dv, slice, c.L.bytes, w, lane);
            }
            fl_step<VT, SW, PD, SAVE, NS, FR>(c, p, lb, sb, buf[j], buf[(j + PD - 1) % PD], t, te, w, true);
        }
    }
#pragma unroll
    for (int j = 0; j < PD; ++j) {
        const int t = Tfull + j;
        if (t < te) fl_step<VT, SW, PD, SAVE, NS, FR>(c, p, lb, sb, buf[j], buf[(j + PD - 1) % PD], t, te, w, false);
    }
}

constexpr int FWD_PD = SDM_FWD_PD;

// Staging registers per lane (16 bytes each) for a block of G records: enough
// for every record of a shape with max(W, R) <= K RG, whose record takes at
// most 20 K RG + 12 bytes rounded up to 16.
template <int SW>
constexpr int nr_for_k(int K) {
    constexpr int RG = SDM_WAVE / (SW / 4);
    return (G * ((20 * K * RG + 12 + 15) / 16 * 16) + SDM_WAVE * 16 - 1) / (SDM_WAVE * 16);
}

struct FwdPlan {
    int SW, K, NR, lds_per_wave, wpb, n_slices;
};

// Launch geometry of the forward scan with SW columns per wave; false if the
// shape cannot be run.
template <int SW>
bool fwd_plan_sw(int W, int R, int dv, int in_dtype, FwdPlan* p) {
    constexpr int RG = SDM_WAVE / (SW / 4);
    const int need = (std::max(W, R) + RG - 1) / RG;   // row passes: at most 4 (64 or 128 rows)
    if (need > 4) return false;
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

// 8 columns per wave, unless that would put 1.5 or more waves on every SIMD:
// then 16 (half the waves, twice the columns each), unless a width is forced.
// At two 8-column waves per SIMD the rows in flight outgrow the L2 and four
// waves sharing each 128-byte line fetch it more than once: measured, the
// per-wave scan at 1920 such waves fetched three times its bytes and ran at
// half the speed of 960 16-column waves.  The other width is taken when the
// chosen one cannot hold the shape (16 columns hold at most 64 rows).
//
// Except, when the width is automatic, for the line-cooperative kernel at
// W = R = 64: at 16 columns it holds 137-155 KB of a CU's 160 KB of LDS, so the
// addressing that sdm_forward runs beside the scan is left the CUs without a
// scan workgroup.  The 8-column line kernel takes half that LDS and moves whole
// lines, so the many-waves penalty above does not apply: at 16 streams with
// d_v = 960 it measured 10.3 ms per forward step against 10.7 ms (13.1 against
// 14.1 with the undo log).
bool fwd_plan(int S, int W, int R, int dv, int in_dtype, FwdPlan* p) {
    const int forced = sdm_scan_slice_width();
    const bool line64 = W == 64 && R == 64 && sdm_line_io_enabled() && dv % (FLW * 8) == 0;
    if (forced == 16 ||
        (forced == 0 && !line64 && 2 * (int64_t)S * ((dv + 7) / 8) >= 3 * (int64_t)sdm_device_simds()))
        return fwd_plan_sw<16>(W, R, dv, in_dtype, p) || fwd_plan_sw<8>(W, R, dv, in_dtype, p);
    return fwd_plan_sw<8>(W, R, dv, in_dtype, p) || fwd_plan_sw<16>(W, R, dv, in_dtype, p);
}

// LDS of the line-cooperative forward kernel (shared part, per-wave part).
template <int SW, int FR, int PD>
size_t fline_lds(bool save, int in_dtype, size_t* per_wave) {
    constexpr int NS = stage_slots<PD>();
    const int vbytes = in_dtype == SDM_DT_BF16 ? 2 : 4;
    *per_wave = (size_t)NS * SW * vbytes + (size_t)PD * FR * SW * 4;
    return (size_t)fline_shared_bytes<SW, FR>(save, NS, fwd_rec_layout(FR, FR).bytes) + FLW * *per_wave;
}

// The line-cooperative kernel's shape: W = R = FR, d_v a multiple of 4 SW
// (whole workgroups), and its LDS within the limit (at 64 rows, 16 columns
// and the undo log: 155 KB).
template <int SW, int FR, int PD>
bool fline_ok(const ScanFwdArgs& a, const FwdPlan& p, bool save, size_t* lds, size_t* per_wave) {
    if (!sdm_line_io_enabled() || a.W != FR || a.R != FR || a.dv % (FLW * SW) != 0 || p.n_slices % FLW != 0)
        return false;
    // the table rows' and y's 32-bit offsets (and the 24-bit multiplies: N, T < 2^24)
    if ((size_t)a.N * a.dv * 4 >= ((size_t)1 << 31) || a.N >= (1 << 24)) return false;
    if ((size_t)a.T * a.dv * 4 >= ((size_t)1 << 31) || a.T >= (1 << 24)) return false;
    *lds = fline_lds<SW, FR, PD>(save, a.in_dtype, per_wave);
    return *lds <= (size_t)LDS_LIMIT;
}

template <typename VT, int SW, bool SAVE, int FR, int PD>
hipError_t launch_fline(const ScanFwdArgs& a, const FwdPlan& p, size_t lds, size_t per_wave, hipStream_t st) {
    auto kl = scan_fwd_line_kernel<VT, SW, PD, SAVE, FR>;
    hipError_t e = hipFuncSetAttribute((const void*)kl, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kl, dim3(p.n_slices / FLW * (a.B * a.H)), dim3(FLW * SDM_WAVE), lds, st,
                       a.ws + SDM_WS_HEADER, static_cast<const VT*>(a.v), a.mem, a.y, a.saved, a.T, a.tb, a.te,
                       a.dv, a.N, p.n_slices, (int)per_wave);
    return hipGetLastError();
}

template <typename VT, int SW, int K, bool SAVE>
hipError_t launch_fwd_k(const ScanFwdArgs& a, const FwdPlan& p, int pd, hipStream_t st) {
    constexpr int NR = nr_for_k<SW>(K);
    const int S = a.B * a.H;
    size_t lds = 0, per_wave = 0;
    constexpr int FR = K * (SDM_WAVE / (SW / 4));   // rows the plan's K passes hold
    if constexpr (FR == 32 || FR == 64) {
        // the prefetch depth was chosen with the same plan (sdm_fwd_pd), so its LDS fits
        if (pd == 16 && fline_ok<SW, FR, 16>(a, p, SAVE, &lds, &per_wave))
            return launch_fline<VT, SW, SAVE, FR, 16>(a, p, lds, per_wave, st);
        if (pd == 8 && fline_ok<SW, FR, 8>(a, p, SAVE, &lds, &per_wave))
            return launch_fline<VT, SW, SAVE, FR, 8>(a, p, lds, per_wave, st);
        if (pd == FWD_PD && fline_ok<SW, FR, FWD_PD>(a, p, SAVE, &lds, &per_wave))
            return launch_fline<VT, SW, SAVE, FR, FWD_PD>(a, p, lds, per_wave, st);
    }
    if (pd != FWD_PD) return hipErrorInvalidConfiguration;   // the per-wave kernel links over FWD_PD tokens
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
hipError_t launch_fwd_kk(const ScanFwdArgs& a, const FwdPlan& p, int pd, hipStream_t st) {
    if (p.SW == 8) {
        if (p.K == 1) return launch_fwd_k<VT, 8, 1, SAVE>(a, p, pd, st);
        if (p.K == 2) return launch_fwd_k<VT, 8, 2, SAVE>(a, p, pd, st);
        return launch_fwd_k<VT, 8, 4, SAVE>(a, p, pd, st);
    }
    if (p.K == 1) return launch_fwd_k<VT, 16, 1, SAVE>(a, p, pd, st);
    if (p.K == 2) return launch_fwd_k<VT, 16, 2, SAVE>(a, p, pd, st);
    return launch_fwd_k<VT, 16, 4, SAVE>(a, p, pd, st);
}

// Whether the line kernel of this plan can run at prefetch depth PD.
template <int PD>
bool fline_fits(const ScanFwdArgs& a, const FwdPlan& p) {
    size_t lds, pw;
    const bool save = a.saved != nullptr;
    if (p.SW == 8) {
        if (a.W == 32) return fline_ok<8, 32, PD>(a, p, save, &lds, &pw);
        if (a.W == 64) return fline_ok<8, 64, PD>(a, p, save, &lds, &pw);
    } else {
        if (a.W == 32) return fline_ok<16, 32, PD>(a, p, save, &lds, &pw);
        if (a.W == 64) return fline_ok<16, 64, PD>(a, p, save, &lds, &pw);
    }
    return false;
}

}  // namespace

// Prefetch depth of the forward scan for these arguments (the prep kernel
// links over the same window).  Four tokens, unless the line-cooperative
// kernel runs with fewer waves than the device has SIMDs: then each stream's
// step time is set by the latency of its row loads over the tokens in flight,
// and a deeper window (16, else 8, as LDS allows) keeps more rows in flight.
int sdm_fwd_pd(const ScanFwdArgs& a) {
    FwdPlan p;
    if (!fwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &p)) return FWD_PD;
    if (!fline_fits<FWD_PD>(a, p)) return FWD_PD;   // per-wave kernel
    const int forced = sdm_scan_prefetch();
    const int want =
        forced ? forced : ((int64_t)a.B * a.H * p.n_slices < sdm_device_simds() ? SDM_FWD_PD_DEEP : FWD_PD);
    if (want >= 16 && fline_fits<16>(a, p)) return 16;
    if (want >= 8 && fline_fits<8>(a, p)) return 8;
    return FWD_PD;
}

size_t sdm_fwd_ws_bytes(int B, int H, int T, int W, int R) {
    return SDM_WS_HEADER + (size_t)B * H * T * fwd_rec_layout(W, R).bytes;
}

bool sdm_fwd_plan_ok(int W, int R, int dv, int in_dtype) {
    FwdPlan p;   // every width fwd_plan may choose falls back to the 8-column plan
    return fwd_plan_sw<8>(W, R, dv, in_dtype, &p);
}

hipError_t sdm_launch_fwd_prep_range(const ScanFwdArgs& a, hipStream_t st) {
    SdmProfScope ps(SDM_K_FWD_PREP, st);
    switch (sdm_fwd_pd(a)) {
        case 16: return sdm_launch_fwd_prep<16>(a, st);
        case 8: return sdm_launch_fwd_prep<8>(a, st);
        default: return sdm_launch_fwd_prep<FWD_PD>(a, st);
    }
}

hipError_t sdm_launch_fwd_scan_range(const ScanFwdArgs& a, hipStream_t st) {
    FwdPlan p;
    if (!fwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &p)) return hipErrorInvalidConfiguration;
    const bool save = a.saved != nullptr;
    const int pd = sdm_fwd_pd(a);
    SdmProfScope ps(SDM_K_FWD_SCAN, st);
    if (a.in_dtype == SDM_DT_BF16)
        return save ? launch_fwd_kk<bf16_t, true>(a, p, pd, st) : launch_fwd_kk<bf16_t, false>(a, p, pd, st);
    return save ? launch_fwd_kk<float, true>(a, p, pd, st) : launch_fwd_kk<float, false>(a, p, pd, st);
}

namespace {
template <int SW, int K>
size_t fwd_lds_k(const ScanFwdArgs& a, const FwdPlan& p, int pd, bool save) {
    constexpr int FR = K * (SDM_WAVE / (SW / 4));
    size_t lds = 0, per_wave = 0;
    if constexpr (FR == 32 || FR == 64) {
        if (pd == 16 && fline_ok<SW, FR, 16>(a, p, save, &lds, &per_wave)) return lds;
        if (pd == 8 && fline_ok<SW, FR, 8>(a, p, save, &lds, &per_wave)) return lds;
        if (pd == FWD_PD && fline_ok<SW, FR, FWD_PD>(a, p, save, &lds, &per_wave)) return lds;
    }
    return (size_t)p.lds_per_wave * p.wpb;
}
}  // namespace

// LDS of one workgroup of the forward scan these arguments launch (the kernel
// and depth sdm_launch_fwd_scan_range picks).
size_t sdm_fwd_scan_lds(const ScanFwdArgs& a) {
    FwdPlan p;
    if (!fwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &p)) return 0;
    const int pd = sdm_fwd_pd(a);
    const bool save = a.saved != nullptr;
    if (p.SW == 8) {
        if (p.K == 1) return fwd_lds_k<8, 1>(a, p, pd, save);
        if (p.K == 2) return fwd_lds_k<8, 2>(a, p, pd, save);
        return fwd_lds_k<8, 4>(a, p, pd, save);
    }
    if (p.K == 1) return fwd_lds_k<16, 1>(a, p, pd, save);
    if (p.K == 2) return fwd_lds_k<16, 2>(a, p, pd, save);
    return fwd_lds_k<16, 4>(a, p, pd, save);
}

hipError_t sdm_launch_scan_fwd(const ScanFwdArgs& a, hipStream_t st) {
    hipError_t e = sdm_launch_fwd_prep_range(a, st);
    if (e != hipSuccess) return e;
    return sdm_launch_fwd_scan_range(a, st);
}
