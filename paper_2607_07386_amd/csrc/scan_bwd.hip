// Backward of the sparse gated-delta scan for gfx950.
//
// Reverse mode of the forward recurrence with the in-place + undo scheme of
// App. A.3: the forward left M_T in the table and saved, per token, the W
// pre-write rows P.  Going t = T-1 .. 0, each step reads M_t and the adjoint
// G on its slots, recomputes D = alpha P, u and e from P (the forward
// intermediates are not stored), updates G and undoes the write with P.
//
// As in the forward, one wave owns one (stream, column slice) for the whole
// sequence.  Rows are prefetched PD tokens ahead (in reverse order); a row
// that a token processed after the load was issued but before its use would
// have modified is taken from LDS rings of the last PD tokens' undo rows
// (for M) and adjoint rows (for G), as recorded by the prep kernel.
// Per-token scalars (dalpha, dbeta, weight gradients) are sums over all d_v
// columns: each slice writes its partial sums and a reduction kernel adds
// the slices.
#include <algorithm>

#include "sdm_common.h"
#include "sdm_internal.h"
#include "sdm_reduce.h"
#include "sdm.h"

namespace {

constexpr int G = 4;
constexpr int MAX_WPB = 4;
constexpr int LDS_LIMIT = 160 * 1024;

template <int PD>
__host__ __device__ constexpr int bstage_lead() {
    return ((G + PD + G - 1) / G) * G;
}
template <int PD>
__host__ __device__ constexpr int bstage_slots() {
    return bstage_lead<PD>() <= 8 ? 8 : (bstage_lead<PD>() <= 16 ? 16 : 32);
}

// Staging of the records (and v slices) of the G tokens [u1 - G + 1, u1] (clamped at lo,
// the first token of the range), the order the backward visits them in.  Loads are
// unconditional; indices past the valid range are clamped and the surplus is never stored.
template <typename VT, int SW, int NR>
__device__ __forceinline__ void bstage_load(u4v (&st)[NR], u2v& stv, const unsigned char* srec,
                                            const VT* sv, int u1, int lo, int dv, int slice, int rec_bytes,
                                            int lane) {
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
    const int ub1 = max(u1, lo);
    const int u0 = max(lo, ub1 - G + 1);
    const int cnt = ub1 - u0 + 1;
    const u4v* src = reinterpret_cast<const u4v*>(srec + (size_t)u0 * rec_bytes);
    const int last = cnt * rec_bytes / 16 - 1;
#pragma unroll
    for (int r = 0; r < NR; ++r) st[r] = src[min(r * SDM_WAVE + lane, last)];
    const int tk = min(lane / ppt, cnt - 1);
    const int pc = min(lane % ppt, (dv - slice * SW) * (int)sizeof(VT) / 8 - 1);
    stv = *reinterpret_cast<const u2v*>(
        reinterpret_cast<const unsigned char*>(sv + (size_t)(u0 + tk) * dv) + pc * 8);
}

template <typename VT, int SW, int NS, int NR>
__device__ __forceinline__ void bstage_store(const u4v (&st)[NR], u2v stv, unsigned char* rring,
                                             unsigned char* vring, int u1, int lo, int rec_bytes, int lane) {
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
    if (u1 < lo) return;
    const int u0 = max(lo, u1 - G + 1);
    const int cnt = u1 - u0 + 1;
    const int nchunk = cnt * rec_bytes / 16;   // <= NR * 64 (checked by the host plan)
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        const int c = r * SDM_WAVE + lane;
        if (c < nchunk) {
            const int tk = (c * 16) / rec_bytes;   // records are whole 16-byte chunks
            const int within = c * 16 - tk * rec_bytes;
            *reinterpret_cast<u4v*>(rring + ((u0 + tk) & (NS - 1)) * rec_bytes + within) = st[r];
        }
    }
    const int tk = lane / ppt, pc = lane % ppt;
    if (tk < cnt) *reinterpret_cast<u2v*>(vring + ((u0 + tk) & (NS - 1)) * VB + pc * 8) = stv;
}

template <int K>
struct BwdBuf {
    v4f Mr[K], Gr[K], Gw[K], Ps[K];
    v4f Dy;
};

struct BwdCtx {
    const unsigned char* rring;
    const unsigned char* vring;
    float* gring;     // [PD][R + W][SW]: adjoint rows after the token (read part, then write part)
    float* pring;     // [PD][W][SW]: undo rows of the token
    float* mtab;      // this lane's columns of row 0 of the stream's memory table
    float* gtab;      // same for the adjoint table
    const float* ssaved;  // saved rows of the stream, this lane's columns
    const float* sdy;     // dy of the stream, this lane's columns
    float* sdv;           // dv of the stream, this lane's columns
    float* spart;         // partial scalars of this (slice, stream)
    BwdRec L;
    int dv, W, R, rg, cq;
    bool colok;
};

template <int K, int RG, int NS>
__device__ __forceinline__ void bissue_rows(BwdBuf<K>& b, const BwdCtx& c, int u) {
    const unsigned char* rec = c.rring + (u & (NS - 1)) * c.L.bytes;
    b.Dy = ld4(c.sdy + (size_t)u * c.dv);
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int m = min(c.rg + RG * k, c.R - 1);
        const int n = min(c.rg + RG * k, c.W - 1);
        const size_t rs = (size_t)reinterpret_cast<const int*>(rec + c.L.off_rslot)[m] * c.dv;
        const size_t ws = (size_t)reinterpret_cast<const int*>(rec)[n] * c.dv;
        b.Mr[k] = ld4(c.mtab + rs);
        b.Gr[k] = ld4(c.gtab + rs);
        b.Gw[k] = ld4(c.gtab + ws);
        b.Ps[k] = ld4(c.ssaved + ((size_t)u * c.W + n) * c.dv);
    }
}

template <typename VT, int SW, int PD, int K, int NS>
__device__ __forceinline__ void bwd_token(const BwdCtx& c, const BwdBuf<K>& b, int t, int lane) {
    constexpr int CQ = SW / 4;
    constexpr int RG = SDM_WAVE / CQ;
    constexpr int VB = SW * (int)sizeof(VT);
    const BwdRec& L = c.L;
    const int RW = c.R + c.W;
    const unsigned char* rec = c.rring + (t & (NS - 1)) * L.bytes;
    const float al = reinterpret_cast<const float*>(rec + L.off_ab)[0];
    const float be = reinterpret_cast<const float*>(rec + L.off_ab)[1];
    const short* lm = reinterpret_cast<const short*>(rec + L.off_lm);
    const short* lgr = reinterpret_cast<const short*>(rec + L.off_lgr);
    const short* lgw = reinterpret_cast<const short*>(rec + L.off_lgw);
    const v4f yb = b.Dy;
    float* prow = c.spart + (size_t)t * (RW + 2);

    // ---- read adjoint: rbar_m = <dy, M_t[j_m]>, G[j_m] += rho_m dy ----
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int m = c.rg + RG * k;
        const bool rok = m < c.R;
        const int mm = rok ? m : 0;
        const int l1 = lm[mm];
        const int i1 = l1 >= 0 ? (((t + (l1 >> 8)) & (PD - 1)) * c.W + min(l1 & 255, c.W - 1)) : 0;
        const v4f Mv = v4sel(l1 >= 0, ld4(c.pring + i1 * SW + c.cq * 4), b.Mr[k]);
        float rb = c.colok ? v4dot(yb, Mv) : 0.f;
#pragma unroll
        for (int q = 1; q < CQ; q <<= 1) rb += xor_lane_f(rb, q);
        if (rok && c.cq == 0) prow[m] = rb;
        const int l2 = lgr[mm];
        const int i2 = l2 >= 0 ? (((t + (l2 >> 8)) & (PD - 1)) * RW + min(l2 & 255, RW - 1)) : 0;
        v4f g = v4sel(l2 >= 0, ld4(c.gring + i2 * SW + c.cq * 4), b.Gr[k]);
        const float rho = rok ? reinterpret_cast<const float*>(rec + L.off_rval)[mm] : 0.f;
        g = v4fma(rho, yb, g);
        if (rok) {
            st4(c.gring + ((t & (PD - 1)) * RW + m) * SW + c.cq * 4, g);
            if (c.colok) st4(c.gtab + (size_t)reinterpret_cast<const int*>(rec + L.off_rslot)[m] * c.dv, g);
        }
    }
    // ---- write adjoint ----
    v4f gn[K], D[K];
    float kap[K];
    v4f up = v4zero(), ebp = v4zero();
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = c.rg + RG * k;
        const bool rok = n < c.W;
        const int nn = rok ? n : 0;
        const int l = lgw[nn];
        const int ig = l >= 0 ? (((t + (l >> 8)) & (PD - 1)) * RW + min(l & 255, RW - 1)) : 0;
        gn[k] = v4sel(rok, v4sel(l >= 0, ld4(c.gring + ig * SW + c.cq * 4), b.Gw[k]), v4zero());
        D[k] = v4sel(rok, al * b.Ps[k], v4zero());
        kap[k] = rok ? reinterpret_cast<const float*>(rec + L.off_wval)[nn] : 0.f;
        up = v4fma(kap[k], D[k], up);
        ebp = v4fma(kap[k], gn[k], ebp);
    }
#pragma unroll
    for (int m = CQ; m < SDM_WAVE; m <<= 1) {
        up += v4shfl_xor(up, m);
        ebp += v4shfl_xor(ebp, m);
    }
    const v4f vv = ld4v(reinterpret_cast<const VT*>(c.vring + (t & (NS - 1)) * VB) + c.cq * 4);
    const v4f vmu = vv - up;
    const v4f e = be * vmu;
    if (c.rg == 0 && c.colok) st4(c.sdv + (size_t)t * c.dv, be * ebp);
    float bb = c.colok ? v4dot(ebp, vmu) : 0.f;
    float ab = 0.f;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int n = c.rg + RG * k;
        if (n < c.W) {
            float kb = c.colok ? (v4dot(gn[k], e) - be * v4dot(ebp, D[k])) : 0.f;
#pragma unroll
            for (int q = 1; q < CQ; q <<= 1) kb += xor_lane_f(kb, q);
            if (c.cq == 0) prow[c.R + n] = kb;
            const v4f Db = v4fma(-be * kap[k], ebp, gn[k]);
            if (c.colok) ab += v4dot(Db, b.Ps[k]);
            const v4f gnew = al * Db;
            st4(c.gring + ((t & (PD - 1)) * RW + c.R + n) * SW + c.cq * 4, gnew);
            st4(c.pring + ((t & (PD - 1)) * c.W + n) * SW + c.cq * 4, b.Ps[k]);
            if (c.colok) {
                const size_t ws = (size_t)reinterpret_cast<const int*>(rec)[n] * c.dv;
                st4(c.gtab + ws, gnew);
                st4(c.mtab + ws, b.Ps[k]);
            }
        }
    }
#pragma unroll
    for (int q = 1; q < CQ; q <<= 1) bb += xor_lane_f(bb, q);
    ab = wave_sum(ab);
    if (lane == 0) {
        prow[RW] = bb;
        prow[RW + 1] = ab;
    }
}

// Partial scalars per (slice, stream, t): [R] rbar, [W] kbar, dbeta, dalpha.
template <typename VT, int SW, int PD, int K, int NR>
__global__ __launch_bounds__(MAX_WPB * SDM_WAVE) void scan_bwd_kernel(
    const unsigned char* __restrict__ recs, const VT* __restrict__ v, float* __restrict__ mem,
    const float* __restrict__ saved, const float* __restrict__ dy, float* __restrict__ Gtab,
    float* __restrict__ dv_out, float* __restrict__ part, int T, int tb, int te, int dv, int W, int R,
    int64_t N, int n_slices, int S, int lds_per_wave) {
    // tokens te-1 down to tb of each stream (layout strides use T)
    constexpr int CQ = SW / 4;
    constexpr int RG = SDM_WAVE / CQ;
    constexpr int LEAD = bstage_lead<PD>();
    constexpr int NS = bstage_slots<PD>();
    constexpr int VB = SW * (int)sizeof(VT);
    // staging blocks of G tokens every G steps; the prefetch depth divides or is a multiple of G
    static_assert(PD % G == 0 || G % PD == 0, "prefetch depth and staging block");
    static_assert(NS >= LEAD && NS >= PD, "record ring too small");

    const int lane = lane_id();
    const int wave = threadIdx.x / SDM_WAVE;
    const int wpb = blockDim.x / SDM_WAVE;
    int group, stream;
    scan_wg_coords<true>((n_slices + wpb - 1) / wpb, group, stream);
    const int slice = group * wpb + wave;
    if (slice >= n_slices) return;

    BwdCtx c;
    c.L = bwd_rec_layout(W, R);
    c.dv = dv;
    c.W = W;
    c.R = R;
    c.rg = lane / CQ;
    c.cq = lane % CQ;
    const int col_raw = slice * SW + c.cq * 4;
    c.colok = col_raw < dv;
    const int col = c.colok ? col_raw : dv - 4;

    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* rring = smem + (size_t)wave * lds_per_wave;
    unsigned char* vring = rring + NS * c.L.bytes;
    c.rring = rring;
    c.vring = vring;
    c.gring = reinterpret_cast<float*>(vring + NS * VB);
    c.pring = c.gring + PD * (R + W) * SW;
    c.mtab = mem + (size_t)stream * N * dv + col;
    c.gtab = Gtab + (size_t)stream * N * dv + col;
    c.ssaved = saved + (size_t)stream * T * W * dv + col;
    c.sdy = dy + (size_t)stream * T * dv + col;
    c.sdv = dv_out + (size_t)stream * T * dv + col;
    c.spart = part + ((size_t)slice * S + stream) * T * (W + R + 2);

    const unsigned char* srec = recs + (size_t)stream * T * c.L.bytes;
    const VT* sv = v + (size_t)stream * T * dv + slice * SW;

    u4v st[NR];
    u2v stv;
    BwdBuf<K> buf[PD];

    // Step i processes token t = te-1-i.  Staging blocks are the G tokens
    // ending at te-1-i for i % G == 0.
    const int T1 = te - 1;
    for (int i0 = 0; i0 < LEAD - G; i0 += G) {
        bstage_load<VT, SW, NR>(st, stv, srec, sv, T1 - i0, tb, dv, slice, c.L.bytes, lane);
        bstage_store<VT, SW, NS, NR>(st, stv, rring, vring, T1 - i0, tb, c.L.bytes, lane);
    }
    bstage_load<VT, SW, NR>(st, stv, srec, sv, T1 - (LEAD - G), tb, dv, slice, c.L.bytes, lane);
#pragma unroll
    for (int j = 0; j < PD; ++j) bissue_rows<K, RG, NS>(buf[j], c, max(T1 - j, tb));

    const int n = te - tb;
    const int nfull = n - n % PD;
    for (int i0 = 0; i0 < nfull; i0 += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            const int t = T1 - (i0 + j);
            if ((i0 + j) % G == 0) {
                bstage_store<VT, SW, NS, NR>(st, stv, rring, vring, t - (LEAD - G), tb, c.L.bytes, lane);
                bstage_load<VT, SW, NR>(st, stv, srec, sv, t - LEAD, tb, dv, slice, c.L.bytes, lane);
            }
            bwd_token<VT, SW, PD, K, NS>(c, buf[j], t, lane);
            bissue_rows<K, RG, NS>(buf[j], c, max(t - PD, tb));
        }
    }
#pragma unroll
    for (int j = 0; j < PD; ++j) {
        const int i = nfull + j;
        if (i < n) bwd_token<VT, SW, PD, K, NS>(c, buf[j], T1 - i, lane);
    }
}

// ---------------------------------------------------------------------------
// Line-cooperative variant (8-column slices, W = R = 32 or 64, d_v a multiple
// of 32).
//
// The four waves of a workgroup are four consecutive 8-column slices of one
// stream, i.e. 32 columns: one 128-byte line of every table row.  With each
// wave moving only its own 32 bytes of a row, the 16 slices of a stream touch
// the 4 lines of a row at different times, and the memory system then serves
// the scattered rows at about 3.9 TB/s; moving whole lines it serves the same
// bytes at about 5 TB/s.  So global table loads and stores go through LDS:
// each wave loads (and stores) a quarter of the rows of a token as whole
// lines, and the pieces a wave computes on are exchanged through LDS, with two
// workgroup barriers per token.  The recurrence itself (links, rings, per-token
// arithmetic) is the same as in scan_bwd_kernel, per wave and per slice.
//
// Per token t (B1, B2 are workgroup barriers):
//   S1  this wave's line rows of token t (loaded earlier) -> LDS row buffer
//   B1
//   S2  line loads of token t - PD + 1
//   S3  each wave reads its pieces, runs the token, and writes its output
//       pieces (G rows read, G rows written) over the pieces it read
//   B2
//   S4  each wave stores its line rows of each output as whole lines; the
//       undo rows (M rows written) are the saved rows it loaded, stored from
//       its registers
// Every LDS position of the row buffer has one owner lane in the line layout
// (S1, S4) and one in the piece layout (S3), so the outputs can take the
// inputs' place: S3 overwrites only pieces its own lane has read, and S4 and
// the next S1 touch only the lane's own line positions.
// A load issued in S2 sees the stores of tokens >= t + 1 (every wave stored
// those before B1), and the tokens t .. t - PD + 2 that it does not see are
// exactly the PD - 1 tokens the prep kernel links to the LDS rings, as in
// the per-wave kernel (whose loads for t - PD follow token t's stores).
// A read row whose slot the same token also writes must end with the write
// adjoint: the write pass marks such rows (a d = 0 link into the read part)
// and S4 skips their read-adjoint store.
constexpr int LW = 4;          // waves (slices) per workgroup
constexpr int LROWB = 160;     // LDS bytes per staged row: 128 + 32 of padding, so that
                               // the per-slice piece reads (stride of one row) hit distinct banks
// Rows per token (W = R = LR, 32 or 64); each lane holds LR / 32 of them in both layouts.
template <int LR>
constexpr int lflags() { return LR + SDM_WAVE; }   // read-row marks, then one dummy entry per lane
template <int LR>
constexpr int lpart() { return 2 * LR + 2; }       // per-token partial sums: rbar[LR], kbar[LR], dbeta, dalpha
template <int LR>
constexpr int line_shared_bytes() { return 4 * LR * LROWB + lflags<LR>() * 4 + LW * lpart<LR>() * 4; }

template <int KR>
struct LineBuf {
    v4f Mr[KR], Gr[KR], Gw[KR], Ps[KR];   // line layout: rows 8 w + lane / 8 + 32 k, columns 4 (lane % 8)
    v4f Dy;                               // piece layout: this lane's 4 columns of dy
};

// Row buffer: [4][LR] rows of LROWB bytes (M read, G read -> G read out,
// G written -> G written out, saved row).
template <int LR>
__device__ __forceinline__ v4f lds4(const unsigned char* base, int a, int r, int q) {
    return *reinterpret_cast<const v4f*>(base + (a * LR + r) * LROWB + q * 16);
}
template <int LR>
__device__ __forceinline__ void lds4_st(unsigned char* base, int a, int r, int q, v4f v) {
    *reinterpret_cast<v4f*>(base + (a * LR + r) * LROWB + q * 16) = v;
}

// Record fields of one token for this lane's rows, read before the token's
// first barrier so that their LDS latency overlaps the barrier wait.
struct LineRow {
    float rho, kap;
    int l1, l2, lw;   // links of M_t[j_m], G[j_m], G[i_n]
};
template <int KR>
struct LineTok {
    LineRow r[KR];   // rows rg + 32 k
    v4f vv;
};

template <typename VT, int NS, int KR>
__device__ __forceinline__ void line_read_tok(LineTok<KR>& x, float& al, float& be, const BwdCtx& c, int t) {
    constexpr int VB = 8 * (int)sizeof(VT);
    const BwdRec& L = c.L;
    const unsigned char* rec = c.rring + (t & (NS - 1)) * L.bytes;
    al = reinterpret_cast<const float*>(rec + L.off_ab)[0];
    be = reinterpret_cast<const float*>(rec + L.off_ab)[1];
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int m = c.rg + 32 * k;
        x.r[k].rho = reinterpret_cast<const float*>(rec + L.off_rval)[m];
        x.r[k].kap = reinterpret_cast<const float*>(rec + L.off_wval)[m];
        x.r[k].l1 = reinterpret_cast<const short*>(rec + L.off_lm)[m];
        x.r[k].l2 = reinterpret_cast<const short*>(rec + L.off_lgr)[m];
        x.r[k].lw = reinterpret_cast<const short*>(rec + L.off_lgw)[m];
    }
    x.vv = ld4v(reinterpret_cast<const VT*>(c.vring + (t & (NS - 1)) * VB) + c.cq * 4);
}

// One token on the pieces (rows rg + 32 k, columns 4 cq.. of slice w) read from
// the row buffer; outputs over those pieces and to the per-wave rings.
template <int LR, int PD>
__device__ __forceinline__ void bwd_token_line(const BwdCtx& c, unsigned char* lb, int* flags, float* psum,
                                               const LineTok<LR / 32>& x, float al, float be, v4f yb, int t,
                                               int w, int lane) {
    using namespace sdm_reduce;
    constexpr int SW = 8;
    constexpr int KR = LR / 32;
    constexpr int RW = 2 * LR;
    const int q = 2 * w + c.cq;           // this lane's column quad within the line
    float* prow = psum + w * lpart<LR>();   // this slice's partial sums of the token (LDS)
    float* gring_t = c.gring + (size_t)((t & (PD - 1)) * RW) * SW + c.cq * 4;

    // ---- read adjoint: rbar_m = <dy, M_t[j_m]>, G[j_m] += rho_m dy ----
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int m = c.rg + 32 * k;
        const int l1 = x.r[k].l1, l2 = x.r[k].l2;
        const int i1 = l1 >= 0 ? (((t + (l1 >> 8)) & (PD - 1)) * LR + min(l1 & 255, LR - 1)) : 0;
        const v4f Mv = v4sel(l1 >= 0, ld4(c.pring + i1 * SW + c.cq * 4), lds4<LR>(lb, 0, m, q));
        const float rb = add_xor<1>(v4dot(yb, Mv));
        const int i2 = l2 >= 0 ? (((t + (l2 >> 8)) & (PD - 1)) * RW + min(l2 & 255, RW - 1)) : 0;
        v4f g = v4sel(l2 >= 0, ld4(c.gring + i2 * SW + c.cq * 4), lds4<LR>(lb, 1, m, q));
        g = v4fma(x.r[k].rho, yb, g);
        st4(gring_t + m * SW, g);
        lds4_st<LR>(lb, 1, m, q, g);
        if (c.cq == 0) prow[m] = rb;
    }

    // ---- write adjoint ----
    v4f gn[KR], D[KR], Ps[KR];
    v4f up = v4zero(), ebp = v4zero();
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int n = c.rg + 32 * k;
        const int l = x.r[k].lw;
        const int ig = l >= 0 ? (((t + (l >> 8)) & (PD - 1)) * RW + min(l & 255, RW - 1)) : 0;
        gn[k] = v4sel(l >= 0, ld4(c.gring + ig * SW + c.cq * 4), lds4<LR>(lb, 2, n, q));
        Ps[k] = lds4<LR>(lb, 3, n, q);
        D[k] = al * Ps[k];
        up = v4fma(x.r[k].kap, D[k], up);
        ebp = v4fma(x.r[k].kap, gn[k], ebp);
    }
    rows_allreduce8<2>(up, ebp);
    const v4f vmu = x.vv - up;
    const v4f e = be * vmu;
    const float bb = add_xor<1>(v4dot(ebp, vmu));
    float abl = 0.f;
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int n = c.rg + 32 * k;
        const float kb = add_xor<1>(v4dot(gn[k], e) - be * v4dot(ebp, D[k]));
        const v4f Db = v4fma(-be * x.r[k].kap, ebp, gn[k]);
        abl += v4dot(Db, Ps[k]);
        const v4f gnew = al * Db;
        st4(gring_t + (LR + n) * SW, gnew);
        st4(c.pring + ((t & (PD - 1)) * LR + n) * SW + c.cq * 4, Ps[k]);
        lds4_st<LR>(lb, 2, n, q, gnew);
        // a d = 0 link into the read part: this token also reads the slot it writes
        const int l = x.r[k].lw;
        const bool same = l >= 0 && (l >> 8) == 0 && (l & 255) < LR;
        flags[same ? (l & 255) : LR + lane] = t;
        if (c.cq == 1) prow[LR + n] = kb;
    }
    const float ab = wave_sum(abl);
    // row 0 also writes dbeta and dalpha, and stores this slice's dv of the token
    if (lane < 2) {
        st4(c.sdv + (size_t)t * c.dv, be * ebp);
        prow[RW + lane] = lane ? ab : bb;
    }
}

// Staging for the line kernel: the records of the G tokens [u1 - G + 1, u1]
// (clamped at lo) go to one ring that the workgroup's waves share (they read
// the same records), 16-byte chunk w 64 + lane + 256 j, j < NC, per lane; each
// wave stages the v slices of its own columns.  Loads are unconditional at
// clamped indices; the surplus is never stored.
template <typename VT, int NC>
__device__ __forceinline__ void bline_stage_load(u4v (&st)[NC], u2v& stv, const unsigned char* srec,
                                                 const VT* sv, int u1, int lo, int dv, int slice, int rec_bytes,
                                                 int w, int lane) {
    constexpr int SW = 8;
    constexpr int VB = SW * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
    const int ub1 = max(u1, lo);
    const int u0 = max(lo, ub1 - G + 1);
    const int cnt = ub1 - u0 + 1;
    const u4v* src = reinterpret_cast<const u4v*>(srec + (size_t)u0 * rec_bytes);
    const int last = cnt * rec_bytes / 16 - 1;
#pragma unroll
    for (int j = 0; j < NC; ++j) st[j] = src[min(w * SDM_WAVE + lane + j * LW * SDM_WAVE, last)];
    const int tk = min(lane / ppt, cnt - 1);
    const int pc = min(lane % ppt, (dv - slice * SW) * (int)sizeof(VT) / 8 - 1);
    stv = *reinterpret_cast<const u2v*>(
        reinterpret_cast<const unsigned char*>(sv + (size_t)(u0 + tk) * dv) + pc * 8);
}
template <typename VT, int NS, int NC>
__device__ __forceinline__ void bline_stage_store(const u4v (&st)[NC], u2v stv, unsigned char* rring,
                                                  unsigned char* vring, int u1, int lo, int rec_bytes, int w,
                                                  int lane) {
    constexpr int VB = 8 * (int)sizeof(VT);
    constexpr int ppt = VB / 8;
    if (u1 < lo) return;
    const int u0 = max(lo, u1 - G + 1);
    const int cnt = u1 - u0 + 1;
    const int nchunk = cnt * rec_bytes / 16;   // <= NC * 256 (checked by the host)
#pragma unroll
    for (int j = 0; j < NC; ++j) {
        const int c = w * SDM_WAVE + lane + j * LW * SDM_WAVE;
        if (c < nchunk) {
            const int tk = (c * 16) / rec_bytes;   // records are whole 16-byte chunks
            const int within = c * 16 - tk * rec_bytes;
            *reinterpret_cast<u4v*>(rring + ((u0 + tk) & (NS - 1)) * rec_bytes + within) = st[j];
        }
    }
    const int tk = lane / ppt, pc = lane % ppt;
    if (tk < cnt) *reinterpret_cast<u2v*>(vring + ((u0 + tk) & (NS - 1)) * VB + pc * 8) = stv;
}

// Slot ids (this lane's line rows) of token u's read rows and written rows.
template <int KR>
__device__ __forceinline__ void line_slots(int2 (&sl)[KR], const BwdCtx& c, int u, int rl, int NS) {
    const unsigned char* rec = c.rring + (u & (NS - 1)) * c.L.bytes;
#pragma unroll
    for (int k = 0; k < KR; ++k)
        sl[k] = make_int2(reinterpret_cast<const int*>(rec + c.L.off_rslot)[rl + 32 * k],
                          reinterpret_cast<const int*>(rec)[rl + 32 * k]);
}

// The stream's memory table, adjoint table and saved rows as buffers (each below
// 2 GiB, rows below 2^24): row s of a table at byte offset s 4 d_v + 4 lc, with
// lc this lane's first line column, saved row (u, r) at (LR u + r) 4 d_v + 4 lc.
// 32-bit offsets through a 24-bit multiply keep the address arithmetic off the
// latency-bound token chain.
struct LinePtrs {
    __amdgpu_buffer_rsrc_t mt, gt, sv;
    uint32_t dv4, lc4;
    int rl;             // this lane's first line row (0..31)
    int lq;             // this lane's column quad within the line
};

typedef unsigned int lu32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ v4f lbuf_ld(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}
__device__ __forceinline__ void lbuf_st(__amdgpu_buffer_rsrc_t r, uint32_t off, v4f x) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(lu32x4, x), r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t lrow_off(const LinePtrs& p, int row) {
    return __umul24((uint32_t)row, p.dv4) + p.lc4;
}

template <int LR>
__device__ __forceinline__ void line_issue(LineBuf<LR / 32>& b, const BwdCtx& c, const LinePtrs& p,
                                           const int2 (&sl)[LR / 32], int u) {
#pragma unroll
    for (int k = 0; k < LR / 32; ++k) {
        b.Mr[k] = lbuf_ld(p.mt, lrow_off(p, sl[k].x));
        b.Gr[k] = lbuf_ld(p.gt, lrow_off(p, sl[k].x));
        b.Gw[k] = lbuf_ld(p.gt, lrow_off(p, sl[k].y));
        b.Ps[k] = lbuf_ld(p.sv, lrow_off(p, u * LR + p.rl + 32 * k));
    }
    b.Dy = ld4(c.sdy + (size_t)u * c.dv);
}

template <typename VT, int LR, int PD, int NS>
__device__ __forceinline__ void line_step(const BwdCtx& c, const LinePtrs& p, unsigned char* lb, int* flags,
                                          float* psum, const LineBuf<LR / 32>& cur, LineBuf<LR / 32>& nxt, int t,
                                          int tb, int w, int lane, bool issue) {
    constexpr int KR = LR / 32;
    constexpr int LP = lpart<LR>();
    constexpr int PPW = (LP + LW - 1) / LW;   // partial sums each wave adds up
    const int u = max(t - PD + 1, tb);
    LineTok<KR> x;
    float al, be;   // kept out of the struct: splats of struct fields become vector loads that pin it to memory
    line_read_tok<VT, NS, KR>(x, al, be, c, t);
    int2 st_sl[KR], ld_sl[KR];
    line_slots<KR>(st_sl, c, t, p.rl, NS);
    line_slots<KR>(ld_sl, c, u, p.rl, NS);
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int r = p.rl + 32 * k;
        lds4_st<LR>(lb, 0, r, p.lq, cur.Mr[k]);
        lds4_st<LR>(lb, 1, r, p.lq, cur.Gr[k]);
        lds4_st<LR>(lb, 2, r, p.lq, cur.Gw[k]);
        lds4_st<LR>(lb, 3, r, p.lq, cur.Ps[k]);
    }
    __syncthreads();
    // every wave stored token t + 1 before the barrier: the loads may go now
    if (issue) line_issue<LR>(nxt, c, p, ld_sl, u);
    bwd_token_line<LR, PD>(c, lb, flags, psum, x, al, be, cur.Dy, t, w, lane);
    __syncthreads();
    // the workgroup's partial sums of the token: wave w adds entries PPW w ..
    // PPW w + PPW - 1 of the four slices and stores them
    const int pi = PPW * w + lane;
    if (lane < PPW && pi < LP)
        c.spart[(size_t)t * LP + pi] = ((psum[pi] + psum[LP + pi]) + psum[2 * LP + pi]) + psum[3 * LP + pi];
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const int r = p.rl + 32 * k;
        if (flags[r] != t) lbuf_st(p.gt, lrow_off(p, st_sl[k].x), lds4<LR>(lb, 1, r, p.lq));
        lbuf_st(p.gt, lrow_off(p, st_sl[k].y), lds4<LR>(lb, 2, r, p.lq));
        lbuf_st(p.mt, lrow_off(p, st_sl[k].y), cur.Ps[k]);
    }
}

template <typename VT, int LR, int PD, int NC>
__global__ __launch_bounds__(LW * SDM_WAVE) void scan_bwd_line_kernel(
    const unsigned char* __restrict__ recs, const VT* __restrict__ v, float* __restrict__ mem,
    const float* __restrict__ saved, const float* __restrict__ dy, float* __restrict__ Gtab,
    float* __restrict__ dv_out, float* __restrict__ part, int T, int tb, int te, int dv, int64_t N,
    int n_slices, int S, int per_wave_lds) {
    // tokens te-1 down to tb of each stream (layout strides use T)
    constexpr int SW = 8;
    constexpr int KR = LR / 32;
    constexpr int LEAD = bstage_lead<PD>();
    constexpr int NS = bstage_slots<PD>();
    constexpr int VB = SW * (int)sizeof(VT);
    static_assert(LR == 32 || LR == 64, "32 or 64 rows per token");
    static_assert(PD % G == 0, "prefetch depth must be a multiple of the staging block");
    static_assert(NS >= LEAD && NS >= PD, "record ring too small");

    const int lane = lane_id();
    const int w = threadIdx.x / SDM_WAVE;
    int group, stream;
    scan_wg_coords<true>(n_slices / LW, group, stream);
    const int slice = group * LW + w;   // n_slices is a multiple of LW: every wave exists

    BwdCtx c;
    c.L = bwd_rec_layout(LR, LR);
    c.dv = dv;
    c.W = LR;
    c.R = LR;
    c.rg = lane / 2;
    c.cq = lane % 2;
    c.colok = true;
    const int col = slice * SW + c.cq * 4;

    // LDS: the shared record ring, then per wave its v ring, adjoint ring and
    // undo ring, then the row buffer, flags and partial sums
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char* rring = smem;
    unsigned char* vring = smem + (size_t)NS * c.L.bytes + (size_t)w * per_wave_lds;
    c.rring = rring;
    c.vring = vring;
    c.gring = reinterpret_cast<float*>(vring + NS * VB);
    c.pring = c.gring + PD * 2 * LR * SW;
    c.mtab = mem + (size_t)stream * N * dv + col;
    c.gtab = Gtab + (size_t)stream * N * dv + col;
    c.ssaved = saved + (size_t)stream * T * LR * dv + col;
    c.sdy = dy + (size_t)stream * T * dv + col;
    c.sdv = dv_out + (size_t)stream * T * dv + col;
    c.spart = part + ((size_t)group * S + stream) * T * lpart<LR>();   // per workgroup (4 slices)
    unsigned char* lb = smem + (size_t)NS * c.L.bytes + (size_t)LW * per_wave_lds;
    int* flags = reinterpret_cast<int*>(lb + 4 * LR * LROWB);
    float* psum = reinterpret_cast<float*>(flags + lflags<LR>());

    LinePtrs p;
    p.rl = 8 * w + lane / 8;
    p.lq = lane % 8;
    const uint32_t lcol = (uint32_t)group * 32 + p.lq * 4;
    const int tbytes = (int)((size_t)N * dv * 4);
    p.mt = __builtin_amdgcn_make_buffer_rsrc(mem + (size_t)stream * N * dv, 0, tbytes, 0x00020000);
    p.gt = __builtin_amdgcn_make_buffer_rsrc(Gtab + (size_t)stream * N * dv, 0, tbytes, 0x00020000);
    p.sv = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(saved) + (size_t)stream * T * LR * dv, 0,
                                             (int)((size_t)T * LR * dv * 4), 0x00020000);
    p.dv4 = (uint32_t)dv * 4;
    p.lc4 = lcol * 4;

    if (w == 0)
        for (int i = lane; i < lflags<LR>(); i += SDM_WAVE) flags[i] = -1;

    const unsigned char* srec = recs + (size_t)stream * T * c.L.bytes;
    const VT* sv = v + (size_t)stream * T * dv + slice * SW;
    u4v st[NC];
    u2v stv;
    LineBuf<KR> buf[PD];

    const int T1 = te - 1;
    for (int i0 = 0; i0 < LEAD - G; i0 += G) {
        bline_stage_load<VT, NC>(st, stv, srec, sv, T1 - i0, tb, dv, slice, c.L.bytes, w, lane);
        bline_stage_store<VT, NS, NC>(st, stv, rring, vring, T1 - i0, tb, c.L.bytes, w, lane);
    }
    bline_stage_load<VT, NC>(st, stv, srec, sv, T1 - (LEAD - G), tb, dv, slice, c.L.bytes, w, lane);
    __syncthreads();   // the first records staged by every wave
#pragma unroll
    for (int j = 0; j < PD - 1; ++j) {
        const int u = max(T1 - j, tb);
        int2 sl[KR];
        line_slots<KR>(sl, c, u, p.rl, NS);
        line_issue<LR>(buf[j], c, p, sl, u);
    }
    __syncthreads();   // flags initialised

    // Token t = te-1-i uses buf[i % PD]; step i loads token t - PD + 1 into
    // buf[(i + PD - 1) % PD], the buffer token t + 1 used.
    const int n = te - tb;
    const int nfull = n - n % PD;
    for (int i0 = 0; i0 < nfull; i0 += PD) {
#pragma unroll
        for (int j = 0; j < PD; ++j) {
            const int t = T1 - (i0 + j);
            if (j % G == 0) {
                bline_stage_store<VT, NS, NC>(st, stv, rring, vring, t - (LEAD - G), tb, c.L.bytes, w, lane);
                bline_stage_load<VT, NC>(st, stv, srec, sv, t - LEAD, tb, dv, slice, c.L.bytes, w, lane);
            }
            line_step<VT, LR, PD, NS>(c, p, lb, flags, psum, buf[j], buf[(j + PD - 1) % PD], t, tb, w, lane,
                                      true);
        }
    }
#pragma unroll
    for (int j = 0; j < PD; ++j) {
        const int i = nfull + j;
        if (i < n)
            line_step<VT, LR, PD, NS>(c, p, lb, flags, psum, buf[j], buf[(j + PD - 1) % PD], T1 - i, tb, w, lane,
                                      false);
    }
}

// Sum the partial scalars (one set per slice, or per workgroup of slices for the
// line-cooperative kernel) of tokens [tb, tb + n) of every stream: rbar -> dr_val,
// kbar -> dw_val, dbeta, dalpha.
__global__ __launch_bounds__(256) void bwd_reduce_kernel(const float* __restrict__ part, int n_parts, int S,
                                                         int T, int tb, int n, int W, int R,
                                                         float* __restrict__ dw_val,
                                                         float* __restrict__ dr_val,
                                                         float* __restrict__ dbeta,
                                                         float* __restrict__ dalpha) {
    const int NP = W + R + 2;
    const int64_t ST = (int64_t)S * T;
    const int64_t total = (int64_t)S * n * NP;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t sr = i / NP;
        const int p = (int)(i % NP);
        const int64_t st = (sr / n) * T + tb + sr % n;
        float acc = 0.f;
        for (int sl = 0; sl < n_parts; ++sl) acc += part[((size_t)sl * ST + st) * NP + p];
        if (p < R)
            dr_val[st * R + p] = acc;
        else if (p < R + W)
            dw_val[st * W + (p - R)] = acc;
        else if (p == R + W)
            dbeta[st] = acc;
        else
            dalpha[st] = acc;
    }
}

constexpr int BPD = SDM_BWD_PD;
constexpr int BPD_LINE = 8;   // the line-cooperative kernel's deeper window
constexpr int BSW_MIN = 8;   // narrowest slice: sizes the per-slice partials
// Prefetch depth of the per-wave kernel with K row passes: BPD tokens, or 2 at
// K = 4 (64 rows at 16 columns, 128 at 8), where BPD tokens of prefetched rows
// (4 x 17 float4 per lane) outgrow the registers.  The records' links follow
// the same depth.
constexpr int bpd_for_k(int K) { return K >= 4 ? 2 : BPD; }

// Staging registers per lane (16 bytes each) for a block of G records: a
// record of a shape with max(W, R) <= K RG takes at most 22 K RG + 8 bytes
// rounded up to 16.
template <int SW>
constexpr int bnr_for_k(int K) {
    constexpr int RG = SDM_WAVE / (SW / 4);
    return (G * ((22 * K * RG + 8 + 15) / 16 * 16) + SDM_WAVE * 16 - 1) / (SDM_WAVE * 16);
}

struct BwdPlan {
    int SW, K, NR, lds_per_wave, wpb, n_slices, PD;
};

template <int SW>
bool bwd_plan_sw(int W, int R, int dv, int in_dtype, BwdPlan* p) {
    constexpr int RG = SDM_WAVE / (SW / 4);
    const int need = (std::max(W, R) + RG - 1) / RG;   // row passes: at most 4 (64 or 128 rows)
    if (need > 4) return false;
    p->SW = SW;
    p->K = need <= 1 ? 1 : (need <= 2 ? 2 : 4);
    p->NR = bnr_for_k<SW>(p->K);
    p->PD = bpd_for_k(p->K);
    const BwdRec L = bwd_rec_layout(W, R);
    if (G * L.bytes > p->NR * SDM_WAVE * 16) return false;
    const int vbytes = in_dtype == SDM_DT_BF16 ? 2 : 4;
    static_assert(bstage_slots<2>() == bstage_slots<BPD>(), "one record ring size for both depths");
    constexpr int NS = bstage_slots<BPD>();
    p->lds_per_wave = NS * L.bytes + NS * SW * vbytes + p->PD * (R + W) * SW * 4 + p->PD * W * SW * 4;
    if (p->lds_per_wave > LDS_LIMIT) return false;
    p->n_slices = (dv + SW - 1) / SW;
    p->wpb = std::min(std::min(MAX_WPB, p->n_slices), LDS_LIMIT / p->lds_per_wave);
    return true;
}

// 8 columns per wave, unless that would put 1.5 or more waves on every SIMD:
// then 16, unless a width is forced (the reason is the forward's); the other
// width when the chosen one cannot hold the shape (16 columns hold at most 64
// rows).
bool bwd_plan(int S, int W, int R, int dv, int in_dtype, BwdPlan* p) {
    const int forced = sdm_scan_slice_width();
    if (forced == 16 || (forced == 0 && 2 * (int64_t)S * ((dv + 7) / 8) >= 3 * (int64_t)sdm_device_simds()))
        return bwd_plan_sw<16>(W, R, dv, in_dtype, p) || bwd_plan_sw<BSW_MIN>(W, R, dv, in_dtype, p);
    return bwd_plan_sw<BSW_MIN>(W, R, dv, in_dtype, p) || bwd_plan_sw<16>(W, R, dv, in_dtype, p);
}

// LDS of the line-cooperative kernel at LR rows and prefetch depth PD: the
// shared record ring, each wave's v, adjoint and undo rings, the row buffer.
template <int LR, int PD>
size_t line_per_wave(int in_dtype) {
    const int vbytes = in_dtype == SDM_DT_BF16 ? 2 : 4;
    return (size_t)bstage_slots<PD>() * 8 * vbytes + (size_t)PD * 2 * LR * 8 * 4 + (size_t)PD * LR * 8 * 4;
}
template <int LR, int PD>
size_t line_lds(int in_dtype) {
    return (size_t)bstage_slots<PD>() * bwd_rec_layout(LR, LR).bytes + LW * line_per_wave<LR, PD>(in_dtype) +
           line_shared_bytes<LR>();
}
// 16-byte record chunks per lane for G records of W = R = LR
template <int LR>
constexpr int line_nc() {
    return (G * ((22 * LR + 8 + 15) / 16 * 16) + LW * SDM_WAVE * 16 - 1) / (LW * SDM_WAVE * 16);
}
static_assert(line_nc<32>() == 1 && line_nc<64>() == 2, "line staging chunks");

// Rows per token of the line-cooperative kernel for this shape, or 0.
int line_rows(const ScanBwdArgs& a) { return a.W == a.R && (a.W == 32 || a.W == 64) ? a.W : 0; }

// The line-cooperative kernel's shape: W = R = 32 (where the per-wave plan
// takes 8-column slices) or 64, d_v a multiple of 32 (whole lines per
// workgroup of four 8-column slices), and its LDS within the limit.  Its table
// and saved-row offsets are 32-bit: each stream's tables and saved rows below
// 2 GiB, their row counts below 2^24.
bool line_shape_ok(const ScanBwdArgs& a, const BwdPlan& p) {
    const int LR = line_rows(a);
    if (LR == 0 || a.dv % 32 != 0) return false;
    const size_t two_gib = (size_t)1 << 31;
    if ((size_t)a.N * a.dv * 4 >= two_gib || a.N >= (1 << 24)) return false;
    if ((size_t)a.T * LR * a.dv * 4 >= two_gib || (size_t)a.T * LR >= ((size_t)1 << 24)) return false;
    if (LR == 32) return p.SW == 8 && line_lds<32, BPD>(a.in_dtype) <= (size_t)LDS_LIMIT;
    return line_lds<64, BPD>(a.in_dtype) <= (size_t)LDS_LIMIT;
}
// Prefetch depth of the line-cooperative kernel: 4 tokens, or 8 when
// sdm_set_scan_prefetch forces 8 or 16 and the LDS holds it (32 rows: the
// shared record ring leaves LDS for the deeper adjoint and undo rings).  At the
// training workload 8 measured no faster (1.13 against 1.12 ms per stage) and
// doubled the records' link search (0.83 against 0.39 ms per stage beside the
// scan).
int line_pd(const ScanBwdArgs& a) {
    const int forced = sdm_scan_prefetch();
    return forced >= 8 && line_rows(a) == 32 && line_lds<32, BPD_LINE>(a.in_dtype) <= (size_t)LDS_LIMIT ? BPD_LINE
                                                                                                        : BPD;
}
bool line_io_ok(const ScanBwdArgs& a, const BwdPlan& p) { return sdm_line_io_enabled() && line_shape_ok(a, p); }
// a.line >= 0: the caller's decision (one per call, so that every range and the
// reduce agree), which must fit the shape
bool use_line(const ScanBwdArgs& a, const BwdPlan& p, bool* ok) {
    *ok = a.line <= 0 || line_shape_ok(a, p);
    return a.line >= 0 ? (a.line != 0 && *ok) : line_io_ok(a, p);
}

// The line-cooperative kernel (line_shape_ok held): d_v / 32 workgroups of four
// 8-column slices per stream, whose partial sums are per workgroup.  It asks
// for more than half a CU's LDS, so that no two of its workgroups share a CU:
// at the 32-row training workload (256 workgroups) two per CU took the scan
// from 1.13 to 1.38 ms per stage, their token chains sharing the SIMDs while
// other CUs idled.
template <typename VT, int LR, int PD>
hipError_t launch_bwd_line(const ScanBwdArgs& a, float* part, hipStream_t st) {
    auto kl = scan_bwd_line_kernel<VT, LR, PD, line_nc<LR>()>;
    const size_t sml = std::max(line_lds<LR, PD>(a.in_dtype), (size_t)LDS_LIMIT / 2 + 1024);
    const size_t pw = line_per_wave<LR, PD>(a.in_dtype);
    hipError_t e = hipFuncSetAttribute((const void*)kl, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sml);
    if (e != hipSuccess) return e;
    const int S = a.B * a.H;
    const int n_slices = a.dv / 8;
    hipLaunchKernelGGL(kl, dim3(n_slices / LW * S), dim3(LW * SDM_WAVE), sml, st, a.ws + SDM_WS_HEADER,
                       static_cast<const VT*>(a.v), a.mem, a.saved, a.dy, a.G, a.dv_out, part, a.T, a.tb, a.te,
                       a.dv, a.N, n_slices, S, (int)pw);
    return hipGetLastError();
}

template <typename VT, int SW, int K>
hipError_t launch_bwd_k(const ScanBwdArgs& a, const BwdPlan& p, float* part, hipStream_t st) {
    constexpr int NR = bnr_for_k<SW>(K);
    const int S = a.B * a.H;
    dim3 grid((p.n_slices + p.wpb - 1) / p.wpb * S);   // XCD-aware order: scan_wg_coords<true>
    const size_t sm = (size_t)p.lds_per_wave * p.wpb;
    auto kfn = scan_bwd_kernel<VT, SW, bpd_for_k(K), K, NR>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, grid, dim3(p.wpb * SDM_WAVE), sm, st, a.ws + SDM_WS_HEADER,
                       static_cast<const VT*>(a.v), a.mem, a.saved, a.dy, a.G, a.dv_out, part, a.T,
                       a.tb, a.te, a.dv, a.W, a.R, a.N, p.n_slices, S, p.lds_per_wave);
    return hipGetLastError();
}

template <typename VT>
hipError_t launch_bwd_kk(const ScanBwdArgs& a, const BwdPlan& p, bool line, float* part, hipStream_t st) {
    if (line) {
        if (line_rows(a) == 64) return launch_bwd_line<VT, 64, BPD>(a, part, st);
        return line_pd(a) == BPD_LINE ? launch_bwd_line<VT, 32, BPD_LINE>(a, part, st)
                                      : launch_bwd_line<VT, 32, BPD>(a, part, st);
    }
    if (p.SW == 8) {
        if (p.K == 1) return launch_bwd_k<VT, 8, 1>(a, p, part, st);
        if (p.K == 2) return launch_bwd_k<VT, 8, 2>(a, p, part, st);
        return launch_bwd_k<VT, 8, 4>(a, p, part, st);
    }
    if (p.K == 1) return launch_bwd_k<VT, 16, 1>(a, p, part, st);
    if (p.K == 2) return launch_bwd_k<VT, 16, 2>(a, p, part, st);
    return launch_bwd_k<VT, 16, 4>(a, p, part, st);
}

size_t bwd_part_offset(int B, int H, int T, int W, int R) {
    const size_t recb = (size_t)B * H * T * bwd_rec_layout(W, R).bytes;
    return SDM_WS_HEADER + ((recb + 255) & ~(size_t)255);
}

}  // namespace

size_t sdm_bwd_ws_bytes(int B, int H, int T, int W, int R, int dv) {
    const int n_slices = (dv + BSW_MIN - 1) / BSW_MIN;   // the most slices any plan uses
    const size_t ST = (size_t)B * H * T;
    size_t bytes = bwd_part_offset(B, H, T, W, R) + (size_t)n_slices * ST * (W + R + 2) * sizeof(float);
    bytes = (bytes + 255) & ~(size_t)255;
    bytes += ST * (size_t)(W + R) * sizeof(float);   // weight gradients when the caller wants none
    return bytes;
}

bool sdm_bwd_plan_ok(int W, int R, int dv, int in_dtype) {
    BwdPlan p;   // every width bwd_plan may choose falls back to the 8-column plan
    return bwd_plan_sw<BSW_MIN>(W, R, dv, in_dtype, &p);
}

bool sdm_bwd_line_io(const ScanBwdArgs& a) {
    BwdPlan plan;
    return bwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &plan) && line_io_ok(a, plan);
}

hipError_t sdm_launch_bwd_prep_range(const ScanBwdArgs& a, hipStream_t st) {
    BwdPlan plan;   // the links' window is the scan's prefetch depth
    if (!bwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &plan)) return hipErrorInvalidConfiguration;
    bool ok;
    const bool line = use_line(a, plan, &ok);
    if (!ok) return hipErrorInvalidConfiguration;
    SdmProfScope ps(SDM_K_BWD_PREP, st);
    if (line) return line_pd(a) == BPD_LINE ? sdm_launch_bwd_prep<BPD_LINE>(a, st) : sdm_launch_bwd_prep<BPD>(a, st);
    return plan.PD == 2 ? sdm_launch_bwd_prep<2>(a, st) : sdm_launch_bwd_prep<BPD>(a, st);
}

hipError_t sdm_launch_bwd_scan_range(const ScanBwdArgs& a, hipStream_t st) {
    BwdPlan plan;
    if (!bwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &plan)) return hipErrorInvalidConfiguration;
    bool ok;
    const bool line = use_line(a, plan, &ok);
    if (!ok) return hipErrorInvalidConfiguration;
    float* part = reinterpret_cast<float*>(a.ws + bwd_part_offset(a.B, a.H, a.T, a.W, a.R));
    SdmProfScope ps(SDM_K_BWD_SCAN, st);
    return a.in_dtype == SDM_DT_BF16 ? launch_bwd_kk<bf16_t>(a, plan, line, part, st)
                                     : launch_bwd_kk<float>(a, plan, line, part, st);
}

hipError_t sdm_launch_bwd_reduce_range(const ScanBwdArgs& a, hipStream_t st) {
    BwdPlan plan;
    if (!bwd_plan(a.B * a.H, a.W, a.R, a.dv, a.in_dtype, &plan)) return hipErrorInvalidConfiguration;
    bool ok;
    const bool line = use_line(a, plan, &ok);
    if (!ok) return hipErrorInvalidConfiguration;
    const int n_parts = line ? a.dv / 32 : plan.n_slices;   // partial sums per (stream, token)
    const float* part = reinterpret_cast<const float*>(a.ws + bwd_part_offset(a.B, a.H, a.T, a.W, a.R));
    const int S = a.B * a.H, n = a.te - a.tb;
    if (S == 0 || n <= 0) return hipSuccess;
    SdmProfScope ps(SDM_K_BWD_REDUCE, st);
    const int64_t total = (int64_t)S * n * (a.W + a.R + 2);
    const unsigned nb = (unsigned)std::min<int64_t>((total + 255) / 256, 65536);
    hipLaunchKernelGGL(bwd_reduce_kernel, dim3(nb), dim3(256), 0, st, part, n_parts, S, a.T, a.tb, n, a.W, a.R,
                       a.dw_val, a.dr_val, a.dbeta, a.dalpha);
    return hipGetLastError();
}

// ---------------------------------------------------------------- memory init
namespace {
// M0 broadcast over B (m0 = [H][per_head4] float4s) or a zero fill.  Block row
// y is one head h (broadcast: every element is read once and written to all B
// tables) or one (b, h) table (zero fill); each thread handles 4 float4s (one
// per 256-thread stride) per pass.
__global__ __launch_bounds__(256) void mem_init_kernel(float4* __restrict__ dst,
                                                       const float4* __restrict__ m0,
                                                       int64_t per_head4, int B, int H) {
    const int row = blockIdx.y;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
    if (m0) {
        const float4* src = m0 + (size_t)row * per_head4;
        for (int64_t i0 = ((int64_t)blockIdx.x * blockDim.x) * 4 + threadIdx.x; i0 < per_head4; i0 += stride) {
            float4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t i = i0 + (int64_t)u * blockDim.x;
                if (i < per_head4) v[u] = src[i];
            }
            for (int b = 0; b < B; ++b) {
                float4* d = dst + ((size_t)b * H + row) * per_head4;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int64_t i = i0 + (int64_t)u * blockDim.x;
                    if (i < per_head4) d[i] = v[u];
                }
            }
        }
    } else {
        float4* d = dst + (size_t)row * per_head4;
        for (int64_t i0 = ((int64_t)blockIdx.x * blockDim.x) * 4 + threadIdx.x; i0 < per_head4; i0 += stride) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t i = i0 + (int64_t)u * blockDim.x;
                if (i < per_head4) d[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    }
}
__global__ __launch_bounds__(256) void copy_kernel(float4* __restrict__ dst, const float4* __restrict__ src,
                                                   int64_t n4) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
    for (int64_t i0 = ((int64_t)blockIdx.x * blockDim.x) * 4 + threadIdx.x; i0 < n4; i0 += stride) {
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t i = i0 + (int64_t)u * blockDim.x;
            if (i < n4) v[u] = src[i];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t i = i0 + (int64_t)u * blockDim.x;
            if (i < n4) dst[i] = v[u];
        }
    }
}
}  // namespace

hipError_t sdm_launch_mem_init(float* dst, const float* m0, int B, int H, int64_t N, int dv,
                               hipStream_t st) {
    const int64_t per_head4 = N * dv / 4;
    const int64_t rows = m0 ? (int64_t)H : (int64_t)B * H;   // heads, or (b, h) tables
    if (per_head4 == 0 || rows == 0 || B == 0) return hipSuccess;
    // about 8192 blocks in all, at least one per row
    const int64_t per_row = std::max<int64_t>(1, std::min<int64_t>((per_head4 + 1023) / 1024,
                                                                   (8192 + rows - 1) / rows));
    hipLaunchKernelGGL(mem_init_kernel, dim3((unsigned)per_row, (unsigned)rows), dim3(256), 0, st,
                       reinterpret_cast<float4*>(dst), reinterpret_cast<const float4*>(m0), per_head4, B, H);
    return hipGetLastError();
}

namespace {
__global__ void zero_words_kernel(unsigned int* p, int n) {
    if ((int)threadIdx.x < n) p[threadIdx.x] = 0u;
}
}  // namespace

hipError_t sdm_launch_zero_words(void* p, int n, hipStream_t st) {
    hipLaunchKernelGGL(zero_words_kernel, dim3(1), dim3(64), 0, st, static_cast<unsigned int*>(p), n);
    return hipGetLastError();
}

hipError_t sdm_launch_copy(float* dst, const float* src, size_t n, hipStream_t st) {
    const int64_t n4 = (int64_t)(n / 4);
    if (n4 == 0) return hipSuccess;
    const unsigned nb = (unsigned)std::min<int64_t>((n4 + 255) / 256, 8192);
    hipLaunchKernelGGL(copy_kernel, dim3(nb), dim3(256), 0, st, reinterpret_cast<float4*>(dst),
                       reinterpret_cast<const float4*>(src), n4);
    return hipGetLastError();
}
