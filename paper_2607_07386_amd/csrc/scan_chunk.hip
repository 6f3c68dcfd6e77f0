// Chunk-parallel schedule of the forward scan (App. A.1, A.2): the recurrence
// of sdm_scan_fwd computed 64 tokens at a time.  Within a chunk starting from
// the table M0, with lambda_{t,i} the sum of log alpha_s over the chunk's
// tokens s <= t that write slot i (decay only on written rows), the decayed
// innovations x_t = beta_t (v_t - u_t) solve
//   (I + diag(beta) A) x = diag(beta) (V - retrieved),
//   A[t][s]   = sum over slots i written by t and s < t of
//               kappa_t(i) kappa_s(i) exp(lambda_{t,i} - lambda_{s,i}),
//   retrieved_t = sum_n kappa_{t,n} exp(lambda_{t,i_n}) M0[i_n],
// the reads are
//   y_t = sum_m rho_{t,m} exp(lambda_{t,j_m}) M0[j_m] + sum_{s<=t} QK[t][s] x_s,
//   QK[t][s]  = sum over slots j read by t and written by s of
//               rho_t(j) kappa_s(j) exp(lambda_{t,j} - lambda_{s,j}),
// and every slot written in the chunk ends at
//   M[i] = exp(lambda_{C,i}) M0[i] + sum_s kappa_s(i) exp(lambda_{C,i} - lambda_{s,i}) x_s.
//
// Two kernels.  chunk_coef_kernel (one workgroup per stream and chunk, all
// chunks at once) needs only the slot lists and gates: it sorts the chunk's
// write entries by (slot, token), takes lambda as a running sum along each
// slot's entries, accumulates A and QK from the pairs inside a slot's entries,
// inverts the unit lower-triangular system into L = (I + diag(beta) A)^-1
// diag(beta), and stores L, QK, the gather weights and the per-slot scatter
// lists as one record per chunk.  chunk_scan_kernel (one workgroup per stream
// and 32-column slice, or 16 when forced) walks the chunks in order: gathers of
// retrieved and of the reads' first term from the chunk-start table,
// x = L (V - retrieved) and y = inter + QK x from LDS, then one store of every
// written slot.  The host side runs both over chunk ranges so that the
// coefficients of the next range overlap the scan of the current one.
#include "sdm_common.h"
#include "sdm_internal.h"

namespace {

constexpr int CC = SDM_CHUNK;       // tokens per chunk
constexpr int CT1 = 256;            // threads of the coefficient kernel
static_assert(CT1 == 4 * CC, "the substitution takes one quad of threads per column of L");
// The scan kernel takes COLS = 32 or 16 columns per workgroup (a 128- or
// 64-byte piece of every row), with one thread per (token, column quad).
template <int COLS>
constexpr int scan_threads() { return CC * COLS / 4; }
constexpr int LDP = CC + 1;         // padded row stride of L and QK in LDS
constexpr int CK_LDS_LIMIT = 160 * 1024;

// Per-chunk record: nseg, then L and QK [C][C], the gather weights
// exp(lambda) kappa [C][W] and exp(lambda) rho [C][R], then per written slot
// (sorted by id) its first entry, id and decay exp(lambda_C), per entry
// (sorted by slot, then token) its token and scatter weight, and per written
// slot one 16-byte unit {id, first entry as (token W + list position) with
// bit 30 set when the slot has further entries, decay, that entry's scatter
// weight} (the narrow kernel's scatter reads one unit per slot).
struct ChunkRec {
    int off_l, off_qk, off_cr, off_cy, off_sbeg, off_sslot, off_sdec, off_etok, off_ecoef, off_sinfo, bytes;
};

__host__ __device__ inline ChunkRec chunk_rec_layout(int W, int R) {
    ChunkRec r;
    const int E = CC * W;
    int o = 16;
    r.off_l = o;     o += CC * CC * 4;
    r.off_qk = o;    o += CC * CC * 4;
    r.off_cr = o;    o += CC * W * 4;
    r.off_cy = o;    o += CC * R * 4;
    r.off_sbeg = o;  o += (E + 1) * 4;
    o = (o + 15) & ~15;
    r.off_sslot = o; o += E * 4;
    r.off_sdec = o;  o += E * 4;
    r.off_etok = o;  o += E * 4;
    r.off_ecoef = o; o += E * 4;
    r.off_sinfo = o; o += E * 16;
    r.bytes = (o + 255) & ~255;
    return r;
}

// Sort length of the coefficient kernel: a power of two, at least one key per thread.
inline int pow2_at_least(int x) {
    int p = CT1;
    while (p < x) p <<= 1;
    return p;
}

inline size_t coef_lds_bytes(int W) {
    const int P = pow2_at_least(CC * W);
    return (size_t)P * 8 + (size_t)3 * CC * W * 4 + (size_t)3 * CC * CC * 4 + 2 * CC * 4 + (CT1 + 1) * 4;
}

__device__ __forceinline__ unsigned long long key_slot(unsigned long long k) { return k >> 16; }
__device__ __forceinline__ int key_tok(unsigned long long k) { return (int)((k >> 8) & 255); }
__device__ __forceinline__ int key_ent(unsigned long long k) { return (int)(k & 255); }

// One stage (block size KB, distance J) of the ascending bitonic network over
// CT1 K keys, thread t holding keys [t K, t K + K): J < K compares a thread's
// own keys, J < 64 K exchanges with lane ^ (J / K) of the same wave, larger J
// goes through LDS (keys[] as the exchange buffer).
template <int K, int KB, int J>
__device__ __forceinline__ void sort_stage(unsigned long long (&kr)[K], unsigned long long* keys, int tid) {
    if constexpr (J < K) {
#pragma unroll
        for (int r = 0; r < K; ++r) {
            if ((r & J) == 0) {
                const bool up = ((tid * K + r) & KB) == 0;
                const unsigned long long a = kr[r], b = kr[r + J];
                const bool sw = (a > b) == up;
                kr[r] = sw ? b : a;
                kr[r + J] = sw ? a : b;
            }
        }
    } else {
        unsigned long long o[K];
        if constexpr (J < 64 * K) {
#pragma unroll
            for (int r = 0; r < K; ++r)
                o[r] = ((unsigned long long)xor_lane<J / K>((uint32_t)(kr[r] >> 32)) << 32) |
                       xor_lane<J / K>((uint32_t)kr[r]);
        } else {
#pragma unroll
            for (int r = 0; r < K; ++r) keys[tid * K + r] = kr[r];
            __syncthreads();
#pragma unroll
            for (int r = 0; r < K; ++r) o[r] = keys[(tid * K + r) ^ J];
            __syncthreads();
        }
        // the lower index of a pair keeps the minimum in ascending blocks
        const bool keep_min = (((tid * K) & J) == 0) == (((tid * K) & KB) == 0);
#pragma unroll
        for (int r = 0; r < K; ++r) {
            const unsigned long long a = kr[r];
            kr[r] = keep_min ? (o[r] < a ? o[r] : a) : (o[r] > a ? o[r] : a);
        }
    }
    if constexpr (J > 1) sort_stage<K, KB, J / 2>(kr, keys, tid);
    else if constexpr (KB < CT1 * K) sort_stage<K, KB * 2, KB>(kr, keys, tid);
}

// The chunk's write entries as sort keys (slot, token, entry), sorted
// ascending into keys[0 .. CT1 K) (entries past E: all-ones keys, last), with
// kappa per entry into kap[].  Returns the out-of-range id flag (ids clamped).
template <int K>
__device__ unsigned int sorted_write_keys(const int32_t* __restrict__ w_idx, const float* __restrict__ w_val,
                                          size_t tok0, int W, int E, int64_t N, float* kap,
                                          unsigned long long* keys) {
    const int tid = threadIdx.x;
    unsigned int bad = 0;
    unsigned long long kr[K];
#pragma unroll
    for (int r = 0; r < K; ++r) {
        const int e = tid * K + r;
        unsigned long long key = ~0ull;
        if (e < E) {
            const int t = e / W, j = e - t * W;
            int64_t id = w_idx[(tok0 + t) * W + j];
            if (id < 0 || id >= N) {
                bad |= 1u;
                id = id < 0 ? 0 : N - 1;
            }
            key = ((unsigned long long)id << 16) | (unsigned long long)(t << 8) | (unsigned long long)j;
            kap[e] = w_val[(tok0 + t) * W + j];
        }
        kr[r] = key;
    }
    sort_stage<K, 2, 1>(kr, keys, tid);
#pragma unroll
    for (int r = 0; r < K; ++r) keys[tid * K + r] = kr[r];
    return bad;
}

// One read entry (token t, position m, slot id, weight rho) whose slot's first
// sorted key is at lo: the slot's decay after token t, the gather weight, and
// its QK terms from the slot's writers up to t.
__device__ __forceinline__ void read_side_entry(const unsigned long long* keys, const float* kap, const float* lams,
                                                float* QK, float* g_cy, int E, int W, int R, int t, int m,
                                                int64_t id, float rho, int lo) {
    int last = lo - 1;
    while (last + 1 < E && key_slot(keys[last + 1]) == (unsigned long long)id && key_tok(keys[last + 1]) <= t)
        ++last;
    const float lr = last >= lo ? lams[last] : 0.f;
    g_cy[t * R + m] = rho * expf(lr);
    for (int f = lo; f <= last; ++f) {
        const unsigned long long kf = keys[f];
        atomicAdd(&QK[t * CC + key_tok(kf)], rho * kap[key_tok(kf) * W + key_ent(kf)] * expf(lr - lams[f]));
    }
}

template <typename VT>
__global__ __launch_bounds__(CT1) void chunk_coef_kernel(
    const int32_t* __restrict__ w_idx, const float* __restrict__ w_val, const int32_t* __restrict__ r_idx,
    const float* __restrict__ r_val, const VT* __restrict__ alpha, const VT* __restrict__ beta, int T, int W,
    int R, int64_t N, int nch, int cb, int ncr, int P, unsigned char* __restrict__ recs,
    unsigned int* __restrict__ err, const float* __restrict__ gA, const float* __restrict__ gbdt, int H) {
    // chunks [cb, cb + ncr) of every stream
    extern __shared__ __align__(16) unsigned char smem[];
    const ChunkRec L = chunk_rec_layout(W, R);
    const int tid = threadIdx.x;
    const int s = blockIdx.x / ncr, c = cb + (blockIdx.x - s * ncr);
    const int t0 = c * CC, n = min(CC, T - t0);
    const int E = n * W;
    const size_t tok0 = (size_t)s * T + t0;

    unsigned long long* keys = reinterpret_cast<unsigned long long*>(smem);   // [P]
    float* kap = reinterpret_cast<float*>(keys + P);    // [C*W] kappa at (t, n)
    float* lamw = kap + CC * W;                          // [C*W] lambda at (t, n)
    float* lams = lamw + CC * W;                         // [C*W] lambda in sorted order
    float* A = lams + CC * W;                            // [C][C]
    float* QK = A + CC * CC;                             // [C][C]
    float* Lm = QK + CC * CC;                            // [C][C]
    float* la = Lm + CC * CC;                            // [C] log alpha
    float* bt = la + CC;                                 // [C] beta
    int* cnt = reinterpret_cast<int*>(bt + CC);          // [CT1 + 1]

    unsigned char* rec = recs + ((size_t)s * nch + c) * L.bytes;
    float* g_cr = reinterpret_cast<float*>(rec + L.off_cr);
    float* g_cy = reinterpret_cast<float*>(rec + L.off_cy);
    int* g_sbeg = reinterpret_cast<int*>(rec + L.off_sbeg);
    int* g_sslot = reinterpret_cast<int*>(rec + L.off_sslot);
    float* g_sdec = reinterpret_cast<float*>(rec + L.off_sdec);
    int* g_etok = reinterpret_cast<int*>(rec + L.off_etok);
    int4* g_sinfo = reinterpret_cast<int4*>(rec + L.off_sinfo);
    float* g_ecoef = reinterpret_cast<float*>(rec + L.off_ecoef);

    // ---- write entries as sort keys (slot, token, entry), sorted ascending ----
    unsigned int bad;
    switch (P / CT1) {
        case 1: bad = sorted_write_keys<1>(w_idx, w_val, tok0, W, E, N, kap, keys); break;
        case 2: bad = sorted_write_keys<2>(w_idx, w_val, tok0, W, E, N, kap, keys); break;
        case 4: bad = sorted_write_keys<4>(w_idx, w_val, tok0, W, E, N, kap, keys); break;
        case 8: bad = sorted_write_keys<8>(w_idx, w_val, tok0, W, E, N, kap, keys); break;
        default: bad = sorted_write_keys<16>(w_idx, w_val, tok0, W, E, N, kap, keys); break;
    }
    // ---- gates ----
    for (int t = tid; t < CC; t += CT1) {
        float lg = 0.f, b = 0.f;
        if (t < n) {
            const float a = to_f32(alpha[tok0 + t]);
            b = to_f32(beta[tok0 + t]);
            if (gA) {   // pre-activations: log alpha = -A softplus(a + b_dt) directly
                lg = sdm_log_alpha(gA, gbdt, s % H, a);
                b = sdm_sigmoid(b);
            } else {
                if (!(a > 0.f)) bad |= 2u;   // the log form needs alpha > 0
                lg = logf(fmaxf(a, 1e-30f));
            }
        }
        la[t] = lg;
        bt[t] = b;
    }
    for (int i = tid; i < 2 * CC * CC / 4; i += CT1)   // A, QK (L is written whole below)
        reinterpret_cast<float4*>(A)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();

    // ---- lambda: running sum of log alpha along each slot's entries (token order) ----
    for (int e = tid; e < E; e += CT1) {
        const unsigned long long ke = keys[e];
        float sum = la[key_tok(ke)];
        for (int f = e - 1; f >= 0 && key_slot(keys[f]) == key_slot(ke); --f) sum += la[key_tok(keys[f])];
        lams[e] = sum;
        lamw[key_tok(ke) * W + key_ent(ke)] = sum;
    }
    __syncthreads();

    // ---- segments (one per distinct written slot), numbered in sorted order ----
    const int ept = (E + CT1 - 1) / CT1;
    const int e0 = min(E, tid * ept), e1 = min(E, e0 + ept);
    int ns = 0;
    for (int e = e0; e < e1; ++e) ns += (e == 0 || key_slot(keys[e]) != key_slot(keys[e - 1])) ? 1 : 0;
    // exclusive prefix of ns over the threads: within the wave by lane shifts,
    // then the totals of the earlier waves
    int incl = ns;
    const int lane = tid & (SDM_WAVE - 1), wave = tid / SDM_WAVE;
#pragma unroll
    for (int d = 1; d < SDM_WAVE; d <<= 1) {
        const int up = __shfl_up(incl, d, SDM_WAVE);
        if (lane >= d) incl += up;
    }
    if (lane == SDM_WAVE - 1) cnt[wave] = incl;
    __syncthreads();
    int before = 0, nseg = 0;
#pragma unroll
    for (int w = 0; w < CT1 / SDM_WAVE; ++w) {
        before += w < wave ? cnt[w] : 0;
        nseg += cnt[w];
    }
    {
        int g = before + incl - ns;
        for (int e = e0; e < e1; ++e) {
            if (!(e == 0 || key_slot(keys[e]) != key_slot(keys[e - 1]))) continue;
            int f = e;
            while (f + 1 < E && key_slot(keys[f + 1]) == key_slot(keys[e])) ++f;
            g_sbeg[g] = e;
            const int slot = (int)key_slot(keys[e]);
            const float dec = expf(lams[f]);
            g_sslot[g] = slot;
            g_sdec[g] = dec;
            const int ft = key_tok(keys[e]), fn = key_ent(keys[e]);
            const float fc = kap[ft * W + fn] * expf(lams[f] - lams[e]);   // = the entry's scatter weight
            g_sinfo[g] = make_int4(slot, (ft * W + fn) | (f > e ? (1 << 30) : 0), __float_as_int(dec),
                                   __float_as_int(fc));
            ++g;
        }
        if (tid == CT1 - 1) {
            g_sbeg[nseg] = E;
            *reinterpret_cast<int*>(rec) = nseg;
        }
    }

    // ---- per entry: scatter weight, and A from every earlier writer of the slot ----
    for (int e = tid; e < E; e += CT1) {
        const unsigned long long ke = keys[e];
        const unsigned long long se = key_slot(ke);
        int f = e;
        while (f + 1 < E && key_slot(keys[f + 1]) == se) ++f;
        const int t = key_tok(ke);
        const float kt = kap[t * W + key_ent(ke)], le = lams[e];
        g_etok[e] = t;
        g_ecoef[e] = kt * expf(lams[f] - le);
        for (int g = e - 1; g >= 0 && key_slot(keys[g]) == se; --g) {
            const unsigned long long kg = keys[g];
            atomicAdd(&A[t * CC + key_tok(kg)], kt * kap[key_tok(kg) * W + key_ent(kg)] * expf(le - lams[g]));
        }
    }
    // ---- gather weights of the write side ----
    for (int e = tid; e < E; e += CT1) g_cr[e] = kap[e] * expf(lamw[e]);
    // ---- read side: lambda of the read slot after token t, gather weight, QK.
    //      Entries go RB at a time, their searches interleaved: the first key of
    //      the slot by a branch-free lower bound over the P sorted keys (the
    //      padding keys past E sort last and are never below an id) ----
    constexpr int RB = 4;
    for (int e0 = tid; e0 < n * R; e0 += RB * CT1) {
        int64_t ids[RB];
        int pos[RB];
#pragma unroll
        for (int b = 0; b < RB; ++b) {
            const int e = min(e0 + b * CT1, n * R - 1);
            const int t = e / R, m = e - t * R;
            int64_t id = r_idx[(tok0 + t) * R + m];
            if (id < 0 || id >= N) {
                bad |= 1u;
                id = id < 0 ? 0 : N - 1;
            }
            ids[b] = id;
            pos[b] = 0;
        }
        for (int step = P >> 1; step >= 1; step >>= 1) {
#pragma unroll
            for (int b = 0; b < RB; ++b)
                if (key_slot(keys[pos[b] + step - 1]) < (unsigned long long)ids[b]) pos[b] += step;
        }
#pragma unroll
        for (int b = 0; b < RB; ++b) {
            const int e = e0 + b * CT1;
            if (e >= n * R) break;
            const int t = e / R, m = e - t * R;
            const int64_t id = ids[b];
            const float rho = r_val[(tok0 + t) * R + m];
            const int lo = pos[b];
            read_side_entry(keys, kap, lams, QK, g_cy, E, W, R, t, m, id, rho, lo);
        }
    }
    __syncthreads();

    // ---- L = (I + diag(beta) A)^-1 diag(beta) by forward substitution over rows,
    //      L[t][c] = beta_t (delta_tc - sum_{u<t} A[t][u] L[u][c]): column c on the
    //      4 lanes of a quad, lane p holding rows [16 p, 16 p + 16) in registers;
    //      each row's sum is 4 partial sums added across the quad.  A is zero on
    //      and above the diagonal and rows not yet formed are zero, so every step
    //      takes all 16 terms.  beta is 0 past the chunk's tokens, so those rows
    //      and columns come out zero. ----
    {
        const int cc = tid >> 2, p = tid & 3;
        float lr[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) lr[i] = 0.f;
#pragma unroll
        for (int t = 0; t < CC; ++t) {
            const float4* arow = reinterpret_cast<const float4*>(A + t * CC + 16 * p);
            float pr[16];
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
                const float4 a4 = arow[i4];
                pr[4 * i4] = a4.x * lr[4 * i4];
                pr[4 * i4 + 1] = a4.y * lr[4 * i4 + 1];
                pr[4 * i4 + 2] = a4.z * lr[4 * i4 + 2];
                pr[4 * i4 + 3] = a4.w * lr[4 * i4 + 3];
            }
#pragma unroll
            for (int h = 8; h >= 1; h >>= 1)   // pairwise: a short dependent chain per row
#pragma unroll
                for (int i = 0; i < h; ++i) pr[i] += pr[i + h];
            float part = pr[0];
            part += xor_lane_f(part, 1);
            part += xor_lane_f(part, 2);
            const float val = bt[t] * ((t == cc ? 1.f : 0.f) - part);
            if (p == (t >> 4)) lr[t & 15] = val;
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) Lm[(16 * p + i) * CC + cc] = lr[i];
    }
    __syncthreads();
    {
        float4* gl = reinterpret_cast<float4*>(rec + L.off_l);     // L then QK, contiguous
        float4* gq = reinterpret_cast<float4*>(rec + L.off_qk);
        const float4* sl = reinterpret_cast<const float4*>(Lm);
        const float4* sq = reinterpret_cast<const float4*>(QK);
        for (int i = tid; i < CC * CC / 4; i += CT1) {
            gl[i] = sl[i];
            gq[i] = sq[i];
        }
    }
    if (bad) atomicOr(err, bad);
}

// LDS of the scan kernel beyond its static arrays: the chunk's slot ids and
// gather weights, and (SEG) its scatter lists.
inline size_t scan_dyn_lds(int W, int R, bool seg) {
    const ChunkRec L = chunk_rec_layout(W, R);
    size_t b = (size_t)CC * (W + R) * 8;
    if (seg) b += (size_t)(L.off_ecoef + CC * W * 4 - L.off_sbeg);
    return b;
}

constexpr int GB = 32;   // row gathers in flight per thread
constexpr int SB = 8;    // scatter rows in flight per thread
// Scatter lists staged in LDS up to this many bytes (the largest that fits the
// LDS limit beside the rest); longer lists are read from the record.
constexpr int SEG_LDS_MAX = 80 * 1024;

template <typename VT, bool SEG, int COLS>
__global__ __launch_bounds__(scan_threads<COLS>()) void chunk_scan_kernel(const int32_t* __restrict__ w_idx,
                                                         const int32_t* __restrict__ r_idx, const VT* __restrict__ v,
                                                         float* __restrict__ mem, float* __restrict__ y,
                                                         const unsigned char* __restrict__ recs, int T, int W, int R,
                                                         int64_t N, int dv, int nch, int cb, int ce, int nslice) {
    // chunks [cb, ce) of the stream, in order
    constexpr int CT2 = scan_threads<COLS>();
    constexpr int CCOLS = COLS;
    constexpr int QPR = COLS / 4;    // column quads per row piece
    // staging loads per thread: gather weights (float4), slot ids per side, scatter lists (float4)
    constexpr int ST_CF = CC * 2 * SDM_CHUNK_MAX_LIST / 4 / CT2;
    constexpr int ST_ID = CC * SDM_CHUNK_MAX_LIST / CT2;
    constexpr int ST_SEG = SEG_LDS_MAX / 16 / CT2;
    constexpr int SEG_RB = ST_SEG < 10 ? ST_SEG : 10;   // scatter-list float4s in registers per round
    __shared__ float Ls[CC * LDP];
    __shared__ float Qs[CC * LDP];
    __shared__ __align__(16) float Rr[CC * CCOLS];
    __shared__ __align__(16) float Xs[CC * CCOLS];
    extern __shared__ __align__(16) unsigned char dyn[];
    const ChunkRec L = chunk_rec_layout(W, R);
    const int WR = W + R;
    int* sid = reinterpret_cast<int*>(dyn);                    // [C][W] write ids, then [C][R] read ids
    float* scf = reinterpret_cast<float*>(sid + CC * WR);      // [C][W] then [C][R] gather weights
    unsigned char* sseg = reinterpret_cast<unsigned char*>(scf + CC * WR);   // scatter lists (SEG)
    const int seg_bytes = L.off_ecoef + CC * W * 4 - L.off_sbeg;

    const int tid = threadIdx.x;
    const int s = blockIdx.x / nslice, sl = blockIdx.x - s * nslice;
    const int q = tid % QPR;                // column quad within the slice
    const int tl = tid / QPR;               // token within the chunk
    const int col = sl * CCOLS + q * 4;
    const bool colok = col < dv;
    float* ms = mem + (size_t)s * N * dv;

    for (int c = cb; c < ce; ++c) {
        const unsigned char* rec = recs + ((size_t)s * nch + c) * L.bytes;
        const int t0 = c * CC, n = min(CC, T - t0);
        const size_t tk0 = (size_t)s * T + t0;
        // ---- stage the chunk's record and slot ids: every load first, then the LDS stores ----
        {
            const float4* gl = reinterpret_cast<const float4*>(rec + L.off_l);
            const float4* gq = reinterpret_cast<const float4*>(rec + L.off_qk);
            const float4* gcf = reinterpret_cast<const float4*>(rec + L.off_cr);   // [C][W] then [C][R]
            const float4* gsg = reinterpret_cast<const float4*>(rec + L.off_sbeg);
            const int ncf = CC * WR / 4, nsg = SEG ? seg_bytes / 16 : 0;
            float4 la[CC * CC / 4 / CT2], qa[CC * CC / 4 / CT2], cf[ST_CF], sg[SEG_RB];
            int iw[ST_ID], ir[ST_ID];
#pragma unroll
            for (int k = 0; k < CC * CC / 4 / CT2; ++k) {
                la[k] = gl[tid + k * CT2];
                qa[k] = gq[tid + k * CT2];
            }
            // unconditional loads at clamped (valid) indices keep these arrays in
            // registers; only the stores below are guarded
#pragma unroll
            for (int k = 0; k < ST_CF; ++k) cf[k] = gcf[min(tid + k * CT2, ncf - 1)];
#pragma unroll
            for (int k = 0; k < ST_ID; ++k) {
                const int i = tid + k * CT2;
                iw[k] = w_idx[tk0 * W + min(i, n * W - 1)];
                ir[k] = r_idx[tk0 * R + min(i, n * R - 1)];
            }
            if constexpr (SEG) {
#pragma unroll
                for (int k = 0; k < SEG_RB; ++k) sg[k] = gsg[min(tid + k * CT2, nsg - 1)];
            }
#pragma unroll
            for (int k = 0; k < CC * CC / 4 / CT2; ++k) {
                const int i = tid + k * CT2;
                const int r = (4 * i) / CC, c4 = (4 * i) % CC;
                float* lrow = Ls + r * LDP + c4;
                float* qrow = Qs + r * LDP + c4;
                lrow[0] = la[k].x; lrow[1] = la[k].y; lrow[2] = la[k].z; lrow[3] = la[k].w;
                qrow[0] = qa[k].x; qrow[1] = qa[k].y; qrow[2] = qa[k].z; qrow[3] = qa[k].w;
            }
#pragma unroll
            for (int k = 0; k < ST_CF; ++k)
                if (tid + k * CT2 < ncf) reinterpret_cast<float4*>(scf)[tid + k * CT2] = cf[k];
#pragma unroll
            for (int k = 0; k < ST_ID; ++k) {
                const int i = tid + k * CT2;
                if (i < n * W) sid[i] = (int)(iw[k] < 0 ? 0 : (iw[k] >= N ? N - 1 : iw[k]));
                if (i < n * R) sid[CC * W + i] = (int)(ir[k] < 0 ? 0 : (ir[k] >= N ? N - 1 : ir[k]));
            }
            if constexpr (SEG) {
                // scatter lists: SEG_RB float4 per thread with the loads above,
                // the rest in further rounds of SEG_RB
#pragma unroll
                for (int k = 0; k < SEG_RB; ++k)
                    if (tid + k * CT2 < nsg) reinterpret_cast<float4*>(sseg)[tid + k * CT2] = sg[k];
                for (int k0 = SEG_RB; k0 < ST_SEG; k0 += SEG_RB) {
#pragma unroll
                    for (int k = 0; k < SEG_RB; ++k) sg[k] = gsg[min(tid + (k0 + k) * CT2, nsg - 1)];
#pragma unroll
                    for (int k = 0; k < SEG_RB; ++k)
                        if (tid + (k0 + k) * CT2 < nsg) reinterpret_cast<float4*>(sseg)[tid + (k0 + k) * CT2] = sg[k];
                }
            }
        }
        __syncthreads();
        // ---- gathers from the chunk-start table, GB rows in flight ----
        float4 inter = make_float4(0.f, 0.f, 0.f, 0.f);
        float4 rr = make_float4(0.f, 0.f, 0.f, 0.f);
        if (tl < n && colok) {
            float4 ret = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int j0 = 0; j0 < WR; j0 += GB) {
                float4 m[GB];
#pragma unroll
                for (int jj = 0; jj < GB; ++jj) {
                    const int j = j0 + jj;
                    // past the lists: row 0 (in bounds, unused)
                    const int id = j < W ? sid[tl * W + j] : (j < WR ? sid[CC * W + tl * R + (j - W)] : 0);
                    m[jj] = load4(ms + (size_t)id * dv + col);
                }
#pragma unroll
                for (int jj = 0; jj < GB; ++jj) {
                    const int j = j0 + jj;
                    if (j < W) {
                        const float w = scf[tl * W + j];
                        ret.x += w * m[jj].x; ret.y += w * m[jj].y; ret.z += w * m[jj].z; ret.w += w * m[jj].w;
                    } else if (j < WR) {
                        const float w = scf[CC * W + tl * R + (j - W)];
                        inter.x += w * m[jj].x; inter.y += w * m[jj].y; inter.z += w * m[jj].z; inter.w += w * m[jj].w;
                    }
                }
            }
            const float4 vv = load4(v + (tk0 + tl) * dv + col);
            rr = make_float4(vv.x - ret.x, vv.y - ret.y, vv.z - ret.z, vv.w - ret.w);
        }
        *reinterpret_cast<float4*>(&Rr[tl * CCOLS + q * 4]) = rr;
        __syncthreads();
        // ---- x = L (V - retrieved) ----
        // (L and QK are zero above the diagonal and past the chunk's tokens, and
        // Rr past them: the products run over all C columns, unrolled)
        {
            float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 16
            for (int u = 0; u < CC; ++u) {
                const float l = Ls[tl * LDP + u];
                const float4 r = *reinterpret_cast<const float4*>(&Rr[u * CCOLS + q * 4]);
                acc.x += l * r.x; acc.y += l * r.y; acc.z += l * r.z; acc.w += l * r.w;
            }
            *reinterpret_cast<float4*>(&Xs[tl * CCOLS + q * 4]) = acc;
        }
        __syncthreads();
        // ---- y = inter + QK x ----
        if (tl < n && colok) {
            float4 acc = inter;
#pragma unroll 16
            for (int u = 0; u < CC; ++u) {
                const float w = Qs[tl * LDP + u];
                const float4 x = *reinterpret_cast<const float4*>(&Xs[u * CCOLS + q * 4]);
                acc.x += w * x.x; acc.y += w * x.y; acc.z += w * x.z; acc.w += w * x.w;
            }
            *reinterpret_cast<float4*>(y + (tk0 + tl) * dv + col) = acc;
        }
        // ---- one store per written slot: decayed chunk-start row plus its tokens' x ----
        {
            // the lists in LDS (SEG) or in the record
            const unsigned char* sb = SEG ? sseg : rec + L.off_sbeg;
            const int nseg = *reinterpret_cast<const int*>(rec);
            const int* sbeg = reinterpret_cast<const int*>(sb);
            const int* sslot = reinterpret_cast<const int*>(sb + (L.off_sslot - L.off_sbeg));
            const float* sdec = reinterpret_cast<const float*>(sb + (L.off_sdec - L.off_sbeg));
            const int* etok = reinterpret_cast<const int*>(sb + (L.off_etok - L.off_sbeg));
            const float* ecoef = reinterpret_cast<const float*>(sb + (L.off_ecoef - L.off_sbeg));
            if (colok) {
                for (int g0 = tl; g0 < nseg; g0 += SB * CC) {
                    float4 m[SB];
#pragma unroll
                    for (int b = 0; b < SB; ++b) {
                        const int g = g0 + b * CC;
                        // past the last segment: reload segment g0's row (in bounds, unused)
                        m[b] = load4(ms + (size_t)sslot[g < nseg ? g : g0] * dv + col);
                    }
                    // every segment has a first entry: the batch takes those together,
                    // then any further entries of its segments
                    int fb[SB];
                    float4 acc[SB];
#pragma unroll
                    for (int b = 0; b < SB; ++b) {
                        const int g = min(g0 + b * CC, nseg - 1);
                        fb[b] = sbeg[g];
                        const float d = sdec[g], w = ecoef[fb[b]];
                        const float4 x = *reinterpret_cast<const float4*>(&Xs[etok[fb[b]] * CCOLS + q * 4]);
                        acc[b] = make_float4(d * m[b].x + w * x.x, d * m[b].y + w * x.y, d * m[b].z + w * x.z,
                                             d * m[b].w + w * x.w);
                    }
#pragma unroll
                    for (int b = 0; b < SB; ++b) {
                        const int g = g0 + b * CC;
                        if (g < nseg) {
                            const int fe = sbeg[g + 1];
                            int f = fb[b] + 1;
                            for (; f < fe; ++f) {
                                const float w = ecoef[f];
                                const float4 x = *reinterpret_cast<const float4*>(&Xs[etok[f] * CCOLS + q * 4]);
                                acc[b].x += w * x.x; acc[b].y += w * x.y; acc[b].z += w * x.z; acc[b].w += w * x.w;
                            }
                            *reinterpret_cast<float4*>(ms + (size_t)sslot[g] * dv + col) = acc[b];
                        }
                    }
                }
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Narrow variant for few streams: one workgroup per (stream, 8-column slice),
// 512 threads, so a stream of d_v = 128 takes 16 workgroups and the chip fills
// at 16 streams.  The 16 workgroups of a stream are placed on one XCD (ids
// congruent mod 8) and read the chunk's record through its L2.  Per chunk:
//   staging   slot ids and gather weights straight to registers (each thread
//             its token's rows of its part), L and QK, v, and this thread's
//             scatter units; none of it depends on an earlier chunk, so chunk
//             c + 1's is loaded while chunk c computes and scatters;
//   gather    thread (token, part p, quad q) loads rows [NPR p, NPR (p + 1))
//             of its token, NPR pieces of 16 bytes in flight, and sums them
//             with their weights; the 4 parts add across lanes;
//   products  thread (token, column): R = v - retrieved, x = L R, y = inter + QK x;
//   scatter   thread holds SBN (segment, quad) units: one load each, one store.
// Every load of a round is issued before its first use, so a chunk costs two
// dependent memory round trips on its path: the gather, and the stores that
// the next chunk's gather must see.
constexpr int NCOL = 8;                 // columns per workgroup
constexpr int NT3 = 512;                // threads
constexpr int NPART = 4;                // row parts per (token, quad) in the gather
constexpr int SB3 = 8;                  // scatter units in flight per thread
constexpr int NLQ = CC * CC / 4 / NT3;  // float4 of L (and of QK) per thread
constexpr int LDN = CC + 4;             // row stride of L, QK and the column-major R, x in
                                        // LDS: 16-byte rows, 8 rows on distinct banks

// Column of the product mapping (token tid / 8): the lane order of the
// gather's (part p, quad q) pairs, 2 p + q -> column 4 q + p, so that a
// gather lane's cross-lane sums are already its product column's.
__device__ __forceinline__ int narrow_pc(int tid) { return 4 * (tid & 1) + ((tid >> 1) & 3); }
__device__ __forceinline__ float4 f4_add_lanes(float4 a) {   // sum over lane bits 1 and 2
    auto add = [](float x) {
        x += __uint_as_float(xor_lane<2>(__float_as_uint(x)));
        return x + __uint_as_float(xor_lane<4>(__float_as_uint(x)));
    };
    return make_float4(add(a.x), add(a.y), add(a.z), add(a.w));
}
__device__ __forceinline__ float f4_elem(float4 a, int e) { return e == 0 ? a.x : e == 1 ? a.y : e == 2 ? a.z : a.w; }

// One chunk's staged registers (see above).
template <int NPR, int SBN>
struct NarrowStage {
    int id[NPR];
    float wt[NPR];
    float4 la[NLQ], qa[NLQ];
    float vv;
    int4 sg[SBN];   // {slot, first entry | flags, decay, first entry's weight}
    int nseg;
};

// Loads chunk c's staging.  VEC: W and R multiples of 4 and 16-byte aligned
// slot lists, so a part's ids and weights go as 16-byte loads.  The scatter
// units are loaded up to the record's capacity (C W), whatever the chunk's
// segment count: units past it are never used.
template <typename VT, int NPR, int SBN, bool VEC>
__device__ __forceinline__ void narrow_stage(NarrowStage<NPR, SBN>& st, const int32_t* __restrict__ w_idx,
                                             const int32_t* __restrict__ r_idx, const VT* __restrict__ v,
                                             const unsigned char* __restrict__ recs, const ChunkRec& L, int s,
                                             int c, int nch, int T, int W, int R, int64_t N, int dv, int col0) {
    const int tid = threadIdx.x;
    const int gt = tid >> 3, gp = (tid >> 1) & 3;
    const int pt = tid >> 3, pc = narrow_pc(tid);
    const unsigned char* rec = recs + ((size_t)s * nch + c) * L.bytes;
    const int t0 = c * CC, n = min(CC, T - t0);
    const size_t tk0 = (size_t)s * T + t0;
    const int WR = W + R;
    const int tg = min(gt, n - 1);            // past the chunk's tokens: token n - 1 (unused)
    const float* g_cr = reinterpret_cast<const float*>(rec + L.off_cr);
    const float* g_cy = reinterpret_cast<const float*>(rec + L.off_cy);
    if constexpr (VEC) {
#pragma unroll
        for (int k = 0; k < NPR; k += 4) {
            const int j = gp * NPR + k;       // a group of 4 lies in one list (W % 4 == 0)
            const bool wr = j < W, rd = !wr && j < WR;
            const int jr = rd ? j - W : 0;
            const int4 x = wr ? *reinterpret_cast<const int4*>(w_idx + (tk0 + tg) * W + j)
                              : *reinterpret_cast<const int4*>(r_idx + (tk0 + tg) * R + jr);
            const float4 w = wr ? *reinterpret_cast<const float4*>(g_cr + tg * W + j)
                                : *reinterpret_cast<const float4*>(g_cy + tg * R + jr);
            const int xs[4] = {x.x, x.y, x.z, x.w};
            const float ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t xi = xs[u];
                st.id[k + u] = (int)(xi < 0 ? 0 : (xi >= N ? N - 1 : xi));
                st.wt[k + u] = (wr || rd) ? ws[u] : 0.f;
            }
        }
    } else {
#pragma unroll
        for (int k = 0; k < NPR; ++k) {
            const int j = gp * NPR + k;
            const bool wr = j < W;
            const int jr = wr ? j : min(j - W, R - 1);
            const int64_t x = wr ? w_idx[(tk0 + tg) * W + j] : r_idx[(tk0 + tg) * R + jr];
            st.id[k] = (int)(x < 0 ? 0 : (x >= N ? N - 1 : x));
            st.wt[k] = j < WR ? (wr ? g_cr[tg * W + j] : g_cy[tg * R + jr]) : 0.f;
        }
    }
    const float4* gl = reinterpret_cast<const float4*>(rec + L.off_l);
    const float4* gq4 = reinterpret_cast<const float4*>(rec + L.off_qk);
#pragma unroll
    for (int k = 0; k < NLQ; ++k) {
        st.la[k] = gl[tid + k * NT3];
        st.qa[k] = gq4[tid + k * NT3];
    }
    st.vv = to_f32(v[(tk0 + min(pt, n - 1)) * dv + col0 + pc]);
    const int4* g_sinfo = reinterpret_cast<const int4*>(rec + L.off_sinfo);
    const int gmax = CC * W - 1;
#pragma unroll
    for (int b = 0; b < SBN; ++b) st.sg[b] = g_sinfo[min((tid + NT3 * b) >> 1, gmax)];
    st.nseg = *reinterpret_cast<const int*>(rec);
}

template <typename VT, int NPR, int SBN, bool REUSE, bool VEC>
__global__ __launch_bounds__(NT3) void chunk_scan_narrow_kernel(
    const int32_t* __restrict__ w_idx, const int32_t* __restrict__ r_idx, const VT* __restrict__ v,
    float* __restrict__ mem, float* __restrict__ y, const unsigned char* __restrict__ recs, int T, int W, int R,
    int64_t N, int dv, int nch, int cb, int ce, int nslice) {
    __shared__ __align__(16) float Ls[CC * LDN];
    __shared__ __align__(16) float Qs[CC * LDN];
    __shared__ __align__(16) float RrT[NCOL * LDN];   // R by column
    __shared__ __align__(16) float XsT[NCOL * LDN];   // x by column (the y product)
    __shared__ __align__(16) float Xs[CC * NCOL];     // x by token (the scatter)
    // REUSE: the gathered write rows [C][W][NCOL], the chunk-start rows the scatter decays
    extern __shared__ __align__(16) float Wrow[];
    const ChunkRec L = chunk_rec_layout(W, R);
    const int tid = threadIdx.x;
    int sl, s;
    scan_wg_coords<true>(nslice, sl, s);
    // gather mapping
    const int gt = tid >> 3, gp = (tid >> 1) & 3, gq = tid & 1;
    // product mapping
    const int pt = tid >> 3, pc = narrow_pc(tid);
    const int col0 = sl * NCOL;
    float* ms = mem + (size_t)s * N * dv + col0;

    NarrowStage<NPR, SBN> cur;
    narrow_stage<VT, NPR, SBN, VEC>(cur, w_idx, r_idx, v, recs, L, s, cb, nch, T, W, R, N, dv, col0);
    for (int c = cb; c < ce; ++c) {
        const unsigned char* rec = recs + ((size_t)s * nch + c) * L.bytes;
        const int t0 = c * CC, n = min(CC, T - t0);
        const size_t tk0 = (size_t)s * T + t0;
        // ---- L and QK to LDS (the previous chunk's products ended before its last barrier) ----
#pragma unroll
        for (int k = 0; k < NLQ; ++k) {
            const int i = tid + k * NT3;
            const int r = (4 * i) / CC, c4 = (4 * i) % CC;
            *reinterpret_cast<float4*>(Ls + r * LDN + c4) = cur.la[k];
            *reinterpret_cast<float4*>(Qs + r * LDN + c4) = cur.qa[k];
        }
        // ---- gather: NPR row pieces in flight ----
        float4 m[NPR];
#pragma unroll
        for (int k = 0; k < NPR; ++k) m[k] = load4(ms + (size_t)cur.id[k] * dv + gq * 4);
        if constexpr (REUSE) {   // write rows -> LDS for the scatter
#pragma unroll
            for (int k = 0; k < NPR; ++k) {
                const int j = gp * NPR + k;
                if (j < W) *reinterpret_cast<float4*>(&Wrow[(gt * W + j) * NCOL + gq * 4]) = m[k];
            }
        }
        float4 ret = make_float4(0.f, 0.f, 0.f, 0.f), itr = make_float4(0.f, 0.f, 0.f, 0.f);
        const bool live = gt < n;
#pragma unroll
        for (int k = 0; k < NPR; ++k) {
            const int j = gp * NPR + k;
            const float w = live ? cur.wt[k] : 0.f;
            if (j < W) {
                ret.x += w * m[k].x; ret.y += w * m[k].y; ret.z += w * m[k].z; ret.w += w * m[k].w;
            } else {
                itr.x += w * m[k].x; itr.y += w * m[k].y; itr.z += w * m[k].z; itr.w += w * m[k].w;
            }
        }
        // the 4 parts of a (token, quad) are lanes 2 p + q of the token's 8: add
        // them across lanes; lane (p, q) then holds column 4 q + p = pc
        ret = f4_add_lanes(ret);
        itr = f4_add_lanes(itr);
        const float rsum = f4_elem(ret, gp), inter = f4_elem(itr, gp);
        // ---- the next chunk's staging (the last chunk reloads its own), in flight from
        //      here (not hoisted above the gather, where it would hold its registers
        //      beside the gathered rows) ----
        __builtin_amdgcn_sched_barrier(0);
        NarrowStage<NPR, SBN> nxt;
        narrow_stage<VT, NPR, SBN, VEC>(nxt, w_idx, r_idx, v, recs, L, s, min(c + 1, ce - 1), nch, T, W, R, N, dv,
                                        col0);
        // ---- R = v - retrieved ----
        RrT[pc * LDN + pt] = pt < n ? cur.vv - rsum : 0.f;
        __syncthreads();
        // ---- x = L R (L is zero above the diagonal and past the chunk's tokens) ----
        {
            float acc = 0.f;
#pragma unroll
            for (int u = 0; u < CC; u += 4) {
                const float4 l4 = *reinterpret_cast<const float4*>(Ls + pt * LDN + u);
                const float4 r4 = *reinterpret_cast<const float4*>(RrT + pc * LDN + u);
                acc += l4.x * r4.x + l4.y * r4.y + l4.z * r4.z + l4.w * r4.w;
            }
            Xs[pt * NCOL + pc] = acc;
            XsT[pc * LDN + pt] = acc;
        }
        __syncthreads();
        // ---- y = inter + QK x ----
        {
            float acc = inter;
#pragma unroll
            for (int u = 0; u < CC; u += 4) {
                const float4 q4 = *reinterpret_cast<const float4*>(Qs + pt * LDN + u);
                const float4 x4 = *reinterpret_cast<const float4*>(XsT + pc * LDN + u);
                acc += q4.x * x4.x + q4.y * x4.y + q4.z * x4.z + q4.w * x4.w;
            }
            if (pt < n) y[(tk0 + pt) * dv + col0 + pc] = acc;
        }
        // ---- scatter: each written slot once: its chunk-start row (from LDS when
        //      REUSE, else reloaded, SB3 in flight), decayed, plus its entries' x ----
        const int nseg = cur.nseg;
#pragma unroll
        for (int b0 = 0; b0 < SBN; b0 += SB3) {
            float4 mm[SB3];
#pragma unroll
            for (int b = 0; b < SB3; ++b) {
                const int q = (tid + NT3 * (b0 + b)) & 1;
                // token W + position of the first entry (clamped: units past the
                // chunk's segments hold whatever the record's tail holds)
                const int fe = min(cur.sg[b0 + b].y & 0xffff, CC * W - 1);
                mm[b] = REUSE ? *reinterpret_cast<const float4*>(&Wrow[fe * NCOL + q * 4])
                              : load4(ms + (size_t)min(max(cur.sg[b0 + b].x, 0), (int)(N - 1)) * dv + q * 4);
            }
#pragma unroll
            for (int b = 0; b < SB3; ++b) {
                const int u = tid + NT3 * (b0 + b);
                const int g = u >> 1, q = u & 1;
                if (g < nseg) {
                    const int4 si = cur.sg[b0 + b];
                    const int fe = si.y;
                    const float d = __int_as_float(si.z), w = __int_as_float(si.w);
                    const float4 x = *reinterpret_cast<const float4*>(&Xs[((fe & 0xffff) / W) * NCOL + q * 4]);
                    float4 acc = make_float4(d * mm[b].x + w * x.x, d * mm[b].y + w * x.y, d * mm[b].z + w * x.z,
                                             d * mm[b].w + w * x.w);
                    if (fe & (1 << 30)) {   // further entries of the slot (rare)
                        const int* g_sbeg = reinterpret_cast<const int*>(rec + L.off_sbeg);
                        const int* g_etok = reinterpret_cast<const int*>(rec + L.off_etok);
                        const float* g_ecoef = reinterpret_cast<const float*>(rec + L.off_ecoef);
                        const int f1 = g_sbeg[g + 1];
                        for (int f = g_sbeg[g] + 1; f < f1; ++f) {
                            const float wf = g_ecoef[f];
                            const float4 xf = *reinterpret_cast<const float4*>(&Xs[g_etok[f] * NCOL + q * 4]);
                            acc.x += wf * xf.x; acc.y += wf * xf.y; acc.z += wf * xf.z; acc.w += wf * xf.w;
                        }
                    }
                    *reinterpret_cast<float4*>(ms + (size_t)si.x * dv + q * 4) = acc;
                }
            }
        }
        __syncthreads();   // the chunk's stores precede the next chunk's gathers
        cur = nxt;
    }
}

template <typename VT>
hipError_t launch_chunk_coef(const ScanFwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H, nch = (a.T + CC - 1) / CC;
    const int cb = a.tb / CC, ce = (a.te + CC - 1) / CC;
    if (ce <= cb) return hipSuccess;
    const int P = pow2_at_least(CC * a.W);
    const size_t lds = coef_lds_bytes(a.W);
    auto kl = chunk_coef_kernel<VT>;
    hipError_t e = hipFuncSetAttribute((const void*)kl, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kl, dim3((unsigned)(S * (ce - cb))), dim3(CT1), lds, st, a.w_idx, a.w_val, a.r_idx, a.r_val,
                       static_cast<const VT*>(a.alpha), static_cast<const VT*>(a.beta), a.T, a.W, a.R, a.N, nch, cb,
                       ce - cb, P,
                       a.ws + SDM_WS_HEADER, reinterpret_cast<unsigned int*>(a.ws), a.gate_A, a.gate_bdt, a.H);
    return hipGetLastError();
}

template <typename VT, int COLS>
hipError_t launch_chunk_scan_cols(const ScanFwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H, nch = (a.T + CC - 1) / CC;
    const int cb = a.tb / CC, ce = (a.te + CC - 1) / CC;
    if (ce <= cb) return hipSuccess;
    const int nslice = (a.dv + COLS - 1) / COLS;
    constexpr size_t static_lds = (size_t)2 * CC * LDP * 4 + (size_t)2 * CC * COLS * 4;
    const size_t seg_bytes = scan_dyn_lds(a.W, a.R, true) - scan_dyn_lds(a.W, a.R, false);
    // (at 16 columns the staged lists push the kernel past its registers: they
    // are read from the record there)
    const bool seg = COLS == 32 && static_lds + scan_dyn_lds(a.W, a.R, true) <= (size_t)CK_LDS_LIMIT &&
                     seg_bytes <= (size_t)SEG_LDS_MAX;
    const size_t lds = scan_dyn_lds(a.W, a.R, seg);
    auto kl = seg ? chunk_scan_kernel<VT, true, COLS> : chunk_scan_kernel<VT, false, COLS>;
    hipError_t e = hipFuncSetAttribute((const void*)kl, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kl, dim3((unsigned)(S * nslice)), dim3(scan_threads<COLS>()), lds, st, a.w_idx, a.r_idx,
                       static_cast<const VT*>(a.v), a.mem, a.y, a.ws + SDM_WS_HEADER, a.T, a.W, a.R, a.N, a.dv,
                       nch, cb, ce, nslice);
    return hipGetLastError();
}

template <typename VT, int NPR, int SBN, bool REUSE>
hipError_t launch_chunk_narrow_t(const ScanFwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H, nch = (a.T + CC - 1) / CC;
    const int cb = a.tb / CC, ce = (a.te + CC - 1) / CC;
    if (ce <= cb) return hipSuccess;
    const int nslice = a.dv / NCOL;
    const size_t lds = REUSE ? (size_t)CC * a.W * NCOL * sizeof(float) : 0;
    const bool vec = a.W % 4 == 0 && a.R % 4 == 0 && (reinterpret_cast<uintptr_t>(a.w_idx) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(a.r_idx) & 15) == 0;
    auto kl = vec ? chunk_scan_narrow_kernel<VT, NPR, SBN, REUSE, true>
                  : chunk_scan_narrow_kernel<VT, NPR, SBN, REUSE, false>;
    hipError_t e = hipFuncSetAttribute((const void*)kl, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kl, dim3((unsigned)(S * nslice)), dim3(NT3), lds, st, a.w_idx, a.r_idx,
                       static_cast<const VT*>(a.v), a.mem, a.y, a.ws + SDM_WS_HEADER, a.T, a.W, a.R, a.N, a.dv, nch,
                       cb, ce, nslice);
    return hipGetLastError();
}

// Rows per part cover W + R; scatter units per thread cover 2 C W (one per
// written slot and quad), in rounds of SB3.  Up to 32 write rows per token the
// gathered rows stay in LDS (64 KB) for the scatter; past that it reloads them.
template <typename VT>
hipError_t launch_chunk_narrow(const ScanFwdArgs& a, hipStream_t st) {
    const bool rows16 = a.W + a.R <= NPART * 16;
    if (a.W <= 32) {
        return rows16 ? launch_chunk_narrow_t<VT, 16, 8, true>(a, st) : launch_chunk_narrow_t<VT, 32, 8, true>(a, st);
    }
    return rows16 ? launch_chunk_narrow_t<VT, 16, 16, false>(a, st) : launch_chunk_narrow_t<VT, 32, 16, false>(a, st);
}

// Workgroup width.  sdm_set_chunk_scan_cols forces 8 (the narrow kernel, d_v a
// multiple of 8), 16 or 32 columns.  Otherwise the narrow kernel runs when its
// workgroups fit the chip at one per CU and it keeps the gathered write rows in
// LDS (W <= 32), and 32 columns run elsewhere.  Measured (whole call, chunk
// coefficients included): long-context shape, 16 streams of 128 columns (256
// narrow workgroups): 27.4 ms narrow against 32.5 ms at 32 columns, the narrow
// kernel at 21.6 us per chunk against 31.0; learned-M0 shape, 32 streams (512
// narrow workgroups, two rounds): 6.8 against 5.4 ms.  The narrow workgroups
// hold 117 KB of LDS, so the next range's coefficient workgroups do not run
// beside them.  16-column workgroups of the wide kernel: 41.0 against 35.2 ms.
int chunk_cols_for(const ScanFwdArgs& a) {
    const int forced = sdm_chunk_cols();
    if (forced == 8 && a.dv % NCOL == 0) return 8;
    if (forced == 16 || forced == 32) return forced;
    const int64_t wgs = (int64_t)a.B * a.H * (a.dv / NCOL);
    if (a.dv % NCOL == 0 && a.W <= 32 && wgs <= sdm_device_simds() / 4) return 8;
    return 32;
}

template <typename VT>
hipError_t launch_chunk_scan(const ScanFwdArgs& a, hipStream_t st) {
    switch (chunk_cols_for(a)) {
        case 8: return launch_chunk_narrow<VT>(a, st);
        case 16: return launch_chunk_scan_cols<VT, 16>(a, st);
        default: return launch_chunk_scan_cols<VT, 32>(a, st);
    }
}

}  // namespace

bool sdm_chunk_shape_ok(int W, int R) {
    return W >= 1 && R >= 1 && W <= SDM_CHUNK_MAX_LIST && R <= SDM_CHUNK_MAX_LIST &&
           coef_lds_bytes(W) <= (size_t)CK_LDS_LIMIT;
}

size_t sdm_chunk_ws_bytes(int B, int H, int T, int W, int R) {
    const size_t nch = ((size_t)T + CC - 1) / CC;
    return SDM_WS_HEADER + (size_t)B * H * nch * chunk_rec_layout(W, R).bytes;
}

hipError_t sdm_launch_chunk_coef(const ScanFwdArgs& a, hipStream_t st) {
    return a.in_dtype == SDM_DT_BF16 ? launch_chunk_coef<bf16_t>(a, st) : launch_chunk_coef<float>(a, st);
}

hipError_t sdm_launch_chunk_scan(const ScanFwdArgs& a, hipStream_t st) {
    return a.in_dtype == SDM_DT_BF16 ? launch_chunk_scan<bf16_t>(a, st) : launch_chunk_scan<float>(a, st);
}
