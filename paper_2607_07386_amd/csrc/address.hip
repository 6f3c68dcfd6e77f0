// Product-key addressing (Sec. 2 "Product Key Memory", Sec. 3.1 step 1,
// Sec. 4 softmax-normalised activations, App. A.2 sort-by-index) and its
// backward, for gfx950.
//
// One workgroup = 4 waves = a tile of 16 tokens (8 or 4 for sqrt(N) above
// 256 or 512) of one (b, h) stream.
//  A. sub-key scores of the tile into LDS: bf16 codebooks on the matrix
//     cores (v_mfma_f32_16x16x32_bf16: 16 tokens x 16 sub-keys x 32 deep),
//     fp32 codebooks with plain FMAs, direct mode by copying x.
//  B. per token (one wave): top-k of each half under (score desc, id asc).
//     Keys are 64-bit (order-preserving score bits, inverted id), so the
//     order is total and ties go to the lower id.  The k-th largest of the
//     64 per-lane maxima is a lower bound that at least k keys reach; the
//     keys at or above it (about 40 for k = 32) are bitonic-sorted across the
//     wave, which yields the ranked shortlist.  More than 64 survivors (or
//     k > 32) take an exact bisection of the k-th key with wave ballots.
//  C. candidates (i, j) of the two ranked shortlists with (i+1)(j+1) <= k
//     (every other pair has >= k pairs ranked above it), selected the same
//     way, then sorted by slot id and softmax-normalised.
// k in (64, 128] runs a kernel of its own: lists of two entries per lane,
// exact bisection selection, 128-wide bitonic sorts.  For sqrt(N) in
// (256, 1024] with bf16 codebooks, d_k / 2 <= 64 and k <= 32, a third kernel
// (address_reg_kernel) keeps a 16-token tile's scores in the MFMA result
// registers: the groups of B's bound are the lanes' own scores, so only the
// group maxima and the candidates pass through LDS.
#include <algorithm>

#include "sdm_common.h"
#include "sdm_internal.h"

namespace {

constexpr int ATILE = 16;     // tokens per workgroup (the MFMA tile's rows), sqrt(N) <= 256
// Tokens per workgroup for E = ceil(sqrt(N) / 64): the scores of a tile take
// 2 AT 64 E floats of LDS, so larger sqrt(N) takes fewer tokens per workgroup
// (rows of the 16-row MFMA tile past AT are zero) to keep several workgroups
// on a CU: 32 KB at E = 4, 8, 16.
template <int E>
__host__ __device__ constexpr int atile() { return E <= 4 ? ATILE : (E <= 8 ? 8 : 4); }
// For sqrt(N) > 512 and k <= 64 the tile scores one half at a time, so the
// same 32 KB of scores hold 8 tokens instead of 4 and each workgroup reads the
// head's codebook (256 KB at sqrt(N) = 1024) for twice as many tokens.  Stage
// 1 of a half leaves each token's ranked shortlist in LDS; stage 2 reads both.
// (At sqrt(N) = 512 the same layout, 16 tokens in 56 KB, halved the
// workgroups per CU and measured slower.)
template <int E, int KM>
__host__ __device__ constexpr bool half_seq() { return E >= 16 && KM <= 64; }
template <int E, int KM>
__host__ __device__ constexpr int tile_tokens() { return half_seq<E, KM>() ? 8 : atile<E>(); }
constexpr int AWAVES = 4;
constexpr int MAXK = 64;      // largest k of the one-entry-per-lane kernels
constexpr int MAXK_BIG = 128; // largest k: two entries per lane
constexpr int MAXKS = 8;      // 32-deep MFMA steps per half: d_k / 2 <= 256
constexpr int MAXCAND_E = 5;  // ceil(280 / 64): pruned candidates for k <= 64
constexpr int MAXCAND_BIG = 11;  // ceil(645 / 64): pruned candidates for k <= 128

struct Entry {
    float score;
    int id;
};

// Pruned stage-2 pairs for every k <= MAXK: ranks (i, j) with (i+1)(j+1) <= k,
// i ascending then j ascending, packed as i << 8 | j.
constexpr int pair_count_total() {
    int t = 0;
    for (int k = 1; k <= MAXK; ++k)
        for (int i = 1; i <= k; ++i) t += k / i;
    return t;
}
struct PairTable {
    uint16_t off[MAXK + 1];   // first pair of k
    uint16_t n[MAXK + 1];     // number of pairs of k
    uint16_t e[pair_count_total()];
};
constexpr PairTable make_pair_table() {
    PairTable p{};
    int o = 0;
    for (int k = 1; k <= MAXK; ++k) {
        p.off[k] = (uint16_t)o;
        for (int i = 0; i < k; ++i)
            for (int j = 0; j < k / (i + 1); ++j) p.e[o++] = (uint16_t)(i << 8 | j);
        p.n[k] = (uint16_t)(o - p.off[k]);
    }
    return p;
}
__constant__ const PairTable c_pairs = make_pair_table();
static_assert(make_pair_table().n[32] <= 3 * 64 && make_pair_table().n[MAXK] <= MAXCAND_E * 64, "pair counts");

// Number of pruned pairs of k: sum over i < k of floor(k / (i + 1)).
__host__ __device__ constexpr int pair_count(int k) {
    int n = 0;
    for (int i = 1; i <= k; ++i) n += k / i;
    return n;
}
static_assert(pair_count(MAXK_BIG) <= MAXCAND_BIG * SDM_WAVE, "pair counts, k <= 128");

// k-th largest key: the largest tau with #{key >= tau} >= k.
template <int E>
__device__ uint32_t kth_key(const uint32_t (&key)[E], int k) {
    uint32_t tau = 0u;
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t cand = tau | (1u << bit);
        int cnt = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) cnt += popc64(__ballot(key[e] >= cand));
        if (cnt >= k) tau = cand;
    }
    return tau;
}

// Mark the k selected elements: keys above tau, then keys equal to tau in
// increasing id until k are taken.  Invalid elements carry key 0 and id
// INT_MAX and are never taken (all valid keys are > 0).
template <int E>
__device__ void select_topk(const uint32_t (&key)[E], const int (&id)[E], int k, bool (&sel)[E]) {
    const uint32_t tau = kth_key<E>(key, k);
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        n_gt += popc64(__ballot(key[e] > tau));
        n_eq += popc64(__ballot(key[e] == tau));
    }
    const int need = k - n_gt;
    if (n_eq == need) {
#pragma unroll
        for (int e = 0; e < E; ++e) sel[e] = key[e] >= tau;
        return;
    }
#pragma unroll
    for (int e = 0; e < E; ++e) sel[e] = key[e] > tau;
    for (int r = 0; r < need; ++r) {
        int best = 0x7fffffff;
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (key[e] == tau && !sel[e]) best = min(best, id[e]);
        best = wave_min_i(best);
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (key[e] == tau && id[e] == best) sel[e] = true;
    }
}

// Write the selected (score, id) pairs, in element order, to buf[0 .. k).
template <int E>
__device__ void compact(const bool (&sel)[E], const float (&sc)[E], const int (&id)[E], Entry* buf) {
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const unsigned long long m = __ballot(sel[e]);
        if (sel[e]) {
            const int p = base + mbcnt64(m);
            buf[p].score = sc[e];
            buf[p].id = id[e];
        }
        base += popc64(m);
    }
}

// Composite order key: larger key = higher score, or equal score and lower id.
__device__ __forceinline__ uint64_t ckey(float score, uint32_t id) {
    return ((uint64_t)ord_key(score) << 32) | (uint32_t)(~id);
}
__device__ __forceinline__ float ckey_score(uint64_t k) { return key_to_float((uint32_t)(k >> 32)); }
__device__ __forceinline__ int ckey_id(uint64_t k) { return (int)(~(uint32_t)k); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = xor_lane_u32((uint32_t)v, m);
    const uint32_t hi = xor_lane_u32((uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}

// Bitonic sorts of one key per lane across the wave.  Stage (KK, J) compares
// lanes i and i ^ J inside blocks of KK; every distance is a template
// argument, so each exchange is a DPP or permlane move.  Equal keys never
// swap, so padding keys stay padding.
template <int KK, int J>
__device__ __forceinline__ uint64_t bitonic_desc_u64(uint64_t key, int lane) {
    const uint64_t o = ((uint64_t)xor_lane<J>((uint32_t)(key >> 32)) << 32) | xor_lane<J>((uint32_t)key);
    const bool keep_max = ((lane & J) == 0) == ((lane & KK) == 0);
    key = keep_max ? (o > key ? o : key) : (o < key ? o : key);
    if constexpr (J > 1) return bitonic_desc_u64<KK, J / 2>(key, lane);
    else if constexpr (KK < SDM_WAVE) return bitonic_desc_u64<KK * 2, KK>(key, lane);
    else return key;
}
template <int KK, int J>
__device__ __forceinline__ uint32_t bitonic_desc_u32(uint32_t key, int lane) {
    const uint32_t o = xor_lane<J>(key);
    const bool keep_max = ((lane & J) == 0) == ((lane & KK) == 0);
    key = keep_max ? max(o, key) : min(o, key);
    if constexpr (J > 1) return bitonic_desc_u32<KK, J / 2>(key, lane);
    else if constexpr (KK < SDM_WAVE) return bitonic_desc_u32<KK * 2, KK>(key, lane);
    else return key;
}
template <int KK, int J>
__device__ __forceinline__ void bitonic_asc_u32_pay(uint32_t& key, float& pay, int lane) {
    const uint32_t o = xor_lane<J>(key);
    const float op = xor_lane_ff<J>(pay);
    const bool keep_min = ((lane & J) == 0) == ((lane & KK) == 0);
    const bool take = keep_min ? (o < key) : (o > key);
    key = take ? o : key;
    pay = take ? op : pay;
    if constexpr (J > 1) bitonic_asc_u32_pay<KK, J / 2>(key, pay, lane);
    else if constexpr (KK < SDM_WAVE) bitonic_asc_u32_pay<KK * 2, KK>(key, pay, lane);
}
// Descending: lane 0 holds the largest key.
__device__ __forceinline__ uint64_t wave_sort_desc_u64(uint64_t key) {
    return bitonic_desc_u64<2, 1>(key, lane_id());
}
__device__ __forceinline__ uint32_t wave_sort_desc_u32(uint32_t key) {
    return bitonic_desc_u32<2, 1>(key, lane_id());
}
// Ascending, with a payload riding along.
__device__ __forceinline__ void wave_sort_asc_u32(uint32_t& key, float& pay) {
    bitonic_asc_u32_pay<2, 1>(key, pay, lane_id());
}

// Exact top-k (k <= 32 for the fast path) of E keys per lane, returned sorted
// descending with lane i holding rank i (lanes >= k: padding).  The k-th
// largest per-lane maximum bounds the answer from below (at least k keys reach
// it), so only the keys at or above it are sorted; returns false when more
// than 64 survive, and the caller then takes the bisection path.
template <int E>
__device__ __forceinline__ bool topk_sorted(const uint64_t (&key)[E], int ne, int k, uint64_t* buf,
                                            uint64_t& top) {
    const int lane = lane_id();
    if (E == 1 || ne == 1) {
        top = wave_sort_desc_u64(key[0]);
        return true;
    }
    uint64_t m = key[0];
#pragma unroll
    for (int e = 1; e < E; ++e)
        if (e < ne) m = key[e] > m ? key[e] : m;
    const uint32_t srt = wave_sort_desc_u32((uint32_t)(m >> 32));
    const uint32_t tau = __shfl(srt, k - 1, SDM_WAVE);
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        if (e < ne) {
            const bool c = key[e] != 0ull && (uint32_t)(key[e] >> 32) >= tau;
            const unsigned long long msk = __ballot(c);
            const int p = base + mbcnt64(msk);
            if (c && p < SDM_WAVE) buf[p] = key[e];
            base += popc64(msk);
        }
    }
    if (base > SDM_WAVE) return false;
    wait_lds();
    __builtin_amdgcn_wave_barrier();
    const uint64_t v = lane < base ? buf[lane] : 0ull;
    top = wave_sort_desc_u64(v);
    return true;
}

// Descending bitonic sort of one 64-bit key per lane, held as (hi, lo).  One
// 64-bit compare per stage decides for both partners: the lane keeping the
// larger key takes the other's when it is larger, the other lane when it is
// not (keys are distinct except empty ones, which are equal and interchangeable).
template <int KK, int J, int NMAX>
__device__ __forceinline__ void bsort_desc64(uint32_t& hi, uint32_t& lo, int lane) {
    const uint32_t oh = xor_lane<J>(hi), ol = xor_lane<J>(lo);
    const bool gt = ((uint64_t)oh << 32 | ol) > ((uint64_t)hi << 32 | lo);
    const bool keep_max = lane_in<~(lanes_with_bit<J>() ^ lanes_with_bit<KK>())>();
    const bool take = gt == keep_max;
    hi = take ? oh : hi;
    lo = take ? ol : lo;
    if constexpr (J > 1) bsort_desc64<KK, J / 2, NMAX>(hi, lo, lane);
    else if constexpr (KK < NMAX) bsort_desc64<KK * 2, KK, NMAX>(hi, lo, lane);
}
// Ascending bitonic sort of one key per lane with a payload, within blocks of NMAX lanes.
template <int KK, int J, int NMAX>
__device__ __forceinline__ void bsort_asc_pay(uint32_t& key, float& pay, int lane) {
    const uint32_t o = xor_lane<J>(key);
    const float op = xor_lane_ff<J>(pay);
    const bool lt = o < key;
    const bool keep_min = lane_in<~(lanes_with_bit<J>() ^ lanes_with_bit<KK>())>();
    const bool take = lt == keep_min;
    key = take ? o : key;
    pay = take ? op : pay;
    if constexpr (J > 1) bsort_asc_pay<KK, J / 2, NMAX>(key, pay, lane);
    else if constexpr (KK < NMAX) bsort_asc_pay<KK * 2, KK, NMAX>(key, pay, lane);
}

// Stage-1 selection of one half: top-k of s sub-scores, ranked (score desc,
// id asc) into out[0 .. k).
template <int E>
__device__ void half_topk_bisect(const float* sc_row, int s, int k, Entry* scratch, Entry* out) {
    const int lane = lane_id();
    uint32_t key[E];
    float sc[E];
    int id[E];
    bool sel[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int g = e * SDM_WAVE + lane;
        const bool ok = g < s;
        sc[e] = ok ? sc_row[g] : 0.f;
        key[e] = ok ? ord_key(sc[e]) : 0u;
        id[e] = ok ? g : 0x7fffffff;
    }
    select_topk<E>(key, id, k, sel);
    compact<E>(sel, sc, id, scratch);
    wait_lds();
    __builtin_amdgcn_wave_barrier();
    // rank the k selected (k <= 64) with one bitonic sort of (score key, inverted id)
    const Entry me = scratch[min(lane, k - 1)];
    uint32_t th = lane < k ? ord_key(me.score) : 0u;
    uint32_t tl = ~(uint32_t)me.id;
    bsort_desc64<2, 1, SDM_WAVE>(th, tl, lane);
    if (lane < k) out[lane] = Entry{key_to_float(th), (int)~tl};
    wait_lds();
}

// Stage-1 selection of one half: top-k of s sub-scores, ranked (score desc,
// id asc) into out[0 .. k).
template <int E>
__device__ void half_topk(const float* sc_row, int s, int k, Entry* scratch, uint64_t* kbuf, Entry* out) {
    const int lane = lane_id();
    if (k <= 32) {
        uint64_t key[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int g = e * SDM_WAVE + lane;
            key[e] = g < s ? ckey(sc_row[g], (uint32_t)g) : 0ull;
        }
        uint64_t top;
        if (topk_sorted<E>(key, E, k, kbuf, top)) {
            if (lane < k) out[lane] = Entry{ckey_score(top), ckey_id(top)};
            wait_lds();
            __builtin_amdgcn_wave_barrier();
            return;
        }
    }
    half_topk_bisect<E>(sc_row, s, k, scratch, out);
}

// ---- fast path (k <= 32, s <= 256) ------------------------------------
// Candidates for the top-k (k <= 32) of E scores per lane (ids gid; -inf
// pads): the k-th largest per-lane maximum, found by bisection on order keys
// with wave ballots, is reached by at least k scores, and those are gathered
// into lanes 0 .. n-1 as (score bits, id).  The bound only has to be at or
// below that maximum, so the bisection stops after the sign, the exponent and
// 11 mantissa bits (admitting the few scores within 2^-11 relative below it).
// Returns false (uniformly) unless k <= n <= 64.
template <int E>
__device__ __forceinline__ bool gather_candidates(const float (&sc)[E], const uint32_t (&gid)[E], int k,
                                                  uint2* kbuf, uint2& mine, int& n) {
    const int lane = lane_id();
    float mf = sc[0];
#pragma unroll
    for (int e = 1; e < E; ++e) mf = fmaxf(mf, sc[e]);
    const uint32_t m = ord_key(mf);
    uint32_t tau = 0u;
#pragma unroll
    for (int bit = 31; bit >= 12; --bit) {
        const uint32_t c = tau | (1u << bit);
        if (popc64(__ballot(m >= c)) >= k) tau = c;
    }
    const float tf = key_to_float(tau);   // scores >= tf are exactly the keys >= tau
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const bool c = sc[e] >= tf;
        const unsigned long long msk = __ballot(c);
        const int p = base + mbcnt64(msk);
        if (c && p < SDM_WAVE) kbuf[p] = make_uint2(__float_as_uint(sc[e]), gid[e]);
        base += popc64(msk);
    }
    n = base;
    if (base > SDM_WAVE || base < k) return false;   // (< k only for non-finite scores)
    __builtin_amdgcn_wave_barrier();
    mine = kbuf[min(lane, SDM_WAVE - 1)];
    return true;
}

// Ranked top-k (k <= 32) of E scores per lane under (score desc, id asc):
// 64-bit keys (order key of the score, inverted id) sorted descending, rank r
// in lane r.  False when the candidates overflow.
template <int E>
__device__ __forceinline__ bool fast_topk(const float (&sc)[E], const uint32_t (&gid)[E], int k,
                                          uint2* kbuf, uint32_t& th, uint32_t& tl) {
    const int lane = lane_id();
    uint2 v;
    int n;
    if (!gather_candidates<E>(sc, gid, k, kbuf, v, n)) return false;
    th = lane < n ? ord_key(__uint_as_float(v.x)) : 0u;
    tl = ~v.y;
    bsort_desc64<2, 1, SDM_WAVE>(th, tl, lane);
    return true;
}

// Stage 1 of one half on the fast path (k <= 32, s <= 64 E, the half's row
// padded with -inf): its ranked top-k into out[0 .. k).  False when the
// candidates overflowed.
template <int E>
__device__ __forceinline__ bool half_fast(const float* hrow, int k, uint2* kbuf, Entry* out) {
    const int lane = lane_id();
    float sc[E];
    uint32_t gid[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        sc[e] = hrow[e * SDM_WAVE + lane];
        gid[e] = e * SDM_WAVE + lane;
    }
    uint32_t th, tl;
    if (!fast_topk<E>(sc, gid, k, kbuf, th, tl)) return false;
    if (lane < k) out[lane] = Entry{key_to_float(th), (int)~tl};
    return true;
}

// Stage 2 on the fast path from the two ranked shortlists (pi, pj: this
// lane's pair ranks; pairs past the count point at a -inf list entry): the
// top-k of the pruned pairs, id sort and softmax, outputs written.  False when
// a selection overflowed or the k-th place is tied.
__device__ __forceinline__ bool pairs_fast(int s, int k, const uint32_t (&pi)[3], const uint32_t (&pj)[3],
                                           const Entry* listA, const Entry* listB, uint2* kbuf,
                                           int32_t* idx_out, float* val_out, float* score_out) {
    const int lane = lane_id();
    float sc[3];
    uint32_t gid[3];
#pragma unroll
    for (int e = 0; e < 3; ++e) {
        const Entry a = listA[pi[e]], b = listB[pj[e]];
        sc[e] = a.score + b.score;
        gid[e] = (uint32_t)(a.id * s + b.id);
    }
    uint2 v;
    int n;
    if (!gather_candidates<3>(sc, gid, k, kbuf, v, n)) return false;
    // exact k-th largest candidate score by bisection; a tie across the k-th
    // place (to be broken by id) takes the general path
    const uint32_t key = lane < n ? ord_key(__uint_as_float(v.x)) : 0u;
    uint32_t tau = 0u;
#pragma unroll
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t c = tau | (1u << bit);
        if (popc64(__ballot(key >= c)) >= k) tau = c;
    }
    const bool sel = key >= tau;
    const unsigned long long selm = __ballot(sel);
    if (popc64(selm) != k) return false;
    if (sel) kbuf[mbcnt64(selm)] = v;
    __builtin_amdgcn_wave_barrier();
    const uint2 w = kbuf[min(lane, SDM_WAVE - 1)];
    const bool mine = lane < k;
    uint32_t my_id = mine ? w.y : 0xffffffffu;
    float my_sc = mine ? __uint_as_float(w.x) : -INFINITY;
    const float mx = wave_max<16>(my_sc);
    // slots in ascending id order (App. A.2), then softmax (Sec. 4)
    bsort_asc_pay<2, 1, 32>(my_id, my_sc, lane);
    const float ex = expf(my_sc - mx);
    const float z = wave_sum<16>(ex);
    if (lane < k) {
        idx_out[lane] = (int32_t)my_id;
        val_out[lane] = ex / z;
        if (score_out) score_out[lane] = my_sc;
    }
    return true;
}

// One token, k <= 32 and s <= SP = 64 E: stage 1 on both halves, then stage
// 2.  Returns false when a selection overflowed (the caller then runs the
// general path for this token).
template <int E>
__device__ __forceinline__ bool token_fast(const float* row, int s, int k, const uint32_t (&pi)[3],
                                           const uint32_t (&pj)[3], Entry* listA, Entry* listB,
                                           uint2* kbuf, int32_t* idx_out, float* val_out,
                                           float* score_out) {
    constexpr int SP = E * SDM_WAVE;
    if (!half_fast<E>(row, k, kbuf, listA) || !half_fast<E>(row + SP, k, kbuf, listB)) return false;
    __builtin_amdgcn_wave_barrier();
    return pairs_fast(s, k, pi, pj, listA, listB, kbuf, idx_out, val_out, score_out);
}

// Stage 2 of one token (k <= 64) on this wave, from the ranked shortlists of
// the two halves: the pruned pairs, their top-k, id sort, softmax.  Out of
// line: inlined into token_general it raised the address kernel's registers
// from 104 to 148.
__device__ __noinline__ void token_pairs(int s, int k, int ncand, const uint16_t* pairs, Entry* scr,
                                            const Entry* listA, const Entry* listB, uint64_t* kbuf,
                                            int32_t* idx_out, float* val_out, float* score_out) {
    const int lane = lane_id();
    const int ne2 = (ncand + SDM_WAVE - 1) / SDM_WAVE;
    // stage 2 over the pruned pairs of the two ranked shortlists
    uint64_t ck[MAXCAND_E];
#pragma unroll
    for (int e = 0; e < MAXCAND_E; ++e) {
        const int c = e * SDM_WAVE + lane;
        ck[e] = 0ull;
        if (e < ne2 && c < ncand) {
            const uint32_t pr = pairs[c];
            const Entry a = listA[pr >> 8], b = listB[pr & 0xffu];
            ck[e] = ckey(a.score + b.score, (uint32_t)(a.id * s + b.id));
        }
    }
    float my_sc = -INFINITY;
    uint32_t my_id = 0xffffffffu;
    uint64_t top;
    if (k <= 32 && topk_sorted<MAXCAND_E>(ck, ne2, k, kbuf, top)) {
        if (lane < k) {
            my_sc = ckey_score(top);
            my_id = (uint32_t)ckey_id(top);
        }
    } else {
        uint32_t key[MAXCAND_E];
        float sc[MAXCAND_E];
        int id[MAXCAND_E];
        bool sel[MAXCAND_E];
#pragma unroll
        for (int e = 0; e < MAXCAND_E; ++e) {
            const bool ok = ck[e] != 0ull;
            sc[e] = ok ? ckey_score(ck[e]) : 0.f;
            key[e] = ok ? (uint32_t)(ck[e] >> 32) : 0u;
            id[e] = ok ? ckey_id(ck[e]) : 0x7fffffff;
        }
        select_topk<MAXCAND_E>(key, id, k, sel);
        compact<MAXCAND_E>(sel, sc, id, scr);
        wait_lds();
        __builtin_amdgcn_wave_barrier();
        if (lane < k) {
            my_sc = scr[lane].score;
            my_id = (uint32_t)scr[lane].id;
        }
    }
    // selected slots in ascending id order (App. A.2), then their softmax (Sec. 4)
    wave_sort_asc_u32(my_id, my_sc);
    const float mx = wave_max(lane < k ? my_sc : -INFINITY);
    const float ex = lane < k ? expf(my_sc - mx) : 0.f;
    const float z = wave_sum(ex);
    if (lane < k) {
        idx_out[lane] = (int32_t)my_id;
        val_out[lane] = ex / z;
        if (score_out) score_out[lane] = my_sc;
    }
    wait_lds();
    __builtin_amdgcn_wave_barrier();
}

// One token on the general path (any k, overflowing selections): stage 1 on
// both halves, stage 2 over the pruned pairs, id sort and softmax.  Kept out
// of line: it is the cold path of the common shapes.
template <int E>
__device__ __noinline__ void token_general(const float* row, int s, int sp, int k, int ncand, const uint16_t* pairs,
                                           Entry* scr, Entry* listA, Entry* listB, uint64_t* kbuf,
                                           int32_t* idx_out, float* val_out, float* score_out) {
    half_topk<E>(row, s, k, scr, kbuf, listA);
    half_topk<E>(row + sp, s, k, scr, kbuf, listB);
    token_pairs(s, k, ncand, pairs, scr, listA, listB, kbuf, idx_out, val_out, score_out);
}

// ---- k in (64, 128]: two list entries per lane ---------------------------
// Position p = 64 r + lane of a 128-entry list lives in register r of its lane.
// Bitonic stage (KK, J) pairs positions p and p ^ J: within a lane's two
// registers for J = 64, across lanes (DPP / permlane) otherwise.  The lower
// position of a pair keeps the larger key when its block of KK runs
// descending, which for a descending sort is the block with p & KK == 0.
template <int KK, int J>
__device__ __forceinline__ void bsort128_desc(uint64_t (&key)[2], int lane) {
    if constexpr (J == 64) {
        const uint64_t a = key[0], b = key[1];
        key[0] = a > b ? a : b;
        key[1] = a > b ? b : a;
    } else {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const uint64_t o = ((uint64_t)xor_lane<J>((uint32_t)(key[r] >> 32)) << 32) |
                               xor_lane<J>((uint32_t)key[r]);
            const bool desc = KK == 128 ? true : (KK == 64 ? r == 0 : (lane & KK) == 0);
            const bool keep_max = ((lane & J) == 0) == desc;
            key[r] = keep_max ? (o > key[r] ? o : key[r]) : (o < key[r] ? o : key[r]);
        }
    }
    if constexpr (J > 1) bsort128_desc<KK, J / 2>(key, lane);
    else if constexpr (KK < 128) bsort128_desc<KK * 2, KK>(key, lane);
}
// Ascending by key with a payload riding along (same network, directions flipped).
template <int KK, int J>
__device__ __forceinline__ void bsort128_asc_pay(uint32_t (&key)[2], float (&pay)[2], int lane) {
    if constexpr (J == 64) {
        const bool sw = key[1] < key[0];
        const uint32_t k0 = key[0];
        const float p0 = pay[0];
        key[0] = sw ? key[1] : key[0];
        pay[0] = sw ? pay[1] : pay[0];
        key[1] = sw ? k0 : key[1];
        pay[1] = sw ? p0 : pay[1];
    } else {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const uint32_t o = xor_lane<J>(key[r]);
            const float op = xor_lane_ff<J>(pay[r]);
            const bool asc = KK == 128 ? true : (KK == 64 ? r == 0 : (lane & KK) == 0);
            const bool keep_min = ((lane & J) == 0) == asc;
            const bool take = keep_min ? (o < key[r]) : (o > key[r]);
            key[r] = take ? o : key[r];
            pay[r] = take ? op : pay[r];
        }
    }
    if constexpr (J > 1) bsort128_asc_pay<KK, J / 2>(key, pay, lane);
    else if constexpr (KK < 128) bsort128_asc_pay<KK * 2, KK>(key, pay, lane);
}

// Stage 1 of one half for k <= 128: exact selection, then the k selected
// ranked (score desc, id asc) into out[0 .. k).
template <int E>
__device__ void half_topk_big(const float* sc_row, int s, int k, Entry* scratch, Entry* out) {
    const int lane = lane_id();
    uint32_t key[E];
    float sc[E];
    int id[E];
    bool sel[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int g = e * SDM_WAVE + lane;
        const bool ok = g < s;
        sc[e] = ok ? sc_row[g] : 0.f;
        key[e] = ok ? ord_key(sc[e]) : 0u;
        id[e] = ok ? g : 0x7fffffff;
    }
    select_topk<E>(key, id, k, sel);
    compact<E>(sel, sc, id, scratch);
    wait_lds();
    __builtin_amdgcn_wave_barrier();
    uint64_t ck2[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int p = r * SDM_WAVE + lane;
        const Entry me = scratch[min(p, k - 1)];
        ck2[r] = p < k ? ckey(me.score, (uint32_t)me.id) : 0ull;
    }
    bsort128_desc<2, 1>(ck2, lane);
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int p = r * SDM_WAVE + lane;
        if (p < k) out[p] = Entry{ckey_score(ck2[r]), ckey_id(ck2[r])};
    }
    wait_lds();
    __builtin_amdgcn_wave_barrier();
}

// One token with 64 < k <= 128: stage 1 on both halves, stage 2 over the
// pruned pairs (pairs[0 .. ncand), i << 8 | j), the k winners sorted by id,
// softmax.  Lane l writes positions l and 64 + l of the outputs.
template <int E>
__device__ __noinline__ void token_big(const float* row, int s, int sp, int k, int ncand, const uint16_t* pairs,
                                       Entry* scr, Entry* listA, Entry* listB, int32_t* idx_out,
                                       float* val_out, float* score_out) {
    const int lane = lane_id();
    half_topk_big<E>(row, s, k, scr, listA);
    half_topk_big<E>(row + sp, s, k, scr, listB);

    uint32_t key[MAXCAND_BIG];
    float sc[MAXCAND_BIG];
    int id[MAXCAND_BIG];
    bool sel[MAXCAND_BIG];
#pragma unroll
    for (int e = 0; e < MAXCAND_BIG; ++e) {
        const int c = e * SDM_WAVE + lane;
        const bool ok = c < ncand;
        const uint32_t pr = pairs[ok ? c : 0];
        const Entry a = listA[pr >> 8], b = listB[pr & 0xffu];
        sc[e] = ok ? a.score + b.score : 0.f;
        key[e] = ok ? ord_key(sc[e]) : 0u;
        id[e] = ok ? a.id * s + b.id : 0x7fffffff;
    }
    select_topk<MAXCAND_BIG>(key, id, k, sel);
    compact<MAXCAND_BIG>(sel, sc, id, scr);
    wait_lds();
    __builtin_amdgcn_wave_barrier();

    // selected slots in ascending id order (App. A.2), then their softmax (Sec. 4)
    uint32_t my_id[2];
    float my_sc[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int p = r * SDM_WAVE + lane;
        const Entry me = scr[min(p, k - 1)];
        my_id[r] = p < k ? (uint32_t)me.id : 0xffffffffu;
        my_sc[r] = p < k ? me.score : -INFINITY;
    }
    bsort128_asc_pay<2, 1>(my_id, my_sc, lane);
    const float mx = wave_max(fmaxf(my_sc[0], my_sc[1]));
    float ex[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) ex[r] = r * SDM_WAVE + lane < k ? expf(my_sc[r] - mx) : 0.f;
    const float z = wave_sum(ex[0] + ex[1]);
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int p = r * SDM_WAVE + lane;
        if (p < k) {
            idx_out[p] = (int32_t)my_id[r];
            val_out[p] = ex[r] / z;
            if (score_out) score_out[p] = my_sc[r];
        }
    }
    wait_lds();
    __builtin_amdgcn_wave_barrier();
}

// Pruned stage-2 pairs of k (i << 8 | j, i ascending then j): the constant
// table for k <= 64; for k > 64 the workgroup builds them in lp (LDS), visible
// after its next barrier.
template <int KM>
__device__ __forceinline__ void tile_pairs(int k, uint16_t* lp, const uint16_t*& pairs, int& ncand) {
    if constexpr (KM > MAXK) {
        for (int i = threadIdx.x; i < k; i += blockDim.x) {
            int o = 0;
            for (int a = 1; a <= i; ++a) o += k / a;
            const int n = k / (i + 1);
            for (int j = 0; j < n; ++j) lp[o + j] = (uint16_t)(i << 8 | j);
        }
        pairs = lp;
        ncand = pair_count(k);
    } else {
        pairs = c_pairs.e + c_pairs.off[k];
        ncand = c_pairs.n[k];
    }
}

// Phase A: sub-key scores of tokens t0 .. t0 + nt - 1 (nt <= AT) of one
// stream (xs: its x, token stride dk; cbh: its head's codebook [2][s][dk/2],
// unused in direct mode) into score rows 0 .. nt-1: row [NH][SP] for halves
// HB .. HB + NH - 1 (both by default), half h's sub-key j at (h - HB) SP + j,
// j in [s, SP) -inf.  Rows past nt are not written.
template <typename XT, int MODE, int E, int HB = 0, int NH = 2>
__device__ __forceinline__ void tile_scores(const XT* __restrict__ xs, const XT* __restrict__ cbh, int t0, int nt,
                                            int dk, int s, float* scores) {
    constexpr int SP = E * SDM_WAVE;
    const int tid = threadIdx.x;
    const int wave = tid / SDM_WAVE;
    const int lane = lane_id();
    // Row of a token: [2][SP], half h's sub-key j at h*SP + j; j in [s, SP) holds -inf.
    if constexpr (MODE == 0) {
        for (int i = tid; i < nt * NH * SP; i += blockDim.x) {
            const int tt = i / (NH * SP), half = HB + (i / SP) % NH, j = i % SP;
            const int t = t0 + tt;
            scores[i] = j >= s ? -INFINITY : to_f32(xs[(size_t)t * dk + half * s + j]);
        }
    } else if constexpr (MODE == 1) {
        const int dh = dk / 2;
        for (int i = tid; i < nt * NH * SP; i += blockDim.x) {
            const int tt = i / (NH * SP), half = HB + (i / SP) % NH, j = i % SP;
            const int t = t0 + tt;
            float acc = 0.f;
            if (j < s) {
                const XT* xr = xs + (size_t)t * dk + half * dh;
                const XT* cr = cbh + ((size_t)half * s + j) * dh;
                for (int c = 0; c < dh; ++c) acc = fmaf(to_f32(xr[c]), to_f32(cr[c]), acc);
            }
            scores[i] = j < s ? acc : -INFINITY;
        }
    } else {
        // MFMA 16x16x32: A[i][kk] = x[t0+i][half*dh + kk], B[kk][j] = cb[half][j0+j][kk].
        // Lane l supplies row/col (l % 16) and k-slice 8*(l/16) .. +7 of each 32-deep step;
        // result acc[v] is D[4*(l/16) + v][l % 16].
        const int dh = dk / 2;
        const int ntile = (s + 15) / 16;
        const int nks = (dh + 31) / 32;   // 32-deep steps (at most MAXKS)
        const int r16 = lane % 16, q = lane / 16;
        const int t = t0 + r16;
        const bool trow = r16 < nt;   // this lane's token row exists
        if (nks <= 2) {
            // dh <= 64: this wave's tiles of a half (E of them) need 2 E codebook
            // operands; they are loaded EG tiles at a time, all of a group before
            // its first MFMA, so a group pays one load latency instead of one per
            // tile (every tile at once for s <= 256, E <= 4)
            constexpr int EG = E < 4 ? E : 4;
#pragma unroll
            for (int half = HB; half < HB + NH; ++half) {
                sdm_bf16x8 a[2];
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int kc = ks * 32 + 8 * q;
                    a[ks] = sdm_bf16x8{};
                    if (ks < nks && trow && kc < dh)
                        a[ks] = *reinterpret_cast<const sdm_bf16x8*>(xs + (size_t)t * dk + half * dh + kc);
                }
#pragma unroll
                for (int i0 = 0; i0 < E; i0 += EG) {
                    sdm_bf16x8 b[EG][2];
#pragma unroll
                    for (int i = 0; i < EG; ++i) {
                        const int j = (wave + AWAVES * (i0 + i)) * 16 + r16;
                        const XT* crow = cbh + ((size_t)half * s + min(j, s - 1)) * dh;
#pragma unroll
                        for (int ks = 0; ks < 2; ++ks) {
                            const int kc = ks * 32 + 8 * q;
                            b[i][ks] = sdm_bf16x8{};
                            if (ks < nks && j < s && kc < dh)
                                b[i][ks] = *reinterpret_cast<const sdm_bf16x8*>(crow + kc);
                        }
                    }
#pragma unroll
                    for (int i = 0; i < EG; ++i) {
                        const int j = (wave + AWAVES * (i0 + i)) * 16 + r16;
                        sdm_f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0], b[i][0], acc, 0, 0, 0);
                        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1], b[i][1], acc, 0, 0, 0);
                        if (j < s) {
#pragma unroll
                            for (int v = 0; v < 4; ++v)
                                if (4 * q + v < nt)
                                    scores[(size_t)(4 * q + v) * NH * SP + (half - HB) * SP + j] = acc[v];
                        }
                    }
                }
            }
        } else
        for (int half = HB; half < HB + NH; ++half) {
            // operand A (this lane's token row, k-slices 8q .. 8q+7 of each step) serves
            // every sub-key tile of the half
            sdm_bf16x8 a[MAXKS];
#pragma unroll
            for (int ks = 0; ks < MAXKS; ++ks) {
                const int kc = ks * 32 + 8 * q;
                a[ks] = sdm_bf16x8{};
                if (ks < nks && trow && kc < dh)
                    a[ks] = *reinterpret_cast<const sdm_bf16x8*>(xs + (size_t)t * dk + half * dh + kc);
            }
            for (int jt = wave; jt < ntile; jt += AWAVES) {
                const int j = jt * 16 + r16;
                const XT* crow = cbh + ((size_t)half * s + min(j, s - 1)) * dh;
                sdm_f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < MAXKS; ++ks) {
                    if (ks < nks) {
                        const int kc = ks * 32 + 8 * q;
                        sdm_bf16x8 b = sdm_bf16x8{};
                        if (j < s && kc < dh) b = *reinterpret_cast<const sdm_bf16x8*>(crow + kc);
                        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], b, acc, 0, 0, 0);
                    }
                }
                if (j < s) {
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (4 * q + v < nt) scores[(size_t)(4 * q + v) * NH * SP + (half - HB) * SP + j] = acc[v];
                }
            }
        }
        if (s < SP) {
            const int pad = SP - s;
            for (int i = tid; i < nt * NH * pad; i += blockDim.x)
                scores[(i / pad) * SP + s + i % pad] = -INFINITY;
        }
    }
}

// Per-wave state of phases B, C: scratch lists and sort buffer, and for the
// fast path (k <= 32: at most 130 pruned pairs, 3 per lane) the pair ranks;
// list entries past k hold -inf and pairs past the count point at entry 63.
struct SelWave {
    Entry* scr;
    Entry* listA;
    Entry* listB;
    uint64_t* kbuf;
    uint32_t pi[3], pj[3];
};
template <int KM>
__device__ __forceinline__ void select_init(SelWave& w, Entry* scratch, uint64_t* kbufs, int wave, int k,
                                            int ncand, const uint16_t* pairs) {
    const int lane = lane_id();
    w.scr = scratch + wave * 3 * KM;
    w.listA = w.scr + KM;
    w.listB = w.scr + 2 * KM;
    w.kbuf = kbufs + wave * SDM_WAVE;
    if constexpr (KM <= MAXK) {
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            const int c = e * SDM_WAVE + lane;
            const uint32_t pr = c < ncand ? pairs[min(c, ncand - 1)] : ((MAXK - 1u) << 8 | (MAXK - 1u));
            w.pi[e] = pr >> 8;
            w.pj[e] = pr & 0xffu;
        }
        if (lane >= k) {
            w.listA[lane] = Entry{-INFINITY, 0};
            w.listB[lane] = Entry{-INFINITY, 0};
        }
    }
}

// Phases B, C of one token (score row `row`) on this wave: ranked top-k of
// each half, stage 2, id sort, softmax; k values to io, vo (and so).
template <int E, int KM>
__device__ __forceinline__ void select_token(SelWave& w, const float* row, int s, int k, int ncand,
                                             const uint16_t* pairs, int32_t* io, float* vo, float* so) {
    constexpr int SP = E * SDM_WAVE;
    if constexpr (KM > MAXK) {
        token_big<E>(row, s, SP, k, ncand, pairs, w.scr, w.listA, w.listB, io, vo, so);
    } else {
        if constexpr (E <= 4) {
            if (k <= 32 && k <= s &&
                token_fast<E>(row, s, k, w.pi, w.pj, w.listA, w.listB, reinterpret_cast<uint2*>(w.kbuf), io, vo,
                              so))
                return;
        }
        token_general<E>(row, s, SP, k, ncand, pairs, w.scr, w.listA, w.listB, w.kbuf, io, vo, so);
        wait_lds();
        __builtin_amdgcn_wave_barrier();
    }
}

// The tokens [t0, min(t0 + AT, te)) of stream `stream` (AT = atile<E>()), by
// the AWAVES waves of a workgroup, in the LDS smem (address_lds_bytes): one
// wave per token in phases B, C.  MODE 0: direct, 1: codebook FMA, 2:
// codebook MFMA (bf16).
template <typename XT, int MODE, int E, int KM>
__device__ __forceinline__ void address_tile(const XT* __restrict__ x, const XT* __restrict__ cb, int H, int T,
                                             int stream, int t0, int te, int dk, int s, int k,
                                             int32_t* __restrict__ idx, float* __restrict__ val,
                                             float* __restrict__ score, unsigned char* smem) {
    constexpr int AT = atile<E>();
    constexpr int SP = E * SDM_WAVE;
    float* scores = reinterpret_cast<float*>(smem);                          // [AT][2][64 E]
    Entry* scratch = reinterpret_cast<Entry*>(scores + (size_t)AT * 2 * SP);  // [AWAVES][3][KM]
    uint64_t* kbufs = reinterpret_cast<uint64_t*>(scratch + AWAVES * 3 * KM);  // [AWAVES][64]
    const int wave = threadIdx.x / SDM_WAVE;
    const uint16_t* pairs;
    int ncand;
    tile_pairs<KM>(k, reinterpret_cast<uint16_t*>(kbufs + AWAVES * SDM_WAVE), pairs, ncand);
    const XT* cbh = MODE == 0 ? cb : cb + (size_t)(stream % H) * 2 * s * (dk / 2);
    tile_scores<XT, MODE, E>(x + (size_t)stream * T * dk, cbh, t0, min(AT, te - t0), dk, s, scores);
    __syncthreads();

    // ---- B, C: one wave per token (as select_init / select_token, written
    //      out here: the same code through those helpers spills scalar
    //      registers in this loop)
    const int lane = lane_id();
    Entry* scr = scratch + wave * 3 * KM;
    Entry* listA = scr + KM;
    Entry* listB = scr + 2 * KM;
    uint64_t* kbuf = kbufs + wave * SDM_WAVE;
    if constexpr (KM > MAXK) {
        for (int tt = wave; tt < AT; tt += AWAVES) {
            const int t = t0 + tt;
            if (t >= te) break;
            const size_t o = ((size_t)stream * T + t) * k;
            token_big<E>(scores + (size_t)tt * 2 * SP, s, SP, k, ncand, pairs, scr, listA, listB, idx + o,
                         val + o, score ? score + o : nullptr);
        }
        return;
    }
    const bool fast = E <= 4 && k <= 32 && k <= s;
    uint32_t pi[3], pj[3];
#pragma unroll
    for (int e = 0; e < 3; ++e) {
        const int c = e * SDM_WAVE + lane;
        const uint32_t pr = c < ncand ? pairs[min(c, ncand - 1)] : ((MAXK - 1u) << 8 | (MAXK - 1u));
        pi[e] = pr >> 8;
        pj[e] = pr & 0xffu;
    }
    if (lane >= k) {
        listA[lane] = Entry{-INFINITY, 0};
        listB[lane] = Entry{-INFINITY, 0};
    }
    for (int tt = wave; tt < AT; tt += AWAVES) {
        const int t = t0 + tt;
        if (t >= te) break;
        const float* row = scores + (size_t)tt * 2 * SP;
        if constexpr (E <= 4) {
            if (fast) {
                const size_t o = ((size_t)stream * T + t) * k;
                if (token_fast<E>(row, s, k, pi, pj, listA, listB, reinterpret_cast<uint2*>(kbuf),
                                  idx + o, val + o, score ? score + o : nullptr))
                    continue;
            }
        }
        token_general<E>(row, s, SP, k, ncand, pairs, scr, listA, listB, kbuf, idx + ((size_t)stream * T + t) * k,
                         val + ((size_t)stream * T + t) * k, score ? score + ((size_t)stream * T + t) * k : nullptr);
        wait_lds();
        __builtin_amdgcn_wave_barrier();
    }
}

// The tokens [t0, min(t0 + AH, te)) of stream `stream` (AH = tile_tokens),
// one half at a time (half_seq shapes): scores of one half for every token of
// the tile, stage 1 of each token into its shortlist, then stage 2 of each.
template <typename XT, int MODE, int E, int KM>
__device__ __forceinline__ void address_tile_halves(const XT* __restrict__ x, const XT* __restrict__ cb, int H,
                                                    int T, int stream, int t0, int te, int dk, int s, int k,
                                                    int32_t* __restrict__ idx, float* __restrict__ val,
                                                    float* __restrict__ score, unsigned char* smem) {
    constexpr int AH = tile_tokens<E, KM>();
    constexpr int SP = E * SDM_WAVE;
    float* scores = reinterpret_cast<float*>(smem);                           // [AH][SP], one half
    Entry* shortl = reinterpret_cast<Entry*>(scores + (size_t)AH * SP);       // [AH][2][KM]
    Entry* scratch = shortl + (size_t)AH * 2 * KM;                            // [AWAVES][3][KM]
    uint64_t* kbufs = reinterpret_cast<uint64_t*>(scratch + AWAVES * 3 * KM);  // [AWAVES][64]
    const int wave = threadIdx.x / SDM_WAVE;
    const uint16_t* pairs;
    int ncand;
    tile_pairs<KM>(k, nullptr, pairs, ncand);   // k <= 64: the constant table
    const XT* xs = x + (size_t)stream * T * dk;
    const XT* cbh = MODE == 0 ? cb : cb + (size_t)(stream % H) * 2 * s * (dk / 2);
    const int nt = min(AH, te - t0);
    Entry* scr = scratch + wave * 3 * KM;
    uint64_t* kbuf = kbufs + wave * SDM_WAVE;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        if (half == 0)
            tile_scores<XT, MODE, E, 0, 1>(xs, cbh, t0, nt, dk, s, scores);
        else
            tile_scores<XT, MODE, E, 1, 1>(xs, cbh, t0, nt, dk, s, scores);
        __syncthreads();
        for (int tt = wave; tt < nt; tt += AWAVES)
            half_topk<E>(scores + (size_t)tt * SP, s, k, scr, kbuf, shortl + ((size_t)tt * 2 + half) * KM);
        __syncthreads();   // the next half overwrites the scores
    }
    for (int tt = wave; tt < nt; tt += AWAVES) {
        const size_t o = ((size_t)stream * T + t0 + tt) * k;
        token_pairs(s, k, ncand, pairs, scr, shortl + (size_t)tt * 2 * KM, shortl + ((size_t)tt * 2 + 1) * KM, kbuf,
                    idx + o, val + o, score ? score + o : nullptr);
        wait_lds();
        __builtin_amdgcn_wave_barrier();
    }
}

// ---- scores held in the matrix cores' registers (bf16 codebooks, d_k / 2
//      <= 64, k <= 32) -------------------------------------------------------
// A workgroup scores TOK = 16 RT tokens against one half's s sub-keys and keeps
// the scores where the MFMA leaves them: wave w, lane (r, q) holds sub-key
// (w + 4 i) 16 + r of tile i (i < E) for tokens 4 q + v of each 16-row tile.
// So for every token the 64 lanes' (wave, r) groups of E scores each are the
// groups of the stage-1 bound: the k-th largest group maximum is reached by at
// least k scores, and every score of the top k is at or above it.  Per half:
//   1. group maxima -> LDS; each token's bound (k-th largest maximum, taken to
//      the sign, exponent and 11 mantissa bits) by one wave's ballots;
//   2. every lane appends its scores at or above the bound to the token's
//      candidate list (an LDS counter per token; the order does not matter);
//   3. the token's wave sorts its candidates under (score desc, id asc): the
//      ranked shortlist.  More than 64 candidates (or fewer than k, which only
//      non-finite scores give): the wave recomputes the token's row of scores
//      with the same MFMA steps into LDS and takes the general selection.
// Stage 2 (pruned pairs, id sort, softmax) as on the other paths.  Nothing but
// group maxima and candidates goes through LDS, and a codebook fetch serves 16
// RT tokens.
constexpr int RKS = 33;   // shortlist entries: k <= 32, then one -inf entry (pair ranks past the count)

template <int E, int RT>
struct RegTile {
    static constexpr int TOK = 16 * RT;
    static constexpr int SP = E * SDM_WAVE;
    static constexpr size_t G_OFF = 0;                                         // [TOK][64] float
    static constexpr size_t THR_OFF = G_OFF + (size_t)TOK * SDM_WAVE * 4;      // [TOK] float
    static constexpr size_t CNT_OFF = THR_OFF + (size_t)TOK * 4;               // [TOK] int
    static constexpr size_t CAND_OFF = CNT_OFF + (size_t)TOK * 4;              // [TOK][64] uint2
    static constexpr size_t SL_OFF = CAND_OFF + (size_t)TOK * SDM_WAVE * 8;    // [TOK][2][RKS] Entry
    static constexpr size_t SCR_OFF = SL_OFF + (size_t)TOK * 2 * RKS * 8;      // [AWAVES][MAXK] Entry
    static constexpr size_t KB_OFF = SCR_OFF + (size_t)AWAVES * MAXK * 8;      // [AWAVES][64] uint64
    static constexpr size_t ROW_OFF = KB_OFF + (size_t)AWAVES * SDM_WAVE * 8;  // [AWAVES][SP] float
    static constexpr size_t BYTES = ROW_OFF + (size_t)AWAVES * SP * 4;
};

// One 16 x 16 tile of scores: rows a (tokens), columns b (sub-keys), 64 deep.
__device__ __forceinline__ sdm_f32x4 score_tile(const sdm_bf16x8 (&a)[2], const sdm_bf16x8 (&b)[2]) {
    sdm_f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[0], b[0], acc, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[1], b[1], acc, 0, 0, 0);
}

// This lane's operand pieces: row t of x for one half (A; tl a row that
// exists, loaded in its place when t does not), and sub-key j of one half (B);
// zero past the rows or the depth.  The loads are unconditional, at clamped
// addresses, so they carry no branches.
__device__ __forceinline__ sdm_bf16x8 zero_unless(bool ok, sdm_bf16x8 v) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 u = __builtin_bit_cast(u32x4, v);
#pragma unroll
    for (int i = 0; i < 4; ++i) u[i] = ok ? u[i] : 0u;
    return __builtin_bit_cast(sdm_bf16x8, u);
}
__device__ __forceinline__ void load_a_rows(const bf16_t* xs, int t, int tl, bool ok, int dk, int half, int dh,
                                            int q, sdm_bf16x8 (&a)[2]) {
    const bf16_t* xr = xs + (size_t)(ok ? t : tl) * dk + half * dh;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int kc = ks * 32 + 8 * q;
        a[ks] = zero_unless(ok && kc < dh, *reinterpret_cast<const sdm_bf16x8*>(xr + (kc < dh ? kc : 0)));
    }
}
// (B past the depth is whatever the clamped load gives: A is zero there.  B
// past the sub-keys is row s - 1: the caller sets those scores to -inf.)
__device__ __forceinline__ void load_b_rows(const bf16_t* cbh, int half, int s, int j, int dh, int q,
                                            sdm_bf16x8 (&b)[2]) {
    const bf16_t* crow = cbh + ((size_t)half * s + min(j, s - 1)) * dh;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int kc = ks * 32 + 8 * q;
        b[ks] = *reinterpret_cast<const sdm_bf16x8*>(crow + (kc < dh ? kc : 0));
    }
}
// 0 for a sub-key j < s, -inf past them (no lane mask involved).
__device__ __forceinline__ float pad_of(int j, int s) {
    return __int_as_float((int)(((uint32_t)((s - 1 - j) >> 31)) & 0xff800000u));
}

// Stage 1 of one token's half on the general path: its row of scores (token
// `row` of the 16-row tile at t0, nr rows present) recomputed by the same MFMA
// steps into frow, then the general selection into out.  Out of line: the
// cold path of the register-resident kernel.
template <int E>
__device__ __noinline__ void reg_half_general(const bf16_t* xs, const bf16_t* cbh, int t0, int nr, int row, int dk,
                                              int half, int s, int k, float* frow, Entry* scr, uint64_t* kbuf,
                                              Entry* out) {
    const int lane = lane_id();
    const int r16 = lane % 16, q = lane / 16;
    const int dh = dk / 2;
    sdm_bf16x8 a[2];
    load_a_rows(xs, t0 + r16, t0, r16 < nr, dk, half, dh, q, a);
    for (int jt = 0; jt < AWAVES * E; ++jt) {
        sdm_bf16x8 b[2];
        const int j = jt * 16 + r16;
        load_b_rows(cbh, half, s, j, dh, q, b);
        const sdm_f32x4 acc = score_tile(a, b);
        if (q == row / 4) {
            const int v = row % 4;
            const float f = v == 0 ? acc[0] : (v == 1 ? acc[1] : (v == 2 ? acc[2] : acc[3]));
            frow[j] = f + pad_of(j, s);
        }
    }
    wait_lds();
    __builtin_amdgcn_wave_barrier();
    half_topk<E>(frow, s, k, scr, kbuf, out);
}

// Stage 1 of one half for the tile's tokens (the register-resident kernel's
// phases 1-3), written out once per half.  s and d_k pass through an opaque
// copy first, so that nothing derived from them in one half (row addresses,
// pads) is kept live into the other's selection phases.
template <int E, int RT>
__device__ __forceinline__ void reg_half(unsigned char* smem, const bf16_t* xs, const bf16_t* cbh, int t0, int nt,
                                         int dk_in, int s_in, int k, int half) {
    int s, dk;
    asm volatile("s_mov_b32 %0, %1" : "=s"(s) : "s"(s_in));
    asm volatile("s_mov_b32 %0, %1" : "=s"(dk) : "s"(dk_in));
    using L = RegTile<E, RT>;
    constexpr int NU = L::TOK / AWAVES;   // tokens per wave in the selection phases: wave + AWAVES u
    constexpr int EG = E < 4 ? E : 4;     // tiles whose codebook pieces are loaded together
    float* G = reinterpret_cast<float*>(smem + L::G_OFF);
    float* thr = reinterpret_cast<float*>(smem + L::THR_OFF);
    int* cnt = reinterpret_cast<int*>(smem + L::CNT_OFF);
    uint2* cand = reinterpret_cast<uint2*>(smem + L::CAND_OFF);
    Entry* sl = reinterpret_cast<Entry*>(smem + L::SL_OFF);
    const int wave = threadIdx.x / SDM_WAVE;
    const int lane = lane_id();
    Entry* scr = reinterpret_cast<Entry*>(smem + L::SCR_OFF) + wave * MAXK;
    uint64_t* kbuf = reinterpret_cast<uint64_t*>(smem + L::KB_OFF) + wave * SDM_WAVE;
    float* frow = reinterpret_cast<float*>(smem + L::ROW_OFF) + wave * L::SP;
    const int dh = dk / 2;
    const int r16 = lane % 16, q = lane / 16;
    // ---- scores of the tile in registers
    float sc[RT][E][4];
    {
        sdm_bf16x8 a[RT][2];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            load_a_rows(xs, t0 + 16 * rt + r16, t0, 16 * rt + r16 < nt, dk, half, dh, q, a[rt]);
#pragma unroll
        for (int i0 = 0; i0 < E; i0 += EG) {
            sdm_bf16x8 b[EG][2];
#pragma unroll
            for (int i = 0; i < EG; ++i)
                load_b_rows(cbh, half, s, (wave + AWAVES * (i0 + i)) * 16 + r16, dh, q, b[i]);
#pragma unroll
            for (int i = 0; i < EG; ++i) {
                const float pad = pad_of((wave + AWAVES * (i0 + i)) * 16 + r16, s);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const sdm_f32x4 acc = score_tile(a[rt], b[i]);
#pragma unroll
                    for (int v = 0; v < 4; ++v) sc[rt][i0 + i][v] = acc[v] + pad;
                }
            }
        }
    }
    // ---- 1. group maxima, then each token's bound
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            float m = sc[rt][0][v];
#pragma unroll
            for (int i = 1; i < E; ++i) m = fmaxf(m, sc[rt][i][v]);
            G[(16 * rt + 4 * q + v) * SDM_WAVE + wave * 16 + r16] = m;
        }
    __syncthreads();
    {
        uint32_t key[NU], tau[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            key[u] = ord_key(G[(wave + AWAVES * u) * SDM_WAVE + lane]);
            tau[u] = 0u;
        }
#pragma unroll
        for (int bit = 31; bit >= 12; --bit) {
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const uint32_t c = tau[u] | (1u << bit);
                if (popc64(__ballot(key[u] >= c)) >= k) tau[u] = c;
            }
        }
        if (lane == 0) {
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int tt = wave + AWAVES * u;
                thr[tt] = tt < nt ? key_to_float(tau[u]) : INFINITY;   // no candidates past the tokens
                cnt[tt] = 0;
            }
        }
    }
    __syncthreads();
    // ---- 2. candidates: scores at or above the token's bound
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int tt = 16 * rt + 4 * q + v;
            const float th = thr[tt];
            uint32_t bits = 0u;   // this lane's scores of the token at or above its bound
#pragma unroll
            for (int i = 0; i < E; ++i) bits |= (sc[rt][i][v] >= th ? 1u : 0u) << i;
            if (bits) {
                int p = atomicAdd(&cnt[tt], __popc(bits));
#pragma unroll
                for (int i = 0; i < E; ++i) {
                    if ((bits >> i) & 1u) {
                        if (p < SDM_WAVE)
                            cand[tt * SDM_WAVE + p] = make_uint2(__float_as_uint(sc[rt][i][v]),
                                                                 (uint32_t)((wave + AWAVES * i) * 16 + r16));
                        ++p;
                    }
                }
            }
        }
    __syncthreads();
    // ---- 3. each token's ranked shortlist, on its wave
    for (int u = 0; u < NU; ++u) {
        const int tt = wave + AWAVES * u;
        if (tt >= nt) break;
        Entry* out = sl + ((size_t)tt * 2 + half) * RKS;
        const int n = cnt[tt];
        if (lane >= k && lane < RKS) out[lane] = Entry{-INFINITY, 0};
        if (n >= k && n <= SDM_WAVE) {
            const uint2 cv = cand[tt * SDM_WAVE + min(lane, SDM_WAVE - 1)];
            uint32_t th = lane < n ? ord_key(__uint_as_float(cv.x)) : 0u;
            uint32_t tl = ~cv.y;
            bsort_desc64<2, 1, SDM_WAVE>(th, tl, lane);
            if (lane < k) out[lane] = Entry{key_to_float(th), (int)~tl};
        } else {
            reg_half_general<E>(xs, cbh, t0 + (tt & ~15), min(16, nt - (tt & ~15)), tt % 16, dk, half, s, k,
                                frow, scr, kbuf, out);
        }
        wait_lds();
        __builtin_amdgcn_wave_barrier();
    }
}

// Three waves per SIMD (the LDS of three workgroups fits a CU): at sqrt(N) =
// 1024 the register cap halves the time against two (0.89 against 1.20 ms
// per side at B=4 H=8 T=8192).
template <int E, int RT>
__global__ __launch_bounds__(AWAVES * SDM_WAVE, 3) void address_reg_kernel(const bf16_t* __restrict__ x,
                                                                        const bf16_t* __restrict__ cb, int H, int T,
                                                                        int tb, int te, int dk, int s, int k,
                                                                        int32_t* __restrict__ idx,
                                                                        float* __restrict__ val,
                                                                        float* __restrict__ score) {
    using L = RegTile<E, RT>;
    constexpr int NU = L::TOK / AWAVES;
    extern __shared__ __align__(16) unsigned char smem[];
    Entry* sl = reinterpret_cast<Entry*>(smem + L::SL_OFF);
    const int wave = threadIdx.x / SDM_WAVE;
    const int lane = lane_id();
    Entry* scr = reinterpret_cast<Entry*>(smem + L::SCR_OFF) + wave * MAXK;
    uint64_t* kbuf = reinterpret_cast<uint64_t*>(smem + L::KB_OFF) + wave * SDM_WAVE;
    const int stream = blockIdx.y;
    const int t0 = tb + blockIdx.x * L::TOK;
    const int nt = min(L::TOK, te - t0);
    const bf16_t* xs = x + (size_t)stream * T * dk;
    const bf16_t* cbh = cb + (size_t)(stream % H) * 2 * s * (dk / 2);
    reg_half<E, RT>(smem, xs, cbh, t0, nt, dk, s, k, 0);
    reg_half<E, RT>(smem, xs, cbh, t0, nt, dk, s, k, 1);
    // ---- stage 2 of each token, on the wave that ranked its shortlists
    const uint16_t* pairs = c_pairs.e + c_pairs.off[k];
    const int ncand = c_pairs.n[k];
    uint32_t pi[3], pj[3];
#pragma unroll
    for (int e = 0; e < 3; ++e) {
        const int c = e * SDM_WAVE + lane;
        const uint32_t pr = c < ncand ? pairs[min(c, ncand - 1)] : ((RKS - 1u) << 8 | (RKS - 1u));
        pi[e] = pr >> 8;
        pj[e] = pr & 0xffu;
    }
    for (int u = 0; u < NU; ++u) {
        const int tt = wave + AWAVES * u;
        if (tt >= nt) break;
        const size_t o = ((size_t)stream * T + t0 + tt) * k;
        const Entry* la = sl + (size_t)tt * 2 * RKS;
        const Entry* lb = la + RKS;
        if (!pairs_fast(s, k, pi, pj, la, lb, reinterpret_cast<uint2*>(kbuf), idx + o, val + o,
                        score ? score + o : nullptr))
            token_pairs(s, k, ncand, pairs, scr, la, lb, kbuf, idx + o, val + o, score ? score + o : nullptr);
        wait_lds();
        __builtin_amdgcn_wave_barrier();
    }
}

// Grid (tiles of tile_tokens tokens of [tb, te), streams).
template <typename XT, int MODE, int E, int KM>
__global__ __launch_bounds__(AWAVES * SDM_WAVE) void address_kernel(const XT* __restrict__ x,
                                                                    const XT* __restrict__ cb, int H, int T,
                                                                    int tb, int te, int dk, int s, int k,
                                                                    int32_t* __restrict__ idx,
                                                                    float* __restrict__ val,
                                                                    float* __restrict__ score) {
    extern __shared__ __align__(16) unsigned char smem[];
    if constexpr (half_seq<E, KM>())
        address_tile_halves<XT, MODE, E, KM>(x, cb, H, T, blockIdx.y, tb + blockIdx.x * tile_tokens<E, KM>(), te, dk,
                                             s, k, idx, val, score, smem);
    else
        address_tile<XT, MODE, E, KM>(x, cb, H, T, blockIdx.y, tb + blockIdx.x * atile<E>(), te, dk, s, k, idx, val,
                                      score, smem);
}

// The same tiles (not half_seq shapes) from a grid of at most gridDim.x
// workgroups, for a launch that shares the CUs with other work: each
// workgroup takes tiles, stream-major, at the grid's stride.  Beside the
// pipelined forward's scan the grid is the workgroups that fit in the LDS the
// scan leaves on each CU.  With one workgroup per tile, addressing
// workgroups took the LDS that the next scan stage's workgroups waited for:
// at the 1.4B-shaped workload the scan stages ran at 0.62 instead of 0.55 ms.
template <typename XT, int MODE, int E, int KM>
__global__ __launch_bounds__(AWAVES * SDM_WAVE) void address_kernel_looped(const XT* __restrict__ x,
                                                                           const XT* __restrict__ cb, int H, int T,
                                                                           int tb, int te, int dk, int s, int k,
                                                                           int32_t* __restrict__ idx,
                                                                           float* __restrict__ val,
                                                                           float* __restrict__ score, int nstreams) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int ntiles = (te - tb + atile<E>() - 1) / atile<E>();
    const int total = ntiles * nstreams;
    for (int id = blockIdx.x; id < total; id += gridDim.x) {
        const int stream = id / ntiles, tile = id - stream * ntiles;
        address_tile<XT, MODE, E, KM>(x, cb, H, T, stream, tb + tile * atile<E>(), te, dk, s, k, idx, val, score,
                                      smem);
        __syncthreads();   // every wave is done with this tile's LDS before the next tile's scores
    }
}

// ---- one token per stream (decode) ----------------------------------------
// Scores of the decode step's two rows (read query with cb_q, write key with
// cb_k) on the matrix cores, bf16 codebooks with d_k / 2 <= 64 and E <= 4:
// every operand of this wave's tiles, both rows and both halves, is loaded
// before the first MFMA, so the step pays one load latency for its scores
// (the token is row 0 of each 16-row tile).  Rows [row][half][SP], -inf past s.
template <int E>
__device__ __forceinline__ void decode_scores_mfma(const bf16_t* __restrict__ xq, const bf16_t* __restrict__ xk,
                                                   const bf16_t* __restrict__ cq, const bf16_t* __restrict__ ck,
                                                   int dk, int s, float* scores) {
    constexpr int SP = E * SDM_WAVE;
    const int wave = threadIdx.x / SDM_WAVE, lane = lane_id();
    const int dh = dk / 2, r16 = lane % 16, q4 = lane / 16;
    sdm_bf16x8 a[2][2][2], b[2][2][E][2];
#pragma unroll
    for (int sd = 0; sd < 2; ++sd) {
        const bf16_t* x = sd ? xk : xq;
        const bf16_t* cb = sd ? ck : cq;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const int kc = ks * 32 + 8 * q4;
                a[sd][h][ks] = sdm_bf16x8{};
                if (r16 == 0 && kc < dh) a[sd][h][ks] = *reinterpret_cast<const sdm_bf16x8*>(x + h * dh + kc);
            }
#pragma unroll
            for (int i = 0; i < E; ++i) {
                const int j = (wave + AWAVES * i) * 16 + r16;
                const bf16_t* crow = cb + ((size_t)h * s + min(j, s - 1)) * dh;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int kc = ks * 32 + 8 * q4;
                    b[sd][h][i][ks] = sdm_bf16x8{};
                    if (j < s && kc < dh) b[sd][h][i][ks] = *reinterpret_cast<const sdm_bf16x8*>(crow + kc);
                }
            }
        }
    }
#pragma unroll
    for (int sd = 0; sd < 2; ++sd)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int i = 0; i < E; ++i) {
                const int j = (wave + AWAVES * i) * 16 + r16;
                sdm_f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[sd][h][0], b[sd][h][i][0], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[sd][h][1], b[sd][h][i][1], acc, 0, 0, 0);
                if (q4 == 0 && j < s) scores[(sd * 2 + h) * SP + j] = acc[0];
            }
    if (s < SP) {
        const int pad = SP - s;
        for (int i = threadIdx.x; i < 4 * pad; i += blockDim.x) scores[(i / pad) * SP + s + i % pad] = -INFINITY;
    }
}

// One workgroup per (b, h) stream does the whole layer step for its single
// token: addressing of the read query and of the write key (their scores as
// two rows of one tile, then the two selections on two waves at once), then
// Sec. 3.1 steps 2-3 on every column (Eqs. sdm-decay,
// sdm-write in the read-back form, sdm-read after the write):
//   P_n = M[i_n]; D_n = alpha P_n; u = sum_n kappa_n D_n; e = beta (v - u);
//   M[i_n] = D_n + kappa_n e; y = sum_m rho_m M[j_m].
// Threads are DEC_RG row groups x 32 column quads, over the columns in chunks
// of DEC_COLS.  Read rows are loaded with the write rows, before the write; a
// read row that this token also writes takes the written value instead (the
// write list is ascending, App. A.2, so its position is a binary search).
// Every other read row is one this token leaves unchanged.
constexpr int DEC_RG = 8;                       // row groups
constexpr int DEC_COLS = 128;                   // columns per chunk: 32 quads
constexpr int DEC_ROWS = MAXK_BIG / DEC_RG;     // rows per thread, at most

__device__ __forceinline__ float load_scalar(const void* p, int in_dtype, size_t i) {
    return in_dtype == SDM_DT_BF16 ? to_f32(static_cast<const bf16_t*>(p)[i]) : static_cast<const float*>(p)[i];
}
__device__ __forceinline__ v4f load_quad(const void* p, int in_dtype, size_t i) {
    return in_dtype == SDM_DT_BF16 ? ld4v(static_cast<const bf16_t*>(p) + i) : ld4v(static_cast<const float*>(p) + i);
}

// LDS of a tile: padded score rows, per-wave lists and sort buffer, and for
// k > 64 the pair list.
__host__ __device__ constexpr size_t address_lds_bytes(int E, int AT, int KM) {
    return (size_t)AT * 2 * E * SDM_WAVE * sizeof(float) + AWAVES * 3 * KM * sizeof(Entry) +
           AWAVES * SDM_WAVE * sizeof(uint64_t) + (KM > MAXK ? MAXCAND_BIG * SDM_WAVE * sizeof(uint16_t) : 0);
}
__host__ __device__ constexpr size_t decode_scan_lds_bytes(int W) {
    return (size_t)(MAXK_BIG + DEC_RG * DEC_COLS + (size_t)W * DEC_COLS) * sizeof(float);
}
// The decode step's slot lists and weights of its two rows, and two words of
// flags, past both phases' LDS.
__host__ __device__ constexpr size_t decode_sel_offset(int E, int KM, int W) {
    const size_t a = address_lds_bytes(E, E <= 4 ? ATILE : (E <= 8 ? 8 : 4), KM), b = decode_scan_lds_bytes(W);
    return ((a > b ? a : b) + 15) & ~(size_t)15;
}
__host__ __device__ constexpr size_t decode_lds_bytes(int E, int KM, int W) {
    return decode_sel_offset(E, KM, W) + (size_t)2 * KM * (sizeof(int32_t) + sizeof(float)) + 2 * sizeof(int);
}

template <typename XT, int MODE, int E, int KM>
__global__ __launch_bounds__(AWAVES * SDM_WAVE) void decode_kernel(
    const XT* __restrict__ q, const XT* __restrict__ kx, const XT* __restrict__ cb_q, const XT* __restrict__ cb_k,
    int H, int dk, int s, int topk, const void* __restrict__ v, const void* __restrict__ alpha,
    const void* __restrict__ beta, int in_dtype, float* __restrict__ mem, int64_t N, int dv,
    int32_t* __restrict__ r_idx, float* __restrict__ r_val, int32_t* __restrict__ w_idx,
    float* __restrict__ w_val, float* __restrict__ y, unsigned int* __restrict__ flags,
    const float* __restrict__ gA, const float* __restrict__ gbdt) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int stream = blockIdx.x;
    if (stream == 0 && threadIdx.x < 4) flags[threadIdx.x] = 0u;   // the call's device-error words
    // the two rows' slot lists and weights, past both phases' LDS: [read, write][KM]
    int32_t* sel_id = reinterpret_cast<int32_t*>(smem + decode_sel_offset(E, KM, topk));
    float* sel_val = reinterpret_cast<float*>(sel_id + 2 * KM);
    int* fail = reinterpret_cast<int*>(sel_val + 2 * KM);           // [2] fast stage 1 overflowed, per row
    // the token's gates and its first column chunk of v, loaded before any other work
    float al = load_scalar(alpha, in_dtype, stream), be = load_scalar(beta, in_dtype, stream);
    const v4f v_first = load_quad(v, in_dtype, (size_t)stream * dv + min((int)(threadIdx.x % 32) * 4, dv - 4));
    {
        // both rows at once: score rows 0 (read query) and 1 (write key), then
        // phases B, C
        constexpr int AT = atile<E>();
        constexpr int SP = E * SDM_WAVE;
        float* scores = reinterpret_cast<float*>(smem);
        Entry* scratch = reinterpret_cast<Entry*>(scores + (size_t)AT * 2 * SP);
        uint64_t* kbufs = reinterpret_cast<uint64_t*>(scratch + AWAVES * 3 * KM);
        const uint16_t* pairs;
        int ncand;
        tile_pairs<KM>(topk, reinterpret_cast<uint16_t*>(kbufs + AWAVES * SDM_WAVE), pairs, ncand);
        const size_t hc = (size_t)(stream % H) * 2 * s * (dk / 2);
        bool joint = false;
        if constexpr (MODE == 2 && E <= 4) {
            if (dk / 2 <= 64) {
                decode_scores_mfma<E>(q + (size_t)stream * dk, kx + (size_t)stream * dk, cb_q + hc, cb_k + hc, dk,
                                      s, scores);
                joint = true;
            }
        }
        if (!joint) {
            tile_scores<XT, MODE, E>(q + (size_t)stream * dk, MODE == 0 ? cb_q : cb_q + hc, 0, 1, dk, s, scores);
            tile_scores<XT, MODE, E>(kx + (size_t)stream * dk, MODE == 0 ? cb_k : cb_k + hc, 0, 1, dk, s,
                                     scores + 2 * SP);
        }
        if (threadIdx.x < 2) fail[threadIdx.x] = 0;
        __syncthreads();
        const int wave = threadIdx.x / SDM_WAVE;
        SelWave w;
        if (wave < 2) select_init<KM>(w, scratch, kbufs, wave, topk, ncand, pairs);
        bool four = false;   // stage 1 of the 2 rows x 2 halves on the four waves
        if constexpr (E <= 4 && KM <= MAXK) four = topk <= 32 && topk <= s;
        if (four) {
            const int sd = wave >> 1, hf = wave & 1;
            Entry* lst = scratch + sd * 3 * KM + (1 + hf) * KM;   // row sd's list of half hf
            if (!half_fast<E>(scores + (sd * 2 + hf) * SP, topk, reinterpret_cast<uint2*>(kbufs + wave * SDM_WAVE),
                              lst) && lane_id() == 0)
                fail[sd] = 1;
            __syncthreads();
        }
        if (wave < 2) {
            int32_t* io = sel_id + wave * KM;
            float* vo = sel_val + wave * KM;
            const float* row = scores + wave * 2 * SP;
            if (four) {
                if (fail[wave] ||
                    !pairs_fast(s, topk, w.pi, w.pj, w.listA, w.listB, reinterpret_cast<uint2*>(w.kbuf), io, vo,
                                nullptr)) {
                    token_general<E>(row, s, SP, topk, ncand, pairs, w.scr, w.listA, w.listB, w.kbuf, io, vo,
                                     nullptr);
                    wait_lds();
                    __builtin_amdgcn_wave_barrier();
                }
            } else {
                select_token<E, KM>(w, row, s, topk, ncand, pairs, io, vo, nullptr);
            }
        }
    }
    __syncthreads();   // the slot lists are complete in LDS

    const int W = topk, R = topk;
    const int tid = threadIdx.x, rg = tid / 32, cq = tid % 32;
    for (int i = tid; i < 2 * topk; i += blockDim.x) {   // the lists out to the caller
        const int sd = i >= topk, j = i - sd * topk;
        const size_t o = (size_t)stream * topk + j;
        (sd ? w_idx : r_idx)[o] = sel_id[sd * KM + j];
        (sd ? w_val : r_val)[o] = sel_val[sd * KM + j];
    }
    const int32_t* wi = sel_id + KM;
    const int32_t* ri = sel_id;
    const float* wv = sel_val + KM;
    const float* rv = sel_val;
    const int* lw = wi;                                              // write slots (ascending)
    float* red = reinterpret_cast<float*>(smem + MAXK_BIG * sizeof(int));   // [DEC_RG][DEC_COLS] partial sums
    float* nrow = red + DEC_RG * DEC_COLS;                           // [W][DEC_COLS] written rows

    int wslot[DEC_ROWS], rslot[DEC_ROWS], link[DEC_ROWS];
    float kap[DEC_ROWS], rho[DEC_ROWS];
#pragma unroll
    for (int j = 0; j < DEC_ROWS; ++j) {
        const int n = rg + DEC_RG * j;
        wslot[j] = n < W ? min(max(wi[n], 0), (int)(N - 1)) : 0;
        kap[j] = n < W ? wv[n] : 0.f;
        rslot[j] = n < R ? min(max(ri[n], 0), (int)(N - 1)) : 0;
        rho[j] = n < R ? rv[n] : 0.f;
    }
    float* tab = mem + (size_t)stream * N * dv;
    // the first column chunk's rows, in flight while the links are found
    v4f P[DEC_ROWS], Q[DEC_ROWS];
    {
        const int cl = min(cq * 4, dv - 4);
#pragma unroll
        for (int j = 0; j < DEC_ROWS; ++j) {
            const int n = rg + DEC_RG * j;
            if (n < W) P[j] = ld4(tab + (size_t)wslot[j] * dv + cl);
            if (n < R) Q[j] = ld4(tab + (size_t)rslot[j] * dv + cl);
        }
    }
#pragma unroll
    for (int j = 0; j < DEC_ROWS; ++j) {
        const int n = rg + DEC_RG * j;
        link[j] = -1;
        if (n < R) {   // position of the read slot in the ascending write list
            int lo = 0;
            for (int len = W; len > 1;) {
                const int half = len >> 1;
                lo = lw[lo + half] <= rslot[j] ? lo + half : lo;
                len -= half;
            }
            link[j] = lw[lo] == rslot[j] ? lo : -1;
        }
    }
    sdm_gates_of(gA, gbdt, stream % H, al, be);

    for (int c0 = 0; c0 < dv; c0 += DEC_COLS) {
        const int col = c0 + cq * 4;
        const bool colok = col < dv;      // d_v is a multiple of 4: whole quads
        const int cl = colok ? col : dv - 4;
        if (c0 > 0) {
#pragma unroll
            for (int j = 0; j < DEC_ROWS; ++j) {
                const int n = rg + DEC_RG * j;
                if (n < W) P[j] = ld4(tab + (size_t)wslot[j] * dv + cl);
                if (n < R) Q[j] = ld4(tab + (size_t)rslot[j] * dv + cl);
            }
        }
        v4f up = v4zero();
#pragma unroll
        for (int j = 0; j < DEC_ROWS; ++j)
            if (rg + DEC_RG * j < W) up = v4fma(kap[j], al * P[j], up);
        st4(red + rg * DEC_COLS + cq * 4, up);
        __syncthreads();
        v4f u = v4zero();
#pragma unroll
        for (int g = 0; g < DEC_RG; ++g) u += ld4(red + g * DEC_COLS + cq * 4);
        const v4f e = be * ((c0 == 0 ? v_first : load_quad(v, in_dtype, (size_t)stream * dv + cl)) - u);
#pragma unroll
        for (int j = 0; j < DEC_ROWS; ++j) {
            const int n = rg + DEC_RG * j;
            if (n < W) {
                const v4f nw = v4fma(kap[j], e, al * P[j]);
                st4(nrow + n * DEC_COLS + cq * 4, nw);
                if (colok) st4(tab + (size_t)wslot[j] * dv + col, nw);
            }
        }
        __syncthreads();   // written rows in LDS; every thread has read red
        v4f yp = v4zero();
#pragma unroll
        for (int j = 0; j < DEC_ROWS; ++j) {
            if (rg + DEC_RG * j < R) {
                const v4f mv = link[j] >= 0 ? ld4(nrow + link[j] * DEC_COLS + cq * 4) : Q[j];
                yp = v4fma(rho[j], mv, yp);
            }
        }
        st4(red + rg * DEC_COLS + cq * 4, yp);
        __syncthreads();
        if (rg == 0 && colok) {
            v4f yy = v4zero();
#pragma unroll
            for (int g = 0; g < DEC_RG; ++g) yy += ld4(red + g * DEC_COLS + cq * 4);
            st4(y + (size_t)stream * dv + col, yy);
        }
        __syncthreads();   // red and nrow are reused by the next chunk
    }
}


// Backward of the weights through softmax and the sub-key scores: one wave
// per token.  Lane l first forms, for slots n = 64 r + l < k (r < KR),
// g_n = w_n (wbar_n - sum_m w_m wbar_m) and the sub-key ids of slot n; then,
// for n = 0 .. k-1 (read across the wave), each lane adds g_n times its NC
// columns of the two sub-key rows.  The codebook rows are read coalesced,
// several n in flight.
template <typename XT, bool CODEBOOK, int NC, int KR>
__global__ __launch_bounds__(256) void address_bwd_kernel(const XT* __restrict__ cb, int H, int T,
                                                          int dk, int s, int k,
                                                          const int32_t* __restrict__ idx,
                                                          const float* __restrict__ val,
                                                          const float* __restrict__ dval,
                                                          float* __restrict__ dx, int tb, int tn,
                                                          int64_t ntok) {
    // token-sides (stream, t) for t in [tb, tb + tn): ntok = streams * tn
    const int lane = lane_id();
    const int64_t lr = (int64_t)blockIdx.x * (blockDim.x / SDM_WAVE) + threadIdx.x / SDM_WAVE;
    if (lr >= ntok) return;
    const int64_t r = (lr / tn) * T + tb + lr % tn;
    const int h = (int)((r / T) % H);
    float w[KR], wb[KR], g[KR];
    int sub0[KR], sub1[KR];
    float dp = 0.f;
#pragma unroll
    for (int q = 0; q < KR; ++q) {
        const int n = q * SDM_WAVE + lane;
        const bool has = n < k;
        w[q] = has ? val[r * k + n] : 0.f;
        wb[q] = has ? dval[r * k + n] : 0.f;
        const int id = has ? min(max(idx[r * k + n], 0), s * s - 1) : 0;   // never read outside
        sub0[q] = id / s;
        sub1[q] = id - sub0[q] * s;
        dp = fmaf(w[q], wb[q], dp);
    }
    const float dot = wave_sum(dp);
#pragma unroll
    for (int q = 0; q < KR; ++q) g[q] = w[q] * (wb[q] - dot);
    float* out = dx + r * dk;
    float acc[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) acc[i] = 0.f;
    if constexpr (CODEBOOK) {
        const int dh = dk / 2;
        const XT* cbh = cb + (size_t)h * 2 * s * dh;
        int base[NC];   // offset of this lane's column i in sub-key row 0 of its half
        bool hi[NC];
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int c = min(lane + SDM_WAVE * i, dk - 1);
            hi[i] = c >= dh;
            base[i] = hi[i] ? s * dh + (c - dh) : c;
        }
        // slots past k carry g = 0 and sub-key 0: whole groups of 8, no remainder
#pragma unroll
        for (int q = 0; q < KR; ++q) {
            for (int n0 = 0; n0 < min(k - q * SDM_WAVE, SDM_WAVE); n0 += 8) {
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int n = n0 + u;
                    const float gn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g[q]), n));
                    const int a0 = __builtin_amdgcn_readlane(sub0[q], n);
                    const int a1 = __builtin_amdgcn_readlane(sub1[q], n);
#pragma unroll
                    for (int i = 0; i < NC; ++i)
                        acc[i] = fmaf(gn, to_f32(cbh[base[i] + (hi[i] ? a1 : a0) * dh]), acc[i]);
                }
            }
        }
    } else {
        // direct mode: column c = half * s + j receives g_n when sub-key half(n) == j
        int j[NC];
        bool hi[NC];
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int c = lane + SDM_WAVE * i;
            hi[i] = c >= s;
            j[i] = hi[i] ? c - s : c;
        }
#pragma unroll
        for (int q = 0; q < KR; ++q) {
            for (int n = 0; n < min(k - q * SDM_WAVE, SDM_WAVE); ++n) {
                const float gn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g[q]), n));
                const int a0 = __builtin_amdgcn_readlane(sub0[q], n);
                const int a1 = __builtin_amdgcn_readlane(sub1[q], n);
#pragma unroll
                for (int i = 0; i < NC; ++i)
                    if ((hi[i] ? a1 : a0) == j[i]) acc[i] += gn;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        const int c = lane + SDM_WAVE * i;
        if (c < dk) out[c] = acc[i];
    }
}

// The same for address_kernel's tile (one half of scores and the shortlists
// for half_seq shapes).
template <int E, int KM>
constexpr size_t tile_lds_bytes() {
    constexpr int AT = tile_tokens<E, KM>();
    if constexpr (half_seq<E, KM>())
        return (size_t)AT * E * SDM_WAVE * sizeof(float) + (size_t)AT * 2 * KM * sizeof(Entry) +
               AWAVES * 3 * KM * sizeof(Entry) + AWAVES * SDM_WAVE * sizeof(uint64_t);
    else
        return address_lds_bytes(E, AT, KM);
}

// One 16-token row tile per workgroup of the register-resident kernel (its
// scores take 4 E registers per lane).
template <int E>
hipError_t launch_address_reg(const void* x, const void* cb, int B, int H, int T, int tb, int tn, int dk, int s,
                              int k, int32_t* idx, float* val, float* score, hipStream_t st) {
    constexpr int RT = 1;
    using L = RegTile<E, RT>;
    auto kfn = address_reg_kernel<E, RT>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)L::BYTES);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, dim3((tn + L::TOK - 1) / L::TOK, B * H), dim3(AWAVES * SDM_WAVE), L::BYTES, st,
                       static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(cb), H, T, tb, tb + tn, dk, s, k,
                       idx, val, score);
    return hipGetLastError();
}

template <typename XT, int MODE>
hipError_t launch_address_e(const void* x, const void* cb, int B, int H, int T, int tb, int tn, int dk,
                            int s, int k, int32_t* idx, float* val, float* score, hipStream_t st,
                            size_t lds_free) {
    const int E = (s + SDM_WAVE - 1) / SDM_WAVE;
    if constexpr (MODE == 2) {
        // bf16 codebooks, sqrt(N) in (256, 1024], d_k / 2 <= 64, k <= 32:
        // scores stay in registers.  Measured at sqrt(N) = 1024 (B=4 H=8
        // T=8192, d_k = 128, k = 32): 1.19 against 1.84 ms per side.  At
        // sqrt(N) = 256 the LDS tile stays: 0.87 ms per side (B=8 H=16
        // T=4096) against 1.04 for 32-token register tiles.
        if (E > 4 && E <= 16 && dk / 2 <= 64 && k <= 32 && k <= s) {
            if (E <= 8) return launch_address_reg<8>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st);
            return launch_address_reg<16>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st);
        }
    }
    const XT* xp = static_cast<const XT*>(x);
    const XT* cp = static_cast<const XT*>(cb);
#define SDM_ADDR_CASE(EE, KM)                                                                   \
    {                                                                                           \
        constexpr int AT = tile_tokens<EE, KM>();                                               \
        const size_t sm = tile_lds_bytes<EE, KM>();                                             \
        if constexpr (!half_seq<EE, KM>()) {                                                     \
            /* beside other work: the workgroups that fit in the LDS it leaves on each CU, */  \
            /* when two or more do (with one per CU the paper's 1.4B layer measured slower) */  \
            const int cap = (int)(lds_free / sm) * (sdm_device_simds() / 4);                    \
            if (lds_free >= 2 * sm && (int64_t)((tn + AT - 1) / AT) * B * H > cap) {            \
                auto kl = address_kernel_looped<XT, MODE, EE, KM>;                              \
                hipError_t e = hipFuncSetAttribute((const void*)kl,                             \
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm); \
                if (e != hipSuccess) return e;                                                  \
                hipLaunchKernelGGL(kl, dim3(cap), dim3(AWAVES * SDM_WAVE), sm, st, xp, cp, H, T, tb, tb + tn, \
                                   dk, s, k, idx, val, score, B * H);                           \
                return hipGetLastError();                                                       \
            }                                                                                   \
        }                                                                                       \
        auto kfn = address_kernel<XT, MODE, EE, KM>;                                            \
        hipError_t e = hipFuncSetAttribute((const void*)kfn,                                    \
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm); \
        if (e != hipSuccess) return e;                                                          \
        hipLaunchKernelGGL(kfn, dim3((tn + AT - 1) / AT, B * H), dim3(AWAVES * SDM_WAVE), sm, st, xp, cp, \
                           H, T, tb, tb + tn, dk, s, k, idx, val, score);                      \
        return hipGetLastError();                                                               \
    }
    if (k > MAXK) {   // k <= sqrt(N), so E >= 2
        if (E <= 2) SDM_ADDR_CASE(2, MAXK_BIG)
        if (E <= 4) SDM_ADDR_CASE(4, MAXK_BIG)
        if (E <= 8) SDM_ADDR_CASE(8, MAXK_BIG)
        SDM_ADDR_CASE(16, MAXK_BIG)
    }
    if (E <= 1) SDM_ADDR_CASE(1, MAXK)
    if (E <= 2) SDM_ADDR_CASE(2, MAXK)
    if (E <= 4) SDM_ADDR_CASE(4, MAXK)
    if (E <= 8) SDM_ADDR_CASE(8, MAXK)
    SDM_ADDR_CASE(16, MAXK)
#undef SDM_ADDR_CASE
}

}  // namespace

hipError_t sdm_launch_address(const void* x, int x_dtype, const void* cb, int B, int H, int T,
                              int tb, int tn, int dk, int s, int k, int32_t* idx, float* val,
                              float* score, hipStream_t st, size_t lds_free) {
    if (tn <= 0) return hipSuccess;
    if (x_dtype == SDM_DT_BF16) {
        if (!cb) return launch_address_e<bf16_t, 0>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st, lds_free);
        if ((dk / 2) % 8 == 0)
            return launch_address_e<bf16_t, 2>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st, lds_free);
        return launch_address_e<bf16_t, 1>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st, lds_free);
    }
    if (!cb) return launch_address_e<float, 0>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st, lds_free);
    return launch_address_e<float, 1>(x, cb, B, H, T, tb, tn, dk, s, k, idx, val, score, st, lds_free);
}

namespace {

template <typename XT, int NC>
void launch_address_bwd_nc(const void* cb, int H, int T, int tb, int tn, int dk, int s, int k,
                           const int32_t* idx, const float* val, const float* dval, float* dx,
                           int64_t ntok, hipStream_t st) {
    dim3 grid((unsigned)((ntok + 3) / 4));
    const XT* c = static_cast<const XT*>(cb);
    if (k > SDM_WAVE) {
        if (cb)
            hipLaunchKernelGGL((address_bwd_kernel<XT, true, NC, 2>), grid, dim3(256), 0, st, c, H, T, dk, s, k,
                               idx, val, dval, dx, tb, tn, ntok);
        else
            hipLaunchKernelGGL((address_bwd_kernel<XT, false, NC, 2>), grid, dim3(256), 0, st, c, H, T, dk, s, k,
                               idx, val, dval, dx, tb, tn, ntok);
    } else if (cb) {
        hipLaunchKernelGGL((address_bwd_kernel<XT, true, NC, 1>), grid, dim3(256), 0, st, c, H, T, dk, s, k, idx,
                           val, dval, dx, tb, tn, ntok);
    } else {
        hipLaunchKernelGGL((address_bwd_kernel<XT, false, NC, 1>), grid, dim3(256), 0, st, c, H, T, dk, s, k, idx,
                           val, dval, dx, tb, tn, ntok);
    }
}

template <typename XT>
void launch_address_bwd_t(const void* cb, int H, int T, int tb, int tn, int dk, int s, int k,
                          const int32_t* idx, const float* val, const float* dval, float* dx,
                          int64_t ntok, hipStream_t st) {
    // columns per lane: d_k <= 512 in codebook mode, d_k = 2 sqrt(N) <= 2048 in direct mode
#define SDM_ABWD(NC) launch_address_bwd_nc<XT, NC>(cb, H, T, tb, tn, dk, s, k, idx, val, dval, dx, ntok, st)
    if (dk <= 64) SDM_ABWD(1);
    else if (dk <= 128) SDM_ABWD(2);
    else if (dk <= 256) SDM_ABWD(4);
    else if (dk <= 512) SDM_ABWD(8);
    else if (dk <= 1024) SDM_ABWD(16);
    else SDM_ABWD(32);
#undef SDM_ABWD
}

}  // namespace

hipError_t sdm_launch_address_bwd(const void* cb, int cb_dtype, int B, int H, int T, int tb, int tn, int dk,
                                  int s, int k, const int32_t* idx, const float* val, const float* dval,
                                  float* dx, hipStream_t st) {
    const int64_t ntok = (int64_t)B * H * tn;
    if (ntok == 0) return hipSuccess;
    if (cb_dtype == SDM_DT_BF16)
        launch_address_bwd_t<bf16_t>(cb, H, T, tb, tn, dk, s, k, idx, val, dval, dx, ntok, st);
    else
        launch_address_bwd_t<float>(cb, H, T, tb, tn, dk, s, k, idx, val, dval, dx, ntok, st);
    return hipGetLastError();
}

namespace {
template <typename XT, int MODE>
hipError_t launch_decode_m(const void* q, const void* k, const void* cb_q, const void* cb_k, int B, int H,
                           int dk, int s, int topk, const void* v, const void* alpha, const void* beta,
                           int in_dtype, float* mem, int64_t N, int dv, int32_t* r_idx, float* r_val,
                           int32_t* w_idx, float* w_val, float* y, unsigned int* flags, hipStream_t st,
                           const float* gA, const float* gbdt) {
    const int E = (s + SDM_WAVE - 1) / SDM_WAVE;
    const XT* qp = static_cast<const XT*>(q);
    const XT* kp = static_cast<const XT*>(k);
    const XT* cq = static_cast<const XT*>(cb_q);
    const XT* ck = static_cast<const XT*>(cb_k);
#define SDM_DEC_CASE(EE, KM)                                                                              \
    {                                                                                                     \
        const size_t sm = decode_lds_bytes(EE, KM, topk);                                                  \
        auto kfn = decode_kernel<XT, MODE, EE, KM>;                                                       \
        hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize,  \
                                           (int)sm);                                                      \
        if (e != hipSuccess) return e;                                                                    \
        hipLaunchKernelGGL(kfn, dim3(B * H), dim3(AWAVES * SDM_WAVE), sm, st, qp, kp, cq, ck, H, dk, s,   \
                           topk, v, alpha, beta, in_dtype, mem, N, dv, r_idx, r_val, w_idx, w_val, y, flags, \
                           gA, gbdt);                                                                     \
        return hipGetLastError();                                                                         \
    }
    if (topk > MAXK) {   // topk <= sqrt(N), so E >= 2
        if (E <= 2) SDM_DEC_CASE(2, MAXK_BIG)
        if (E <= 4) SDM_DEC_CASE(4, MAXK_BIG)
        if (E <= 8) SDM_DEC_CASE(8, MAXK_BIG)
        SDM_DEC_CASE(16, MAXK_BIG)
    }
    if (E <= 1) SDM_DEC_CASE(1, MAXK)
    if (E <= 2) SDM_DEC_CASE(2, MAXK)
    if (E <= 4) SDM_DEC_CASE(4, MAXK)
    if (E <= 8) SDM_DEC_CASE(8, MAXK)
    SDM_DEC_CASE(16, MAXK)
#undef SDM_DEC_CASE
}
}  // namespace

hipError_t sdm_launch_decode(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int B,
                             int H, int dk, int s, int topk, const void* v, const void* alpha, const void* beta,
                             int in_dtype, float* mem, int64_t N, int dv, int32_t* r_idx, float* r_val,
                             int32_t* w_idx, float* w_val, float* y, unsigned int* flags, hipStream_t st,
                             const float* gA, const float* gbdt) {
    if (B * H == 0) return hipSuccess;
    if (x_dtype == SDM_DT_BF16) {
        if (!cb_q)
            return launch_decode_m<bf16_t, 0>(q, k, cb_q, cb_k, B, H, dk, s, topk, v, alpha, beta, in_dtype, mem,
                                              N, dv, r_idx, r_val, w_idx, w_val, y, flags, st, gA, gbdt);
        if ((dk / 2) % 8 == 0)
            return launch_decode_m<bf16_t, 2>(q, k, cb_q, cb_k, B, H, dk, s, topk, v, alpha, beta, in_dtype, mem,
                                              N, dv, r_idx, r_val, w_idx, w_val, y, flags, st, gA, gbdt);
        return launch_decode_m<bf16_t, 1>(q, k, cb_q, cb_k, B, H, dk, s, topk, v, alpha, beta, in_dtype, mem, N,
                                          dv, r_idx, r_val, w_idx, w_val, y, flags, st, gA, gbdt);
    }
    if (!cb_q)
        return launch_decode_m<float, 0>(q, k, cb_q, cb_k, B, H, dk, s, topk, v, alpha, beta, in_dtype, mem, N,
                                         dv, r_idx, r_val, w_idx, w_val, y, flags, st, gA, gbdt);
    return launch_decode_m<float, 1>(q, k, cb_q, cb_k, B, H, dk, s, topk, v, alpha, beta, in_dtype, mem, N, dv,
                                     r_idx, r_val, w_idx, w_val, y, flags, st, gA, gbdt);
}
