// Per-token records for the forward and backward scans (the read-after-write
// staging step), for gfx950.
//
// One workgroup handles PT consecutive tokens of one (b, h) stream.  Slot ids
// are clamped to [0, N) (a bad id is flagged, never dereferenced).  For every
// row a scan token reads, the record says where its current value lives when
// the token in flight that last modified it is still inside the scan's
// prefetch window: the link (d << 8 | entry) names that token (d tokens
// away) and its ring entry; -1 means the row is read from HBM.
//
// Links come from pairwise intersections of slot lists.  Addressing returns
// each list sorted by slot id, so an intersection is the two-pointer merge of
// App. A.2 (O(W + R)); lists that are not sorted fall back to all pairs.
// Several intersections can hit the same row; atomicMin on an order key
// keeps the one the scan would see last.  Records are then written out word
// by word, coalesced.
#include <climits>

#include "sdm_common.h"
#include "sdm_internal.h"

namespace {

constexpr int PT = 64;   // tokens per workgroup

__device__ __forceinline__ bool strictly_sorted(const int* a, int n) {
    for (int i = 1; i < n; ++i)
        if (a[i] <= a[i - 1]) return false;
    return true;
}

// Calls f(a, b) for every A[a] == B[b].
template <typename F>
__device__ __forceinline__ void intersect(const int* A, int na, bool sa, const int* B, int nb, bool sb,
                                          F f) {
    if (sa && sb) {
        int a = 0, b = 0;
        while (a < na && b < nb) {
            const int x = A[a], y = B[b];
            if (x == y) {
                f(a, b);
                ++a;
                ++b;
            } else if (x < y) {
                ++a;
            } else {
                ++b;
            }
        }
    } else {
        for (int a = 0; a < na; ++a)
            for (int b = 0; b < nb; ++b)
                if (A[a] == B[b]) f(a, b);
    }
}

__device__ __forceinline__ int clamp_slot(int s, int64_t N, unsigned int& bad) {
    if (s < 0 || s >= N) {
        bad = 1u;
        return 0;
    }
    return s;
}

__device__ __forceinline__ void load_gates(const void* alpha, const void* beta, int in_dtype,
                                           size_t o, float& al, float& be) {
    if (in_dtype == SDM_DT_BF16) {
        al = to_f32(static_cast<const bf16_t*>(alpha)[o]);
        be = to_f32(static_cast<const bf16_t*>(beta)[o]);
    } else {
        al = static_cast<const float*>(alpha)[o];
        be = static_cast<const float*>(beta)[o];
    }
}

// ---------------------------------------------------------------- forward
// Token t, write row n: latest writer t-d, 1 <= d < PD, of the same slot.
// Token t, read row m: latest writer t-d, 0 <= d < PD (d = 0: t itself).
// Entry = position of the slot in that writer's write list.
template <int PD>
__global__ __launch_bounds__(256) void fwd_prep_kernel(const int32_t* __restrict__ w_idx,
                                                       const float* __restrict__ w_val,
                                                       const int32_t* __restrict__ r_idx,
                                                       const float* __restrict__ r_val,
                                                       const void* __restrict__ alpha,
                                                       const void* __restrict__ beta, int in_dtype,
                                                       int T, int W, int R, int64_t N,
                                                       unsigned char* __restrict__ recs,
                                                       unsigned int* __restrict__ err) {
    extern __shared__ int sm[];
    const FwdRec L = fwd_rec_layout(W, R);
    const int stream = blockIdx.y;
    const int t0 = blockIdx.x * PT;
    const int tb = t0 - (PD - 1);           // first token whose write list is needed
    const int ntok = min(PT, T - t0);
    const int nw = ntok + PD - 1;           // write lists held
    const int nrow = W + R;
    int* wl = sm;                           // [nw][W]
    int* rl = wl + (PT + PD - 1) * W;       // [ntok][R]
    int* lk = rl + PT * R;                  // [ntok][W + R] order keys
    int* wsorted = lk + PT * nrow;          // [nw]
    int* rsorted = wsorted + PT + PD - 1;   // [ntok]
    const size_t sbase = (size_t)stream * T;
    unsigned int bad = 0u;

    for (int i = threadIdx.x; i < nw * W; i += blockDim.x) {
        const int t = tb + i / W;
        wl[i] = t >= 0 ? clamp_slot(w_idx[(sbase + t) * W + i % W], N, bad) : -1;
    }
    for (int i = threadIdx.x; i < ntok * R; i += blockDim.x)
        rl[i] = clamp_slot(r_idx[(sbase + t0) * R + i], N, bad);
    for (int i = threadIdx.x; i < PT * nrow; i += blockDim.x) lk[i] = INT_MAX;
    __syncthreads();
    for (int i = threadIdx.x; i < nw + ntok; i += blockDim.x) {
        if (i < nw)
            wsorted[i] = strictly_sorted(wl + i * W, W);
        else
            rsorted[i - nw] = strictly_sorted(rl + (i - nw) * R, R);
    }
    __syncthreads();

    const int nj = (PD - 1) + PD;   // write-write d = 1..PD-1, read-write d = 0..PD-1
    for (int j = threadIdx.x; j < ntok * nj; j += blockDim.x) {
        const int tl = j / nj, kind = j % nj;
        const bool wr = kind < PD - 1;
        const int d = wr ? kind + 1 : kind - (PD - 1);
        if (t0 + tl - d < 0) continue;
        const int src = tl + PD - 1 - d;   // write list of token t - d
        int* keys = lk + tl * nrow;
        if (wr) {
            intersect(wl + (tl + PD - 1) * W, W, wsorted[tl + PD - 1], wl + src * W, W, wsorted[src],
                      [&](int a, int b) { atomicMin(&keys[a], (d << 8) | b); });
        } else {
            intersect(rl + tl * R, R, rsorted[tl], wl + src * W, W, wsorted[src],
                      [&](int a, int b) { atomicMin(&keys[W + a], (d << 8) | b); });
        }
    }
    __syncthreads();

    // records, one 32-bit word per thread step
    const int words = L.bytes / 4;
    uint32_t* out = reinterpret_cast<uint32_t*>(recs + (sbase + t0) * L.bytes);
    for (int i = threadIdx.x; i < ntok * words; i += blockDim.x) {
        const int tl = i / words, off = (i % words) * 4;
        const size_t tok = sbase + t0 + tl;
        uint32_t v = 0u;
        if (off < L.off_wval) {
            v = (uint32_t)wl[(tl + PD - 1) * W + off / 4];
        } else if (off < L.off_rslot) {
            v = __float_as_uint(w_val[tok * W + (off - L.off_wval) / 4]);
        } else if (off < L.off_rval) {
            v = (uint32_t)rl[tl * R + (off - L.off_rslot) / 4];
        } else if (off < L.off_link) {
            v = __float_as_uint(r_val[tok * R + (off - L.off_rval) / 4]);
        } else if (off < L.off_link + 2 * nrow) {
            const int e = (off - L.off_link) / 2;   // two int16 links per word
            const int k0 = lk[tl * nrow + e];
            const int k1 = e + 1 < nrow ? lk[tl * nrow + e + 1] : INT_MAX;
            const uint32_t l0 = k0 == INT_MAX ? 0xffffu : (uint32_t)k0 & 0xffffu;
            const uint32_t l1 = k1 == INT_MAX ? 0xffffu : (uint32_t)k1 & 0xffffu;
            v = l0 | (l1 << 16);
        } else if (off == L.off_ab || off == L.off_ab + 4) {
            float al, be;
            load_gates(alpha, beta, in_dtype, tok, al, be);
            v = __float_as_uint(off == L.off_ab ? al : be);
        }
        out[i] = v;
    }
    if (bad) atomicOr(err, 1u);
}

// ---------------------------------------------------------------- backward
// The backward visits t = T-1 .. 0.  For token t:
//  lm[m]  (M_t[j_m]): the earliest later writer t+d, 1 <= d < PD, whose undo
//         restored the row; entry n = its write position.
//  lgr[m] (G[j_m]) and lgw[n] (G[i_n]): the earliest later token t+d that
//         changed the adjoint row, either by its write adjoint (entry R + n,
//         preferred within one token: it runs after the read adjoint) or by
//         its read adjoint (entry m).  For lgw, d = 0 with a read entry means
//         this token's own read adjoint, which runs first.
// Order keys: ((2 d + is_read) << 8) | entry, so atomicMin keeps the row's
// current source.
template <int PD>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const int32_t* __restrict__ w_idx,
                                                       const float* __restrict__ w_val,
                                                       const int32_t* __restrict__ r_idx,
                                                       const float* __restrict__ r_val,
                                                       const void* __restrict__ alpha,
                                                       const void* __restrict__ beta, int in_dtype,
                                                       int T, int W, int R, int64_t N,
                                                       unsigned char* __restrict__ recs,
                                                       unsigned int* __restrict__ err) {
    extern __shared__ int sm[];
    const BwdRec L = bwd_rec_layout(W, R);
    const int stream = blockIdx.y;
    const int t0 = blockIdx.x * PT;
    const int ntok = min(PT, T - t0);
    const int span = min(PT + PD - 1, T - t0);   // tokens t0 .. t0+span-1 (later ones included)
    const int nrow = W + R;
    int* wl = sm;                                // [span][W]
    int* rl = wl + (PT + PD - 1) * W;            // [span][R]
    int* km = rl + (PT + PD - 1) * R;            // [ntok][R]  lm keys
    int* kgr = km + PT * R;                      // [ntok][R]  lgr keys
    int* kgw = kgr + PT * R;                     // [ntok][W]  lgw keys
    int* wsorted = kgw + PT * W;                 // [span]
    int* rsorted = wsorted + PT + PD - 1;        // [span]
    const size_t sbase = (size_t)stream * T;
    unsigned int bad = 0u;

    for (int i = threadIdx.x; i < span * W; i += blockDim.x)
        wl[i] = clamp_slot(w_idx[(sbase + t0) * W + i], N, bad);
    for (int i = threadIdx.x; i < span * R; i += blockDim.x)
        rl[i] = clamp_slot(r_idx[(sbase + t0) * R + i], N, bad);
    for (int i = threadIdx.x; i < PT * (2 * R + W); i += blockDim.x) km[i] = INT_MAX;   // km, kgr, kgw
    __syncthreads();
    for (int i = threadIdx.x; i < 2 * span; i += blockDim.x) {
        if (i < span)
            wsorted[i] = strictly_sorted(wl + i * W, W);
        else
            rsorted[i - span] = strictly_sorted(rl + (i - span) * R, R);
    }
    __syncthreads();

    // jobs per token: d = 0: (w(t), r(t)); d = 1..PD-1: (r(t), w(t+d)), (r(t), r(t+d)),
    // (w(t), w(t+d)), (w(t), r(t+d))
    const int nj = 1 + 4 * (PD - 1);
    for (int j = threadIdx.x; j < ntok * nj; j += blockDim.x) {
        const int tl = j / nj, kind = j % nj;
        const int* wt = wl + tl * W;
        const int* rt = rl + tl * R;
        if (kind == 0) {
            intersect(wt, W, wsorted[tl], rt, R, rsorted[tl],
                      [&](int n, int m) { atomicMin(&kgw[tl * W + n], (1 << 8) | m); });
            continue;
        }
        const int d = (kind - 1) / 4 + 1, q = (kind - 1) % 4;
        if (tl + d >= span) continue;   // past the end of the sequence
        const int u = tl + d;
        const int* wu = wl + u * W;
        const int* ru = rl + u * R;
        if (q == 0) {
            intersect(rt, R, rsorted[tl], wu, W, wsorted[u], [&](int m, int n) {
                atomicMin(&km[tl * R + m], (d << 8) | n);
                atomicMin(&kgr[tl * R + m], ((2 * d) << 8) | (R + n));
            });
        } else if (q == 1) {
            intersect(rt, R, rsorted[tl], ru, R, rsorted[u],
                      [&](int m, int m2) { atomicMin(&kgr[tl * R + m], ((2 * d + 1) << 8) | m2); });
        } else if (q == 2) {
            intersect(wt, W, wsorted[tl], wu, W, wsorted[u],
                      [&](int n, int n2) { atomicMin(&kgw[tl * W + n], ((2 * d) << 8) | (R + n2)); });
        } else {
            intersect(wt, W, wsorted[tl], ru, R, rsorted[u],
                      [&](int n, int m2) { atomicMin(&kgw[tl * W + n], ((2 * d + 1) << 8) | m2); });
        }
    }
    __syncthreads();

    const int words = L.bytes / 4;
    uint32_t* out = reinterpret_cast<uint32_t*>(recs + (sbase + t0) * L.bytes);
    // order key -> link (d << 8 | entry); -1 when no source inside the window
    auto link_of = [](int key, bool two_d) -> uint32_t {
        if (key == INT_MAX) return 0xffffu;
        const int d = two_d ? (key >> 9) : (key >> 8);
        return (uint32_t)((d << 8) | (key & 255)) & 0xffffu;
    };
    const int nlink = 2 * R + W;
    for (int i = threadIdx.x; i < ntok * words; i += blockDim.x) {
        const int tl = i / words, off = (i % words) * 4;
        const size_t tok = sbase + t0 + tl;
        uint32_t v = 0u;
        if (off < L.off_wval) {
            v = (uint32_t)wl[tl * W + off / 4];
        } else if (off < L.off_rslot) {
            v = __float_as_uint(w_val[tok * W + (off - L.off_wval) / 4]);
        } else if (off < L.off_rval) {
            v = (uint32_t)rl[tl * R + (off - L.off_rslot) / 4];
        } else if (off < L.off_lm) {
            v = __float_as_uint(r_val[tok * R + (off - L.off_rval) / 4]);
        } else if (off < L.off_lm + 2 * nlink) {
            const int e = (off - L.off_lm) / 2;
            auto at = [&](int ee) -> uint32_t {
                if (ee >= nlink) return 0xffffu;
                if (ee < R) return link_of(km[tl * R + ee], false);
                if (ee < 2 * R) return link_of(kgr[tl * R + ee - R], true);
                return link_of(kgw[tl * W + ee - 2 * R], true);
            };
            v = at(e) | (at(e + 1) << 16);
        } else if (off == L.off_ab || off == L.off_ab + 4) {
            float al, be;
            load_gates(alpha, beta, in_dtype, tok, al, be);
            v = __float_as_uint(off == L.off_ab ? al : be);
        }
        out[i] = v;
    }
    if (bad) atomicOr(err, 1u);
}

template <int PD>
size_t fwd_prep_lds(int W, int R) {
    return sizeof(int) * ((size_t)(PT + PD - 1) * W + (size_t)PT * R + (size_t)PT * (W + R) +
                          (PT + PD - 1) + PT);
}
template <int PD>
size_t bwd_prep_lds(int W, int R) {
    return sizeof(int) * ((size_t)(PT + PD - 1) * (W + R) + (size_t)PT * (2 * R + W) +
                          2 * (PT + PD - 1));
}

}  // namespace

template <int PD>
hipError_t sdm_launch_fwd_prep(const ScanFwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H;
    dim3 grid((a.T + PT - 1) / PT, S);
    const size_t sm = fwd_prep_lds<PD>(a.W, a.R);
    auto kfn = fwd_prep_kernel<PD>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, grid, dim3(256), sm, st, a.w_idx, a.w_val, a.r_idx, a.r_val, a.alpha,
                       a.beta, a.in_dtype, a.T, a.W, a.R, a.N, a.ws + SDM_WS_HEADER,
                       reinterpret_cast<unsigned int*>(a.ws));
    return hipGetLastError();
}

template <int PD>
hipError_t sdm_launch_bwd_prep(const ScanBwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H;
    dim3 grid((a.T + PT - 1) / PT, S);
    const size_t sm = bwd_prep_lds<PD>(a.W, a.R);
    auto kfn = bwd_prep_kernel<PD>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, grid, dim3(256), sm, st, a.w_idx, a.w_val, a.r_idx, a.r_val, a.alpha,
                       a.beta, a.in_dtype, a.T, a.W, a.R, a.N, a.ws + SDM_WS_HEADER,
                       reinterpret_cast<unsigned int*>(a.ws));
    return hipGetLastError();
}

template hipError_t sdm_launch_fwd_prep<SDM_FWD_PD>(const ScanFwdArgs&, hipStream_t);
template hipError_t sdm_launch_bwd_prep<SDM_BWD_PD>(const ScanBwdArgs&, hipStream_t);
