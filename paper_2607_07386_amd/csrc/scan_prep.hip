// Per-token records for the forward and backward scans (the read-after-write
// staging step), for gfx950.
//
// One workgroup handles PT consecutive tokens of one (b, h) stream.  Slot ids
// are clamped to [0, N) (a bad id is flagged, never dereferenced).  For every
// row a scan token reads, the record says where its current value lives when
// the token in flight that last modified it is still inside the scan's
// prefetch window: the forward's link is that token's row in the scan's ring
// ((t - d) mod PD) W + entry, d tokens away; the backward's names the token and
// entry as (d << 8 | entry); -1 means the row is read from HBM.
//
// One thread per (token, row) searches the slot lists of the candidate tokens
// in the window.  Addressing returns every list in ascending slot order, so a
// search is a fixed-length branch-free binary search (ceil(log2 W) LDS reads,
// the same for every lane); a list that is not strictly increasing is
// searched linearly instead (first occurrence).  Candidates are visited
// farthest first and a hit overwrites, so the nearest one wins without a
// data-dependent exit.  Records are then written out word by word, coalesced
// (the backward's in 16-byte pieces when W and R are multiples of 8; the same
// pieces for the forward's measured slower in the pipelined forward, where the
// record writes share the device with the scan: 6.71 against 6.63 ms per step).
#include "sdm_common.h"
#include "sdm_internal.h"

namespace {

constexpr int PT = 64;   // tokens per workgroup

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

// Position of slot in lst[0, n), or -1.  srt: lst is strictly increasing.
__device__ __forceinline__ int find_slot(const int* lst, int n, bool srt, int slot) {
    if (srt) {
        int lo = 0;
        for (int len = n; len > 1;) {
            const int half = len >> 1;
            lo = lst[lo + half] <= slot ? lo + half : lo;
            len -= half;
        }
        return lst[lo] == slot ? lo : -1;
    }
    for (int i = 0; i < n; ++i)
        if (lst[i] == slot) return i;
    return -1;
}

// srt[l] = 1 when list l of the n lists [nl][len] in lst is strictly increasing.
__device__ __forceinline__ void mark_sorted(const int* lst, int nl, int len, int* srt) {
    for (int i = threadIdx.x; i < nl; i += blockDim.x) srt[i] = 1;
    __syncthreads();
    for (int i = threadIdx.x; i < nl * len; i += blockDim.x)
        if (i % len != 0 && lst[i] <= lst[i - 1]) srt[i / len] = 0;
}

// ---------------------------------------------------------------- forward
// Token t, row n of either list: the latest writer t-d, 1 <= d < PD, of the
// same slot, as that writer's row in the scan's ring of written rows,
// ((t - d) mod PD) W + e, with e the position of the slot in its write list,
// so the scan reads the ring without index arithmetic.  A read row whose slot
// token t itself writes (entry n) ends the token at alpha P + kappa_n e, with P
// the slot's value before the token, which is where the link points: its
// weight in the record is rho alpha, and the token's record holds
// yc = sum of rho kappa_n over such rows, so that y = sum rho' P + yc e needs
// nothing the token writes.  Records are made for tokens [ta, te) of each
// stream; writers before ta are not linked (a scan started at ta finds their
// rows in HBM).
template <int PD>
__global__ __launch_bounds__(256) void fwd_prep_kernel(const int32_t* __restrict__ w_idx,
                                                       const float* __restrict__ w_val,
                                                       const int32_t* __restrict__ r_idx,
                                                       const float* __restrict__ r_val,
                                                       const void* __restrict__ alpha,
                                                       const void* __restrict__ beta, int in_dtype,
                                                       int T, int ta, int te, int W, int R, int64_t N,
                                                       unsigned char* __restrict__ recs,
                                                       unsigned int* __restrict__ err,
                                                       const float* __restrict__ gA,
                                                       const float* __restrict__ gbdt, int H) {
    extern __shared__ __align__(16) int sm[];
    const FwdRec L = fwd_rec_layout(W, R);
    const int stream = blockIdx.y;
    const int t0 = ta + blockIdx.x * PT;
    const int tb = t0 - (PD - 1);           // first token whose write list is needed
    const int ntok = min(PT, te - t0);
    const int nw = ntok + PD - 1;           // write lists held
    const int nrow = W + R;
    int* wl = sm;                                        // [PT+PD-1][W]
    int* rl = wl + (PT + PD - 1) * W;                    // [PT][R]
    int* wsrt = rl + PT * R;                             // [PT+PD-1]
    const int MW = (R + 31) / 32;
    unsigned int* omask = reinterpret_cast<unsigned int*>(wsrt + PT + PD - 1);   // [PT][MW]: read rows the token writes
    short* lk = reinterpret_cast<short*>(omask + PT * MW);       // [PT][W + R] links
    const size_t sbase = (size_t)stream * T;
    unsigned int bad = 0u;
    for (int i = threadIdx.x; i < PT * MW; i += blockDim.x) omask[i] = 0u;

    for (int i = threadIdx.x; i < nw * W; i += blockDim.x) {
        const int t = tb + i / W;
        wl[i] = t >= ta ? clamp_slot(w_idx[(sbase + t) * W + i % W], N, bad) : -1;
    }
    for (int i = threadIdx.x; i < ntok * R; i += blockDim.x)
        rl[i] = clamp_slot(r_idx[(sbase + t0) * R + i], N, bad);
    __syncthreads();
    mark_sorted(wl, nw, W, wsrt);
    __syncthreads();

    for (int i = threadIdx.x; i < ntok * nrow; i += blockDim.x) {
        const int tl = i / nrow, r = i % nrow;
        const bool wrow = r < W;
        const int slot = wrow ? wl[(tl + PD - 1) * W + r] : rl[tl * R + (r - W)];
        const int dhi = min(PD - 1, t0 + tl - ta);   // no writer before token ta
        short link = -1;
        for (int d = dhi; d >= 1; --d) {
            const int u = tl + PD - 1 - d;       // write list of token t - d
            const int n = find_slot(wl + u * W, W, wsrt[u] != 0, slot);
            if (n >= 0) link = (short)(((t0 + tl - d) & (PD - 1)) * W + n);   // ring row of (t - d, n)
        }
        lk[i] = link;
        if (!wrow) {
            const int u = tl + PD - 1, m = r - W;   // this token's own write list
            if (find_slot(wl + u * W, W, wsrt[u] != 0, slot) >= 0) atomicOr(&omask[tl * MW + m / 32], 1u << (m % 32));
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
            const int m = (off - L.off_rval) / 4;
            float rho = r_val[tok * R + m];
            if ((omask[tl * MW + m / 32] >> (m % 32)) & 1u) {   // rare: rho alpha
                float al, be;
                load_gates(alpha, beta, in_dtype, tok, al, be);
                sdm_gates_of(gA, gbdt, stream % H, al, be);
                rho *= al;
            }
            v = __float_as_uint(rho);
        } else if (off < L.off_link + 2 * nrow) {
            const int e = (off - L.off_link) / 2;   // two int16 links per word
            const uint32_t l0 = (uint16_t)lk[tl * nrow + e];
            const uint32_t l1 = e + 1 < nrow ? (uint16_t)lk[tl * nrow + e + 1] : 0xffffu;
            v = l0 | (l1 << 16);
        } else if (off == L.off_ab || off == L.off_ab + 4) {
            float al, be;
            load_gates(alpha, beta, in_dtype, tok, al, be);
            sdm_gates_of(gA, gbdt, stream % H, al, be);
            v = __float_as_uint(off == L.off_ab ? al : be);
        } else if (off == L.off_ab + 8) {
            // yc: rho kappa_n summed over the (rare) read rows of slots the token writes, in row order
            const int u = tl + PD - 1;
            float yc = 0.f;
            for (int wd = 0; wd < MW; ++wd) {
                for (unsigned int b = omask[tl * MW + wd]; b; b &= b - 1) {
                    const int m = 32 * wd + __ffs((int)b) - 1;
                    const int n = find_slot(wl + u * W, W, wsrt[u] != 0, rl[tl * R + m]);
                    yc += r_val[tok * R + m] * w_val[tok * W + n];
                }
            }
            v = __float_as_uint(yc);
        }
        out[i] = v;
    }
    if (bad) atomicOr(err, 1u);
}

__host__ __device__ constexpr int round4(int x) { return (x + 3) & ~3; }

// ---------------------------------------------------------------- backward
// The backward visits t = T-1 .. 0.  For token t:
//  lm[m]  (M_t[j_m]): the earliest later writer t+d, 1 <= d < PD, whose undo
//         restored the row; entry n = its write position.
//  lgr[m] (G[j_m]) and lgw[n] (G[i_n]): the earliest later token t+d that
//         changed the adjoint row, either by its write adjoint (entry R + n,
//         which wins within one token: it runs after the read adjoint) or by
//         its read adjoint (entry m).  For lgw, d = 0 with a read entry means
//         this token's own read adjoint, which runs first.
template <int PD, bool VEC>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const int32_t* __restrict__ w_idx,
                                                       const float* __restrict__ w_val,
                                                       const int32_t* __restrict__ r_idx,
                                                       const float* __restrict__ r_val,
                                                       const void* __restrict__ alpha,
                                                       const void* __restrict__ beta, int in_dtype,
                                                       int T, int tb, int te, int W, int R, int64_t N,
                                                       unsigned char* __restrict__ recs,
                                                       unsigned int* __restrict__ err,
                                                       const float* __restrict__ gA,
                                                       const float* __restrict__ gbdt, int H) {
    // records of tokens [tb, te); links only to tokens below te (the backward
    // of later tokens, in an earlier call, left its rows in HBM)
    extern __shared__ __align__(16) int sm[];
    const BwdRec L = bwd_rec_layout(W, R);
    const int stream = blockIdx.y;
    const int t0 = tb + blockIdx.x * PT;
    const int ntok = min(PT, te - t0);
    const int span = min(PT + PD - 1, te - t0);   // tokens t0 .. t0+span-1 (later ones included)
    const int nlink = 2 * R + W;
    int* wl = sm;                                          // [PT+PD-1][W]
    int* rl = wl + (PT + PD - 1) * W;                      // [PT+PD-1][R]
    int* wsrt = rl + (PT + PD - 1) * R;                    // [PT+PD-1]
    int* rsrt = wsrt + round4(PT + PD - 1);                // [PT+PD-1]
    short* lk = reinterpret_cast<short*>(rsrt + round4(PT + PD - 1));   // [PT][2R + W]: lm, lgr, lgw (16-B aligned)
    const size_t sbase = (size_t)stream * T;
    unsigned int bad = 0u;

    for (int i = threadIdx.x; i < span * W; i += blockDim.x)
        wl[i] = clamp_slot(w_idx[(sbase + t0) * W + i], N, bad);
    for (int i = threadIdx.x; i < span * R; i += blockDim.x)
        rl[i] = clamp_slot(r_idx[(sbase + t0) * R + i], N, bad);
    __syncthreads();
    mark_sorted(wl, span, W, wsrt);
    mark_sorted(rl, span, R, rsrt);
    __syncthreads();

    const int nrow = W + R;
    for (int i = threadIdx.x; i < ntok * nrow; i += blockDim.x) {
        const int tl = i / nrow, r = i % nrow;
        const bool wrow = r < W;
        const int slot = wrow ? wl[tl * W + r] : rl[tl * R + (r - W)];
        short lg = -1, lm = -1;
        for (int d = min(PD - 1, span - 1 - tl); d >= 1; --d) {   // farthest first, nearest wins
            const int u = tl + d;
            const int n = find_slot(wl + u * W, W, wsrt[u] != 0, slot);
            const int m = find_slot(rl + u * R, R, rsrt[u] != 0, slot);
            if (n >= 0) {
                lg = (short)((d << 8) | (R + n));
                lm = (short)((d << 8) | n);
            } else if (m >= 0) {
                lg = (short)((d << 8) | m);
            }
        }
        if (wrow) {
            const int m = find_slot(rl + tl * R, R, rsrt[tl] != 0, slot);   // this token's read adjoint
            if (m >= 0) lg = (short)m;
            lk[tl * nlink + 2 * R + r] = lg;
        } else {
            lk[tl * nlink + (r - W)] = lm;
            lk[tl * nlink + R + (r - W)] = lg;
        }
    }
    __syncthreads();

    if (VEC) {
        // records in 16-byte pieces (W, R multiples of 8: every field 16-byte aligned)
        const int cw = W / 4, cr = R / 4, cl = nlink / 8;
        const int cpr = L.bytes / 16;           // 2 cw + 2 cr + cl + 1
        const float inv = 1.f / (float)cpr;
        int4* out = reinterpret_cast<int4*>(recs + (sbase + t0) * L.bytes);
        for (int i = threadIdx.x; i < ntok * cpr; i += blockDim.x) {
            int tl = (int)(((float)i + 0.5f) * inv);   // i / cpr (exact: i < 2^16)
            const int c = i - tl * cpr;
            const size_t tok = sbase + t0 + tl;
            int4 v;
            if (c < cw) {
                v = *reinterpret_cast<const int4*>(wl + tl * W + 4 * c);
            } else if (c < 2 * cw) {
                v = *reinterpret_cast<const int4*>(w_val + tok * W + 4 * (c - cw));
            } else if (c < 2 * cw + cr) {
                v = *reinterpret_cast<const int4*>(rl + tl * R + 4 * (c - 2 * cw));
            } else if (c < 2 * cw + 2 * cr) {
                v = *reinterpret_cast<const int4*>(r_val + tok * R + 4 * (c - 2 * cw - cr));
            } else if (c < 2 * cw + 2 * cr + cl) {
                v = *reinterpret_cast<const int4*>(lk + tl * nlink + 8 * (c - 2 * cw - 2 * cr));
            } else {
                float al, be;
                load_gates(alpha, beta, in_dtype, tok, al, be);
                sdm_gates_of(gA, gbdt, stream % H, al, be);
                v = make_int4((int)__float_as_uint(al), (int)__float_as_uint(be), 0, 0);
            }
            out[i] = v;
        }
        if (bad) atomicOr(err, 1u);
        return;
    }
    const int words = L.bytes / 4;
    uint32_t* out = reinterpret_cast<uint32_t*>(recs + (sbase + t0) * L.bytes);
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
            const uint32_t l0 = (uint16_t)lk[tl * nlink + e];
            const uint32_t l1 = e + 1 < nlink ? (uint16_t)lk[tl * nlink + e + 1] : 0xffffu;
            v = l0 | (l1 << 16);
        } else if (off == L.off_ab || off == L.off_ab + 4) {
            float al, be;
            load_gates(alpha, beta, in_dtype, tok, al, be);
            sdm_gates_of(gA, gbdt, stream % H, al, be);
            v = __float_as_uint(off == L.off_ab ? al : be);
        }
        out[i] = v;
    }
    if (bad) atomicOr(err, 1u);
}

template <int PD>
size_t fwd_prep_lds(int W, int R) {
    return sizeof(int) * ((size_t)(PT + PD - 1) * (W + 1) + (size_t)PT * R + (size_t)PT * ((R + 31) / 32)) +
           sizeof(short) * (size_t)PT * (W + R);
}
template <int PD>
size_t bwd_prep_lds(int W, int R) {
    return sizeof(int) * ((size_t)(PT + PD - 1) * (W + R) + 2 * round4(PT + PD - 1)) +
           sizeof(short) * (size_t)PT * (2 * R + W);
}

}  // namespace

template <int PD>
hipError_t sdm_launch_fwd_prep(const ScanFwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H;
    dim3 grid((a.te - a.tb + PT - 1) / PT, S);
    const size_t sm = fwd_prep_lds<PD>(a.W, a.R);
    auto kfn = fwd_prep_kernel<PD>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, grid, dim3(256), sm, st, a.w_idx, a.w_val, a.r_idx, a.r_val, a.alpha,
                       a.beta, a.in_dtype, a.T, a.tb, a.te, a.W, a.R, a.N, a.ws + SDM_WS_HEADER,
                       reinterpret_cast<unsigned int*>(a.ws), a.gate_A, a.gate_bdt, a.H);
    return hipGetLastError();
}

template <int PD>
hipError_t sdm_launch_bwd_prep(const ScanBwdArgs& a, hipStream_t st) {
    const int S = a.B * a.H;
    dim3 grid((a.te - a.tb + PT - 1) / PT, S);
    const size_t sm = bwd_prep_lds<PD>(a.W, a.R);
    // 16-byte record pieces: every field 16-byte aligned, and the weights readable as 16 bytes
    const bool vec = a.W % 8 == 0 && a.R % 8 == 0 && (reinterpret_cast<uintptr_t>(a.w_val) & 15) == 0 &&
                     (reinterpret_cast<uintptr_t>(a.r_val) & 15) == 0;
    auto kfn = vec ? bwd_prep_kernel<PD, true> : bwd_prep_kernel<PD, false>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, grid, dim3(256), sm, st, a.w_idx, a.w_val, a.r_idx, a.r_val, a.alpha,
                       a.beta, a.in_dtype, a.T, a.tb, a.te, a.W, a.R, a.N, a.ws + SDM_WS_HEADER,
                       reinterpret_cast<unsigned int*>(a.ws), a.gate_A, a.gate_bdt, a.H);
    return hipGetLastError();
}

// ---------------------------------------------------------------- debug id check
// One thread per (token, side): flags bit 0 if a slot id lies outside [0, N),
// bit 1 if an id repeats within the token's list (the backward's replace step
// G[i_n] = alpha Dbar_n needs distinct write ids).  Debug builds of a call
// only: O(K^2) compares per list.
namespace {
__global__ __launch_bounds__(256) void check_ids_kernel(const int32_t* __restrict__ w_idx, int W,
                                                        const int32_t* __restrict__ r_idx, int R,
                                                        int64_t ntok, int64_t N, unsigned int* __restrict__ flag) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= 2 * ntok) return;
    const bool wside = i < ntok;
    const int K = wside ? W : R;
    const int32_t* lst = wside ? w_idx + i * W : r_idx + (i - ntok) * R;
    unsigned int bad = 0u;
    for (int a = 0; a < K; ++a) {
        const int32_t s = lst[a];
        if (s < 0 || s >= N) bad |= 1u;
        for (int b = a + 1; b < K; ++b)
            if (lst[b] == s) bad |= 2u;
    }
    if (bad) atomicOr(flag, bad);
}
}  // namespace

hipError_t sdm_launch_check_ids(const int32_t* w_idx, int W, const int32_t* r_idx, int R, int64_t ntok,
                                int64_t N, unsigned int* flag, hipStream_t st) {
    const int64_t n = 2 * ntok;
    const unsigned int blocks = (unsigned int)((n + 255) / 256);
    hipLaunchKernelGGL(check_ids_kernel, dim3(blocks), dim3(256), 0, st, w_idx, W, r_idx, R, ntok, N, flag);
    return hipGetLastError();
}

template hipError_t sdm_launch_fwd_prep<SDM_FWD_PD>(const ScanFwdArgs&, hipStream_t);
template hipError_t sdm_launch_fwd_prep<8>(const ScanFwdArgs&, hipStream_t);
template hipError_t sdm_launch_fwd_prep<16>(const ScanFwdArgs&, hipStream_t);
template hipError_t sdm_launch_bwd_prep<SDM_BWD_PD>(const ScanBwdArgs&, hipStream_t);
template hipError_t sdm_launch_bwd_prep<2>(const ScanBwdArgs&, hipStream_t);
template hipError_t sdm_launch_bwd_prep<8>(const ScanBwdArgs&, hipStream_t);
