// The steps either side of the sparse recurrence, for gfx950:
//   gates     Sec. 3.1 step 2: alpha = exp(-A softplus(a + b_dt)), beta = sigma(b)
//             from the pre-activations a = W_a x, b = W_b x (per head, per token),
//             and their reverse mode;
//   epilogue  Sec. 3.1 step 4 / Fig. 2: o = y rstd gamma phi(g) per (b, h, t) row
//             of d_v values, rstd = 1 / sqrt(mean(y^2) + eps), phi = identity or
//             SiLU, and its reverse mode.
// All of it is elementwise or a reduction over one row (HBM-bound); the sums
// over many rows (dA, db_dt, dgamma) are taken in a fixed order so that results
// do not depend on scheduling.
#include <algorithm>

#include "sdm_common.h"
#include "sdm_internal.h"

namespace {

template <typename VT>
__device__ __forceinline__ float ld1(const VT* p, size_t i) {
    return to_f32(p[i]);
}

// ---------------------------------------------------------------- gates
template <typename VT>
__global__ __launch_bounds__(256) void gates_kernel(const VT* __restrict__ a, const VT* __restrict__ b,
                                                    const float* __restrict__ A, const float* __restrict__ bdt,
                                                    int H, int T, int64_t n, float* __restrict__ alpha,
                                                    float* __restrict__ beta) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    float al = ld1(a, i), be = ld1(b, i);
    sdm_gates_of(A, bdt, (int)((i / T) % H), al, be);
    alpha[i] = al;
    beta[i] = be;
}

// One workgroup per head: every (b, t) of the head, in a fixed order per
// thread, then a fixed tree over the threads.  dz = dalpha * (-A alpha
// sigma(z)), da = dz, db = dbeta beta (1 - beta); dA and db_dt are the head's
// sums of dalpha * (-softplus(z) alpha) and of dz.
constexpr int GB_THREADS = 256;
template <typename VT>
__global__ __launch_bounds__(GB_THREADS) void gates_bwd_kernel(
    const VT* __restrict__ a, const VT* __restrict__ b, const float* __restrict__ A,
    const float* __restrict__ bdt, const float* __restrict__ dalpha, const float* __restrict__ dbeta, int B,
    int H, int T, float* __restrict__ da, float* __restrict__ db, float* __restrict__ dA,
    float* __restrict__ db_dt) {
    __shared__ float red[2][GB_THREADS];
    const int h = blockIdx.x;
    const float Ah = A[h], bh = bdt[h];
    float sA = 0.f, sb = 0.f;
    const int64_t per_head = (int64_t)B * T;
    for (int64_t j = threadIdx.x; j < per_head; j += GB_THREADS) {
        const int bb = (int)(j / T), t = (int)(j % T);
        const size_t i = ((size_t)bb * H + h) * T + t;
        const float z = ld1(a, i) + bh;
        const float sp = sdm_softplus(z);
        const float al = expf(-Ah * sp);
        const float dal = dalpha[i];
        const float dz = dal * (-Ah * al * sdm_sigmoid(z));
        da[i] = dz;
        sb += dz;
        sA += dal * (-sp * al);
        const float be = sdm_sigmoid(ld1(b, i));
        db[i] = dbeta[i] * be * (1.f - be);
    }
    red[0][threadIdx.x] = sA;
    red[1][threadIdx.x] = sb;
    __syncthreads();
    for (int m = GB_THREADS / 2; m > 0; m >>= 1) {
        if (threadIdx.x < m) {
            red[0][threadIdx.x] += red[0][threadIdx.x + m];
            red[1][threadIdx.x] += red[1][threadIdx.x + m];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        dA[h] = red[0][0];
        db_dt[h] = red[1][0];
    }
}

// ---------------------------------------------------------------- epilogue
// LPR lanes per row (4 columns per lane per step), 64 / LPR rows per wave,
// four waves per workgroup.
__device__ __forceinline__ float act_f(float g, int act) { return act ? g * sdm_sigmoid(g) : g; }
__device__ __forceinline__ float act_grad(float g, int act) {
    if (!act) return 1.f;
    const float sg = sdm_sigmoid(g);
    return sg * (1.f + g * (1.f - sg));
}

template <int LPR>
__device__ __forceinline__ float row_sum(float v) {
#pragma unroll
    for (int m = LPR / 2; m >= 1; m >>= 1) v += xor_lane_f(v, m);
    return v;
}

// 1 / sqrt(mean(y^2) + eps) of one row; every lane of the row's group gets it
template <int LPR>
__device__ __forceinline__ float row_rstd(const float* yr, int dv, int q, float eps) {
    float ss = 0.f;
    for (int c = q * 4; c < dv; c += 4 * LPR) {
        const v4f v = ld4(yr + c);
        ss = fmaf(v.x, v.x, ss);
        ss = fmaf(v.y, v.y, ss);
        ss = fmaf(v.z, v.z, ss);
        ss = fmaf(v.w, v.w, ss);
    }
    ss = row_sum<LPR>(ss);
    return 1.f / sqrtf(ss / (float)dv + eps);
}

// Rows are the tokens [tb, tb + tn) of every stream of T tokens: row r of
// [0, S tn) is stream r / tn, token tb + r % tn.
template <typename GT, int LPR>
__global__ __launch_bounds__(256) void norm_gate_kernel(const float* __restrict__ y, const GT* __restrict__ g,
                                                        const float* __restrict__ gamma, float eps, int act,
                                                        int64_t rows, int T, int tb, int tn, int dv,
                                                        float* __restrict__ o, float* __restrict__ rstd) {
    constexpr int RPW = 64 / LPR;
    const int lane = threadIdx.x & 63, q = lane % LPR;
    const int64_t vrow = ((int64_t)blockIdx.x * 4 + threadIdx.x / 64) * RPW + lane / LPR;
    const bool ok = vrow < rows;
    const int64_t vr = ok ? vrow : rows - 1;   // every lane takes part in the row sums
    const int64_t row = (vr / tn) * T + tb + vr % tn;
    const int64_t rr = row;
    const float* yr = y + rr * dv;
    const float rs = row_rstd<LPR>(yr, dv, q, eps);
    if (!ok) return;
    if (rstd && q == 0) rstd[row] = rs;
    for (int c = q * 4; c < dv; c += 4 * LPR) {
        const v4f v = ld4(yr + c);
        const v4f gg = ld4v(g + rr * dv + c);
        const v4f gm = gamma ? ld4(gamma + c) : v4f{1.f, 1.f, 1.f, 1.f};
        v4f out;
        out.x = v.x * rs * gm.x * act_f(gg.x, act);
        out.y = v.y * rs * gm.y * act_f(gg.y, act);
        out.z = v.z * rs * gm.z * act_f(gg.z, act);
        out.w = v.w * rs * gm.w * act_f(gg.w, act);
        st4(o + rr * dv + c, out);
    }
}

// Reverse mode.  n = y rstd:  dg = do gamma n phi'(g);  dn = do phi(g) gamma;
// dy = rstd (dn - n mean(dn n)).  dgamma: each workgroup sums do phi(g) n over
// its rows in a fixed order (per lane across the rows its row group visits,
// then over row groups and waves through LDS) into part[workgroup][d_v].
template <typename GT, int LPR, int NQ>
__global__ __launch_bounds__(256) void norm_gate_bwd_kernel(
    const float* __restrict__ y, const GT* __restrict__ g, const float* __restrict__ gamma, float eps, int act,
    const float* __restrict__ dout, int64_t rows, int dv, int iters, float* __restrict__ dy,
    float* __restrict__ dg, float* __restrict__ part) {
    constexpr int RPW = 64 / LPR;
    extern __shared__ float gsum[];   // [4 * RPW][dv]
    const int lane = threadIdx.x & 63, q = lane % LPR, wave = threadIdx.x / 64;
    const int grp = wave * RPW + lane / LPR;     // row group of this lane in the workgroup
    v4f acc[NQ];
#pragma unroll
    for (int j = 0; j < NQ; ++j) acc[j] = v4zero();
    for (int it = 0; it < iters; ++it) {
        const int64_t row = ((int64_t)blockIdx.x * iters + it) * (4 * RPW) + grp;
        const bool ok = row < rows;
        const int64_t rr = ok ? row : rows - 1;
        const float* yr = y + rr * dv;
        const float rs = row_rstd<LPR>(yr, dv, q, eps);
        // mean(dn n) over the row
        float dot = 0.f;
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            const int c = q * 4 + j * 4 * LPR;
            if (c < dv) {
                const v4f v = ld4(yr + c), d = ld4(dout + rr * dv + c);
                const v4f gg = ld4v(g + rr * dv + c);
                const v4f gm = gamma ? ld4(gamma + c) : v4f{1.f, 1.f, 1.f, 1.f};
                dot += d.x * act_f(gg.x, act) * gm.x * v.x + d.y * act_f(gg.y, act) * gm.y * v.y +
                       d.z * act_f(gg.z, act) * gm.z * v.z + d.w * act_f(gg.w, act) * gm.w * v.w;
            }
        }
        dot = row_sum<LPR>(dot) * rs / (float)dv;   // mean(dn n) = rstd mean(dn y)
        if (!ok) continue;
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            const int c = q * 4 + j * 4 * LPR;
            if (c < dv) {
                const v4f v = ld4(yr + c), d = ld4(dout + rr * dv + c);
                const v4f gg = ld4v(g + rr * dv + c);
                const v4f gm = gamma ? ld4(gamma + c) : v4f{1.f, 1.f, 1.f, 1.f};
                v4f n, ph, odg, ody;
                n.x = v.x * rs; n.y = v.y * rs; n.z = v.z * rs; n.w = v.w * rs;
                ph.x = act_f(gg.x, act); ph.y = act_f(gg.y, act); ph.z = act_f(gg.z, act); ph.w = act_f(gg.w, act);
                odg.x = d.x * gm.x * n.x * act_grad(gg.x, act);
                odg.y = d.y * gm.y * n.y * act_grad(gg.y, act);
                odg.z = d.z * gm.z * n.z * act_grad(gg.z, act);
                odg.w = d.w * gm.w * n.w * act_grad(gg.w, act);
                ody.x = rs * (d.x * ph.x * gm.x - n.x * dot);
                ody.y = rs * (d.y * ph.y * gm.y - n.y * dot);
                ody.z = rs * (d.z * ph.z * gm.z - n.z * dot);
                ody.w = rs * (d.w * ph.w * gm.w - n.w * dot);
                st4(dg + rr * dv + c, odg);
                st4(dy + rr * dv + c, ody);
                acc[j].x += d.x * ph.x * n.x;
                acc[j].y += d.y * ph.y * n.y;
                acc[j].z += d.z * ph.z * n.z;
                acc[j].w += d.w * ph.w * n.w;
            }
        }
    }
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        const int c = q * 4 + j * 4 * LPR;
        if (c < dv) st4(gsum + (size_t)grp * dv + c, acc[j]);
    }
    __syncthreads();
    for (int c = threadIdx.x; c < dv; c += blockDim.x) {
        float sum = 0.f;
        for (int r = 0; r < 4 * RPW; ++r) sum += gsum[(size_t)r * dv + c];
        part[(size_t)blockIdx.x * dv + c] = sum;
    }
}

// out[c] = sum over blocks of part[block][c], blocks in order
__global__ __launch_bounds__(256) void colsum_kernel(const float* __restrict__ part, int nblk, int dv,
                                                     float* __restrict__ out) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= dv) return;
    float sum = 0.f;
    for (int b = 0; b < nblk; ++b) sum += part[(size_t)b * dv + c];
    out[c] = sum;
}

int lanes_per_row(int dv) {
    const int quads = dv / 4;
    return quads <= 8 ? 8 : quads <= 16 ? 16 : quads <= 32 ? 32 : 64;
}

template <typename GT, int LPR>
hipError_t launch_norm_gate_l(const float* y, const void* g, const float* gamma, float eps, int act, int64_t S,
                              int T, int tb, int tn, int dv, float* o, float* rstd, hipStream_t st) {
    constexpr int RPB = 4 * (64 / LPR);
    const int64_t rows = S * tn;
    const unsigned blocks = (unsigned)((rows + RPB - 1) / RPB);
    hipLaunchKernelGGL((norm_gate_kernel<GT, LPR>), dim3(blocks), dim3(256), 0, st, y, static_cast<const GT*>(g),
                       gamma, eps, act, rows, T, tb, tn, dv, o, rstd);
    return hipGetLastError();
}

template <typename GT>
hipError_t launch_norm_gate_t(const float* y, const void* g, const float* gamma, float eps, int act, int64_t S,
                              int T, int tb, int tn, int dv, float* o, float* rstd, hipStream_t st) {
    switch (lanes_per_row(dv)) {
        case 8: return launch_norm_gate_l<GT, 8>(y, g, gamma, eps, act, S, T, tb, tn, dv, o, rstd, st);
        case 16: return launch_norm_gate_l<GT, 16>(y, g, gamma, eps, act, S, T, tb, tn, dv, o, rstd, st);
        case 32: return launch_norm_gate_l<GT, 32>(y, g, gamma, eps, act, S, T, tb, tn, dv, o, rstd, st);
        default: return launch_norm_gate_l<GT, 64>(y, g, gamma, eps, act, S, T, tb, tn, dv, o, rstd, st);
    }
}

// Rows per workgroup of the backward: iters steps of 4 * RPW rows, sized so
// that about 2048 workgroups cover the rows (the dgamma partials then hold
// 2048 x d_v floats).
constexpr int64_t NG_BWD_TARGET_BLOCKS = 2048;

template <int LPR>
void ng_bwd_geometry(int64_t rows, int* iters, int64_t* nblk) {
    constexpr int RPB = 4 * (64 / LPR);
    const int64_t steps = (rows + RPB - 1) / RPB;
    const int64_t it = std::max<int64_t>(1, (steps + NG_BWD_TARGET_BLOCKS - 1) / NG_BWD_TARGET_BLOCKS);
    *iters = (int)it;
    *nblk = (steps + it - 1) / it;
}

template <typename GT, int LPR, int NQ>
hipError_t launch_ng_bwd_q(const float* y, const void* g, const float* gamma, float eps, int act,
                           const float* dout, int64_t rows, int dv, float* dy, float* dg, float* part,
                           hipStream_t st, int iters, int64_t nblk) {
    constexpr int RPW = 64 / LPR;
    const size_t lds = (size_t)4 * RPW * dv * sizeof(float);
    auto kfn = norm_gate_bwd_kernel<GT, LPR, NQ>;
    hipError_t e = hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kfn, dim3((unsigned)nblk), dim3(256), lds, st, y, static_cast<const GT*>(g), gamma, eps, act,
                       dout, rows, dv, iters, dy, dg, part);
    return hipGetLastError();
}

template <typename GT, int LPR>
hipError_t launch_ng_bwd_l(const float* y, const void* g, const float* gamma, float eps, int act, const float* dout,
                           int64_t rows, int dv, float* dy, float* dg, float* part, hipStream_t st) {
    int iters;
    int64_t nblk;
    ng_bwd_geometry<LPR>(rows, &iters, &nblk);
    const int nq = (dv / 4 + LPR - 1) / LPR;
    if (nq <= 1) return launch_ng_bwd_q<GT, LPR, 1>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st, iters, nblk);
    if (nq <= 2) return launch_ng_bwd_q<GT, LPR, 2>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st, iters, nblk);
    if (nq <= 4) return launch_ng_bwd_q<GT, LPR, 4>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st, iters, nblk);
    if (nq <= 8) return launch_ng_bwd_q<GT, LPR, 8>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st, iters, nblk);
    return launch_ng_bwd_q<GT, LPR, 16>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st, iters, nblk);
}

template <typename GT>
hipError_t launch_ng_bwd_t(const float* y, const void* g, const float* gamma, float eps, int act, const float* dout,
                           int64_t rows, int dv, float* dy, float* dg, float* part, hipStream_t st) {
    switch (lanes_per_row(dv)) {
        case 8: return launch_ng_bwd_l<GT, 8>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st);
        case 16: return launch_ng_bwd_l<GT, 16>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st);
        case 32: return launch_ng_bwd_l<GT, 32>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st);
        default: return launch_ng_bwd_l<GT, 64>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st);
    }
}

}  // namespace

hipError_t sdm_launch_gates(const void* a, const void* b, int dtype, const float* A, const float* bdt, int B, int H,
                            int T, float* alpha, float* beta, hipStream_t st) {
    const int64_t n = (int64_t)B * H * T;
    if (n == 0) return hipSuccess;
    const unsigned blocks = (unsigned)((n + 255) / 256);
    if (dtype == SDM_DT_BF16)
        hipLaunchKernelGGL(gates_kernel<bf16_t>, dim3(blocks), dim3(256), 0, st, static_cast<const bf16_t*>(a),
                           static_cast<const bf16_t*>(b), A, bdt, H, T, n, alpha, beta);
    else
        hipLaunchKernelGGL(gates_kernel<float>, dim3(blocks), dim3(256), 0, st, static_cast<const float*>(a),
                           static_cast<const float*>(b), A, bdt, H, T, n, alpha, beta);
    return hipGetLastError();
}

hipError_t sdm_launch_gates_bwd(const void* a, const void* b, int dtype, const float* A, const float* bdt,
                                const float* dalpha, const float* dbeta, int B, int H, int T, float* da, float* db,
                                float* dA, float* db_dt, hipStream_t st) {
    if (H == 0) return hipSuccess;
    if (dtype == SDM_DT_BF16)
        hipLaunchKernelGGL(gates_bwd_kernel<bf16_t>, dim3(H), dim3(GB_THREADS), 0, st, static_cast<const bf16_t*>(a),
                           static_cast<const bf16_t*>(b), A, bdt, dalpha, dbeta, B, H, T, da, db, dA, db_dt);
    else
        hipLaunchKernelGGL(gates_bwd_kernel<float>, dim3(H), dim3(GB_THREADS), 0, st, static_cast<const float*>(a),
                           static_cast<const float*>(b), A, bdt, dalpha, dbeta, B, H, T, da, db, dA, db_dt);
    return hipGetLastError();
}

hipError_t sdm_launch_norm_gate(const float* y, const void* g, int g_dtype, const float* gamma, float eps, int act,
                                int64_t S, int T, int tb, int tn, int dv, float* o, float* rstd, hipStream_t st) {
    if (S * tn == 0) return hipSuccess;
    return g_dtype == SDM_DT_BF16
               ? launch_norm_gate_t<bf16_t>(y, g, gamma, eps, act, S, T, tb, tn, dv, o, rstd, st)
               : launch_norm_gate_t<float>(y, g, gamma, eps, act, S, T, tb, tn, dv, o, rstd, st);
}

size_t sdm_norm_gate_bwd_ws(int64_t rows, int dv) {
    int iters;
    int64_t nblk = 0;
    switch (lanes_per_row(dv)) {
        case 8: ng_bwd_geometry<8>(rows, &iters, &nblk); break;
        case 16: ng_bwd_geometry<16>(rows, &iters, &nblk); break;
        case 32: ng_bwd_geometry<32>(rows, &iters, &nblk); break;
        default: ng_bwd_geometry<64>(rows, &iters, &nblk); break;
    }
    return (size_t)std::max<int64_t>(nblk, 1) * dv * sizeof(float);
}

hipError_t sdm_launch_norm_gate_bwd(const float* y, const void* g, int g_dtype, const float* gamma, float eps,
                                    int act, const float* dout, int64_t rows, int dv, float* dy, float* dg,
                                    float* dgamma, float* part, hipStream_t st) {
    if (rows == 0) {   // dgamma = 0: a column sum over no blocks (a kernel, not a memset)
        if (!dgamma) return hipSuccess;
        hipLaunchKernelGGL(colsum_kernel, dim3((dv + 255) / 256), dim3(256), 0, st, part, 0, dv, dgamma);
        return hipGetLastError();
    }
    hipError_t e = g_dtype == SDM_DT_BF16
                       ? launch_ng_bwd_t<bf16_t>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st)
                       : launch_ng_bwd_t<float>(y, g, gamma, eps, act, dout, rows, dv, dy, dg, part, st);
    if (e != hipSuccess || !dgamma) return e;
    const int64_t nblk = (int64_t)(sdm_norm_gate_bwd_ws(rows, dv) / (dv * sizeof(float)));
    hipLaunchKernelGGL(colsum_kernel, dim3((dv + 255) / 256), dim3(256), 0, st, part, (int)nblk, dv, dgamma);
    return hipGetLastError();
}
