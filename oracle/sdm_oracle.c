/*
 * CPU oracle for the Sparse Delta Memory (SDM) recurrence.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The HIP library never
 * links, includes or calls it, and it shares no code with it.
 *
 * Plain C, fp64 state and arithmetic, one (b, h) stream at a time, every step
 * in the order the paper states it.  No blocking, no fusion, no reordering.
 *
 *   Addressing   Sec. 2 "Product Key Memory" (outer sum of two score vectors,
 *                top-k of top-k identity), Sec. 3.1 step 1 (top-W / top-R of
 *                the outer-sum scores), Sec. 4 "SDM Configuration" (read and
 *                write activations are softmax-normalised), App. A.2 (the
 *                selected indices are sorted by slot index).
 *   Forward      Sec. 3.1 step 2, Eq. (sdm-decay) and Eq. (sdm-write) in the
 *                read-back form of Fig. 2 (v~ = M~^T k, dv = v - v~), step 3
 *                Eq. (sdm-read) on the post-write memory M_t.
 *   Backward     reverse mode of the forward; past memory states are
 *                recovered by undoing the in-place writes (App. A.3).
 *   Gates        Sec. 3.1 step 2: the forget gate from A, b_dt and its
 *                projection, the input gate from its projection; reverse mode.
 *   Epilogue     Sec. 3.1 step 4 and Fig. 2: RMS norm of each head's read
 *                vector times the element-wise output gate; reverse mode.
 *
 * Readings where the paper is silent (listed with their reasons in the
 * design notes): codebook scoring when d_k != 2 sqrt(N); ties ordered by
 * slot id ascending; the flat slot id of pair (a, b) is a*sqrt(N) + b; the
 * top-k decision can be taken on fp32-rounded scores (the precision the GPU
 * kernel decides in) or on exact fp64 scores.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------ selection */
typedef struct {
    double score;
    int64_t id;
} cand_t;

/* total order: score descending, then id ascending */
static int cmp_desc(const void* pa, const void* pb) {
    const cand_t* a = (const cand_t*)pa;
    const cand_t* b = (const cand_t*)pb;
    if (a->score > b->score) return -1;
    if (a->score < b->score) return 1;
    if (a->id < b->id) return -1;
    if (a->id > b->id) return 1;
    return 0;
}

static int cmp_id(const void* pa, const void* pb) {
    const cand_t* a = (const cand_t*)pa;
    const cand_t* b = (const cand_t*)pb;
    return (a->id > b->id) - (a->id < b->id);
}

/* the two sub-score vectors of one token (Sec. 3.1 step 1: the projected
 * vector is split into halves).  With a codebook, half h scores sub-key j as
 * <x[h*dk/2 : (h+1)*dk/2], C[h][j]>, summed over c in increasing order.
 * Without one (dk == 2 s), the halves of x are the scores themselves. */
static void sub_scores(const double* x, const double* cb_head, int dk, int s,
                       int round_f32, double* s0, double* s1) {
    for (int h = 0; h < 2; ++h) {
        double* out = h ? s1 : s0;
        for (int j = 0; j < s; ++j) {
            double acc;
            if (cb_head) {
                int dh = dk / 2;
                const double* c = cb_head + ((size_t)h * s + j) * dh;
                acc = 0.0;
                for (int i = 0; i < dh; ++i) acc += x[h * dh + i] * c[i];
            } else {
                acc = x[h * s + j];
            }
            out[j] = round_f32 ? (double)(float)acc : acc;
        }
    }
}

/* score of slot (a, b): s0[a] + s1[b].  In fp32-decision mode the sum is
 * the fp32 sum of the two fp32 sub-scores. */
static double pair_score(double a, double b, int f32) {
    if (f32) {
        float fa = (float)a, fb = (float)b;
        float r = fa + fb;
        return (double)r;
    }
    return a + b;
}

/* sort the k selected slots by id and softmax their scores (max-subtracted) */
static void finish(cand_t* sel, int k, int32_t* idx, double* val, double* score) {
    qsort(sel, (size_t)k, sizeof(cand_t), cmp_id);
    double mx = sel[0].score;
    for (int n = 1; n < k; ++n)
        if (sel[n].score > mx) mx = sel[n].score;
    double z = 0.0;
    for (int n = 0; n < k; ++n) z += exp(sel[n].score - mx);
    for (int n = 0; n < k; ++n) {
        idx[n] = (int32_t)sel[n].id;
        val[n] = exp(sel[n].score - mx) / z;
        if (score) score[n] = sel[n].score;
    }
}

/*
 * Addressing by the top-k-of-top-k identity of Sec. 2:
 * top_k(s0 (+) s1) = top_k(top_k(s0) (+) top_k(s1)).
 *
 * x       [B][H][T][dk]
 * cb      [H][2][s][dk/2] or NULL (direct mode, dk == 2 s)
 * idx     [B][H][T][k]   selected slot ids, ascending
 * val     [B][H][T][k]   softmax weights in the same order
 * score   [B][H][T][k]   raw scores of the selected slots (may be NULL)
 */
int orc_address(const double* x, const double* cb, int B, int H, int T, int dk, int64_t N,
                int k, int decide_f32, int32_t* idx, double* val, double* score) {
    int s = (int)llround(sqrt((double)N));
    if ((int64_t)s * s != N || k < 1 || k > s) return -1;
    if (!cb && dk != 2 * s) return -1;
    if (cb && (dk % 2)) return -1;
    int64_t ntok = (int64_t)B * H * T;
#pragma omp parallel
    {
        double* s0 = (double*)malloc(sizeof(double) * s);
        double* s1 = (double*)malloc(sizeof(double) * s);
        cand_t* c0 = (cand_t*)malloc(sizeof(cand_t) * s);
        cand_t* c1 = (cand_t*)malloc(sizeof(cand_t) * s);
        cand_t* pr = (cand_t*)malloc(sizeof(cand_t) * (size_t)k * k);
#pragma omp for schedule(dynamic, 64)
        for (int64_t r = 0; r < ntok; ++r) {
            int h = (int)((r / T) % H);
            const double* cbh = cb ? cb + (size_t)h * 2 * s * (dk / 2) : NULL;
            sub_scores(x + r * dk, cbh, dk, s, decide_f32, s0, s1);
            /* stage 1: top-k of each half */
            for (int j = 0; j < s; ++j) {
                c0[j].score = s0[j]; c0[j].id = j;
                c1[j].score = s1[j]; c1[j].id = j;
            }
            qsort(c0, (size_t)s, sizeof(cand_t), cmp_desc);
            qsort(c1, (size_t)s, sizeof(cand_t), cmp_desc);
            /* stage 2: the k*k outer sums of the two shortlists */
            for (int i = 0; i < k; ++i)
                for (int j = 0; j < k; ++j) {
                    cand_t* p = &pr[i * k + j];
                    p->score = pair_score(c0[i].score, c1[j].score, decide_f32);
                    p->id = c0[i].id * (int64_t)s + c1[j].id;
                }
            qsort(pr, (size_t)k * k, sizeof(cand_t), cmp_desc);
            finish(pr, k, idx + r * k, val + r * k, score ? score + r * k : NULL);
        }
        free(s0); free(s1); free(c0); free(c1); free(pr);
    }
    return 0;
}

/* Addressing by definition: all N outer-sum scores, full sort, first k. */
int orc_address_brute(const double* x, const double* cb, int B, int H, int T, int dk, int64_t N,
                      int k, int decide_f32, int32_t* idx, double* val, double* score) {
    int s = (int)llround(sqrt((double)N));
    if ((int64_t)s * s != N || k < 1 || k > N) return -1;
    if (!cb && dk != 2 * s) return -1;
    int64_t ntok = (int64_t)B * H * T;
#pragma omp parallel
    {
        double* s0 = (double*)malloc(sizeof(double) * s);
        double* s1 = (double*)malloc(sizeof(double) * s);
        cand_t* all = (cand_t*)malloc(sizeof(cand_t) * (size_t)N);
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < ntok; ++r) {
            int h = (int)((r / T) % H);
            const double* cbh = cb ? cb + (size_t)h * 2 * s * (dk / 2) : NULL;
            sub_scores(x + r * dk, cbh, dk, s, decide_f32, s0, s1);
            for (int a = 0; a < s; ++a)
                for (int b = 0; b < s; ++b) {
                    all[(size_t)a * s + b].score = pair_score(s0[a], s1[b], decide_f32);
                    all[(size_t)a * s + b].id = (int64_t)a * s + b;
                }
            qsort(all, (size_t)N, sizeof(cand_t), cmp_desc);
            finish(all, k, idx + r * k, val + r * k, score ? score + r * k : NULL);
        }
        free(s0); free(s1); free(all);
    }
    return 0;
}

/* ------------------------------------------------------------ forward */
/*
 * One step of Sec. 3.1 for one stream, on the memory table M [N][dv]:
 *   P_n  = M_{t-1}[i_n]                     (the W selected rows)
 *   Mt_n = alpha * P_n                      Eq. (sdm-decay), written rows only
 *   u    = sum_n kappa_n * Mt_n             read-back M~_t^T k_t (Fig. 2)
 *   e    = beta * (v - u)                   beta_t * Delta v_t
 *   M_t[i_n] = Mt_n + kappa_n * e           Eq. (sdm-write)
 *   y_t  = sum_m rho_m * M_t[j_m]           Eq. (sdm-read), post-write memory
 * Rows outside the write set are not touched.
 *
 * S streams, each with its own table; arrays are [S][T][...], mem [S][N][dv],
 * saved [S][T][W][dv] receives P (the undo log of App. A.3) when not NULL.
 */
int orc_scan_fwd(int S, int T, int dv, int64_t N, int W, int R,
                 const int32_t* widx, const double* wval, const int32_t* ridx, const double* rval,
                 const double* v, const double* alpha, const double* beta,
                 double* mem, double* y, double* saved) {
#pragma omp parallel
    {
        double* P = (double*)malloc(sizeof(double) * (size_t)W * dv);
        double* D = (double*)malloc(sizeof(double) * (size_t)W * dv);
        double* u = (double*)malloc(sizeof(double) * dv);
        double* e = (double*)malloc(sizeof(double) * dv);
#pragma omp for schedule(dynamic, 1)
        for (int sI = 0; sI < S; ++sI) {
            double* M = mem + (size_t)sI * N * dv;
            for (int t = 0; t < T; ++t) {
                size_t st = (size_t)sI * T + t;
                const int32_t* I = widx + st * W;
                const double* kap = wval + st * W;
                const int32_t* J = ridx + st * R;
                const double* rho = rval + st * R;
                double a = alpha[st], b = beta[st];
                for (int n = 0; n < W; ++n)
                    for (int c = 0; c < dv; ++c) P[(size_t)n * dv + c] = M[(size_t)I[n] * dv + c];
                for (int n = 0; n < W; ++n)
                    for (int c = 0; c < dv; ++c) D[(size_t)n * dv + c] = a * P[(size_t)n * dv + c];
                for (int c = 0; c < dv; ++c) {
                    double acc = 0.0;
                    for (int n = 0; n < W; ++n) acc += kap[n] * D[(size_t)n * dv + c];
                    u[c] = acc;
                }
                for (int c = 0; c < dv; ++c) e[c] = b * (v[st * dv + c] - u[c]);
                for (int n = 0; n < W; ++n)
                    for (int c = 0; c < dv; ++c)
                        M[(size_t)I[n] * dv + c] = D[(size_t)n * dv + c] + kap[n] * e[c];
                for (int c = 0; c < dv; ++c) {
                    double acc = 0.0;
                    for (int m = 0; m < R; ++m) acc += rho[m] * M[(size_t)J[m] * dv + c];
                    y[st * dv + c] = acc;
                }
                if (saved)
                    memcpy(saved + st * (size_t)W * dv, P, sizeof(double) * (size_t)W * dv);
            }
        }
        free(P); free(D); free(u); free(e);
    }
    return 0;
}

/* ------------------------------------------------------------ backward */
/*
 * Reverse mode of orc_scan_fwd.  Enter with mem = M_T, G = dL/dM_T; leave
 * with mem = M_0 (restored by undoing each step from the saved P rows, as in
 * App. A.3) and G = dL/dM_0.  Per step t, last first:
 *
 *   read    rbar_m = <ybar, M_t[j_m]>;  G[j_m] += rho_m * ybar
 *   write   g_n = G[i_n];  D_n = alpha P_n;  u = sum kappa_n D_n;  e = beta (v-u)
 *           ebar = sum_n kappa_n g_n
 *           vbar = beta ebar;  betabar = <ebar, v - u>
 *           kbar_n = <g_n, e> - beta <ebar, D_n>
 *           Dbar_n = g_n - beta kappa_n ebar;  alphabar = sum_n <Dbar_n, P_n>
 *           G[i_n] = alpha Dbar_n          (replaces: the slots are distinct)
 *   undo    M[i_n] = P_n
 */
int orc_scan_bwd(int S, int T, int dv, int64_t N, int W, int R,
                 const int32_t* widx, const double* wval, const int32_t* ridx, const double* rval,
                 const double* v, const double* alpha, const double* beta,
                 double* mem, const double* saved, const double* dy, double* G,
                 double* dv_out, double* dalpha, double* dbeta, double* dwval, double* drval) {
#pragma omp parallel
    {
        double* D = (double*)malloc(sizeof(double) * (size_t)W * dv);
        double* g = (double*)malloc(sizeof(double) * (size_t)W * dv);
        double* Db = (double*)malloc(sizeof(double) * (size_t)W * dv);
        double* u = (double*)malloc(sizeof(double) * dv);
        double* e = (double*)malloc(sizeof(double) * dv);
        double* eb = (double*)malloc(sizeof(double) * dv);
#pragma omp for schedule(dynamic, 1)
        for (int sI = 0; sI < S; ++sI) {
            double* M = mem + (size_t)sI * N * dv;
            double* Gs = G + (size_t)sI * N * dv;
            for (int t = T - 1; t >= 0; --t) {
                size_t st = (size_t)sI * T + t;
                const int32_t* I = widx + st * W;
                const double* kap = wval + st * W;
                const int32_t* J = ridx + st * R;
                const double* rho = rval + st * R;
                const double* P = saved + st * (size_t)W * dv;
                const double* yb = dy + st * dv;
                double a = alpha[st], b = beta[st];
                /* read */
                for (int m = 0; m < R; ++m) {
                    double acc = 0.0;
                    for (int c = 0; c < dv; ++c) acc += yb[c] * M[(size_t)J[m] * dv + c];
                    drval[st * R + m] = acc;
                }
                for (int m = 0; m < R; ++m)
                    for (int c = 0; c < dv; ++c) Gs[(size_t)J[m] * dv + c] += rho[m] * yb[c];
                /* write: recompute the step's intermediates from P */
                for (int n = 0; n < W; ++n)
                    for (int c = 0; c < dv; ++c) {
                        D[(size_t)n * dv + c] = a * P[(size_t)n * dv + c];
                        g[(size_t)n * dv + c] = Gs[(size_t)I[n] * dv + c];
                    }
                for (int c = 0; c < dv; ++c) {
                    double acc = 0.0;
                    for (int n = 0; n < W; ++n) acc += kap[n] * D[(size_t)n * dv + c];
                    u[c] = acc;
                    e[c] = b * (v[st * dv + c] - u[c]);
                    double ea = 0.0;
                    for (int n = 0; n < W; ++n) ea += kap[n] * g[(size_t)n * dv + c];
                    eb[c] = ea;
                }
                double bb = 0.0;
                for (int c = 0; c < dv; ++c) {
                    dv_out[st * dv + c] = b * eb[c];
                    bb += eb[c] * (v[st * dv + c] - u[c]);
                }
                dbeta[st] = bb;
                double ab = 0.0;
                for (int n = 0; n < W; ++n) {
                    double ge = 0.0, ed = 0.0;
                    for (int c = 0; c < dv; ++c) {
                        ge += g[(size_t)n * dv + c] * e[c];
                        ed += eb[c] * D[(size_t)n * dv + c];
                    }
                    dwval[st * W + n] = ge - b * ed;
                    for (int c = 0; c < dv; ++c) {
                        double db = g[(size_t)n * dv + c] - b * kap[n] * eb[c];
                        Db[(size_t)n * dv + c] = db;
                        ab += db * P[(size_t)n * dv + c];
                    }
                }
                dalpha[st] = ab;
                for (int n = 0; n < W; ++n)
                    for (int c = 0; c < dv; ++c) Gs[(size_t)I[n] * dv + c] = a * Db[(size_t)n * dv + c];
                /* undo */
                for (int n = 0; n < W; ++n)
                    for (int c = 0; c < dv; ++c) M[(size_t)I[n] * dv + c] = P[(size_t)n * dv + c];
            }
        }
        free(D); free(g); free(Db); free(u); free(e); free(eb);
    }
    return 0;
}

/*
 * Gradient of the addressing w.r.t. x, given dL/dval for the selected slots.
 * The selection itself is piecewise constant and passes no gradient.
 *   softmax   sbar_n = w_n (wbar_n - sum_m w_m wbar_m)
 *   outer sum slot id = a*s + b:  s0bar[a] += sbar_n, s1bar[b] += sbar_n
 *   scoring   xbar[h*dk/2 + c] = sum_j shbar[j] C[h][j][c]   (codebook mode)
 *             xbar[h*s + j]    = shbar[j]                     (direct mode)
 */
int orc_address_bwd(const double* cb, int B, int H, int T, int dk, int64_t N, int k,
                    const int32_t* idx, const double* val, const double* dval, double* dx) {
    int s = (int)llround(sqrt((double)N));
    if ((int64_t)s * s != N) return -1;
    int64_t ntok = (int64_t)B * H * T;
#pragma omp parallel
    {
        double* sb = (double*)malloc(sizeof(double) * 2 * s);
#pragma omp for schedule(static)
        for (int64_t r = 0; r < ntok; ++r) {
            int h = (int)((r / T) % H);
            const int32_t* I = idx + r * k;
            const double* w = val + r * k;
            const double* wb = dval + r * k;
            double dot = 0.0;
            for (int n = 0; n < k; ++n) dot += w[n] * wb[n];
            for (int j = 0; j < 2 * s; ++j) sb[j] = 0.0;
            for (int n = 0; n < k; ++n) {
                double g = w[n] * (wb[n] - dot);
                sb[I[n] / s] += g;
                sb[s + I[n] % s] += g;
            }
            double* out = dx + r * dk;
            if (cb) {
                int dh = dk / 2;
                const double* cbh = cb + (size_t)h * 2 * s * dh;
                for (int hh = 0; hh < 2; ++hh)
                    for (int c = 0; c < dh; ++c) {
                        double acc = 0.0;
                        for (int j = 0; j < s; ++j) acc += sb[hh * s + j] * cbh[((size_t)hh * s + j) * dh + c];
                        out[hh * dh + c] = acc;
                    }
            } else {
                for (int j = 0; j < 2 * s; ++j) out[j] = sb[j];
            }
        }
        free(sb);
    }
    return 0;
}

/* ------------------------------------------------------------ gates
 * Sec. 3.1 step 2: the forget gate alpha_t = exp(-A softplus(W_a x_t + b_dt))
 * and the input gate beta_t = sigma(W_b x_t), one of each per head and token.
 * The projections W_a x_t and W_b x_t arrive as the pre-activations a and b
 * [S, T] (S = B*H streams, head h = s mod H); A and b_dt are per head [H]
 * (Sec. 4 initialises A in [0, 16] and b_dt from inverse softplus of
 * [0.001, 0.1]). */
static double softplus(double z) {
    /* log(1 + e^z), written so that neither branch overflows */
    return z > 0.0 ? z + log1p(exp(-z)) : log1p(exp(z));
}

static double sigmoid(double z) {
    return z >= 0.0 ? 1.0 / (1.0 + exp(-z)) : exp(z) / (1.0 + exp(z));
}

int orc_gates(int S, int H, int T, const double* a, const double* b, const double* A, const double* b_dt,
              double* alpha, double* beta) {
    if (S < 0 || H < 1 || T < 0) return -1;
    for (int64_t s = 0; s < S; ++s) {
        const int h = (int)(s % H);
        for (int t = 0; t < T; ++t) {
            const int64_t i = s * T + t;
            alpha[i] = exp(-A[h] * softplus(a[i] + b_dt[h]));
            beta[i] = sigmoid(b[i]);
        }
    }
    return 0;
}

/* Reverse mode of orc_gates.  With z = a + b_dt: d alpha / dz = -A alpha
 * sigma(z) (softplus' = sigma), d alpha / dA = -softplus(z) alpha,
 * d beta / db = beta (1 - beta).  dA and db_dt sum over every (b, t) of the
 * head. */
int orc_gates_bwd(int S, int H, int T, const double* a, const double* b, const double* A,
                  const double* b_dt, const double* dalpha, const double* dbeta, double* da, double* db,
                  double* dA, double* db_dt) {
    if (S < 0 || H < 1 || T < 0) return -1;
    for (int h = 0; h < H; ++h) dA[h] = db_dt[h] = 0.0;
    for (int64_t s = 0; s < S; ++s) {
        const int h = (int)(s % H);
        for (int t = 0; t < T; ++t) {
            const int64_t i = s * T + t;
            const double z = a[i] + b_dt[h];
            const double al = exp(-A[h] * softplus(z));
            const double dz = dalpha[i] * (-A[h] * al * sigmoid(z));
            da[i] = dz;
            db_dt[h] += dz;
            dA[h] += dalpha[i] * (-softplus(z) * al);
            const double be = sigmoid(b[i]);
            db[i] = dbeta[i] * be * (1.0 - be);
        }
    }
    return 0;
}

/* ------------------------------------------------------------ output epilogue
 * Sec. 3.1 step 4 ("Norm, Gating, and Head Mixing") and Fig. 2's
 * g_t (.) Norm(y_t): per (b, h, t) row of d_v values,
 *   rstd = 1 / sqrt(mean_c y[c]^2 + eps),  o[c] = y[c] rstd gamma[c] phi(g[c]),
 * with gamma [d_v] the norm's scale (shared by heads) and phi the gate's
 * activation: act = 0 identity (the text's element-wise gate), act = 1
 * SiLU, phi(g) = g sigma(g).  W_o, which mixes the heads afterwards, is a
 * plain GEMM and not part of this step. */
static double gate_act(double g, int act) { return act ? g * sigmoid(g) : g; }

static double gate_act_grad(double g, int act) {
    if (!act) return 1.0;
    const double sg = sigmoid(g);
    return sg * (1.0 + g * (1.0 - sg));
}

int orc_norm_gate(int64_t rows, int dv, const double* y, const double* g, const double* gamma, double eps,
                  int act, double* o, double* rstd) {
    if (rows < 0 || dv < 1 || (act != 0 && act != 1)) return -1;
    for (int64_t r = 0; r < rows; ++r) {
        const double* yr = y + r * dv;
        double ss = 0.0;
        for (int c = 0; c < dv; ++c) ss += yr[c] * yr[c];
        const double rs = 1.0 / sqrt(ss / dv + eps);
        rstd[r] = rs;
        for (int c = 0; c < dv; ++c) o[r * dv + c] = yr[c] * rs * gamma[c] * gate_act(g[r * dv + c], act);
    }
    return 0;
}

/* Reverse mode of orc_norm_gate, with n = y rstd:
 *   dg = do gamma n phi'(g);  dn = do phi(g) gamma;  dgamma = sum over rows of do phi(g) n;
 *   dy = rstd (dn - n mean_c(dn n)). */
int orc_norm_gate_bwd(int64_t rows, int dv, const double* y, const double* g, const double* gamma, double eps,
                      int act, const double* dout, double* dy, double* dg, double* dgamma) {
    if (rows < 0 || dv < 1 || (act != 0 && act != 1)) return -1;
    for (int c = 0; c < dv; ++c) dgamma[c] = 0.0;
    double* dn = (double*)malloc(sizeof(double) * dv);
    if (!dn) return -1;
    for (int64_t r = 0; r < rows; ++r) {
        const double* yr = y + r * dv;
        double ss = 0.0;
        for (int c = 0; c < dv; ++c) ss += yr[c] * yr[c];
        const double rs = 1.0 / sqrt(ss / dv + eps);
        double dot = 0.0;
        for (int c = 0; c < dv; ++c) {
            const int64_t i = r * dv + c;
            const double n = yr[c] * rs;
            const double ph = gate_act(g[i], act);
            dg[i] = dout[i] * gamma[c] * n * gate_act_grad(g[i], act);
            dgamma[c] += dout[i] * ph * n;
            dn[c] = dout[i] * ph * gamma[c];
            dot += dn[c] * n;
        }
        dot /= dv;
        for (int c = 0; c < dv; ++c) dy[r * dv + c] = rs * (dn[c] - yr[c] * rs * dot);
    }
    free(dn);
    return 0;
}

int orc_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the parallel loops that follow (n >= 1); timing only. */
void orc_set_threads(int n) {
#ifdef _OPENMP
    omp_set_num_threads(n < 1 ? 1 : n);
#else
    (void)n;
#endif
}
