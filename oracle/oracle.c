/*
 * oracle.c -- reference CPU implementation of batched linear-chain CRF inference.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, float64 checker that the
 * GPU path is compared against.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * What it computes (Torch-Struct, Rush 2020, Sec. 5.1 and 5.2):
 *   - a sequence of L tokens z_0..z_{L-1}, each taking one of C labels, scored by
 *     edge log-potentials l[t, z_t, z_{t+1}] for t = 0..L-2 (Sec. 5.2, the linear-chain
 *     example: the first index of an edge potential is the earlier label, summed first);
 *   - the log-partition A(l) = log sum_z exp sum_t l[t, z_t, z_{t+1}]  (Sec. 5.1, CRF
 *     definition; Sec. 5.2, forward algorithm in the (logsumexp, +) semiring);
 *   - the edge marginals p(z_t = i, z_{t+1} = j) = dA/dl[t,i,j] (Sec. 5.1, gradient
 *     identity), here by the classical two-pass forward-backward recursion;
 *   - the max score A*(l) = max_z sum_t l[t,z_t,z_{t+1}] and its argmax path, the
 *     (max, +) instance of the same recursion (Sec. 5.2; Table 2, "Max" semiring),
 *     with ties resolved by taking the lowest label index at every backtrace step;
 *   - the entropy H = -sum_z p(z) log p(z) of the chain distribution (Sec. 5.1; the
 *     quantity of Table 2's "Entropy" semiring), from the edge marginals by the chain
 *     rule, and the log-probability log p(z) of a given label sequence (Sec. 5.1);
 *   - samples from p(z) by forward filtering, backward sampling with caller-supplied
 *     uniforms (Table 2's "Sample" semiring draws from the same distribution);
 *   - the semi-Markov CRF of Table 1 (segment labels, parts N K C^2): log Z, segment
 *     marginals and the best segmentation by the segmental forward-backward recursion.
 *
 * Conventions (the paper leaves these open; the readings are listed in the design notes):
 *   - pot is [B, N-1, C, C] row-major: pot[((b*(N-1)+t)*C+i)*C+j] = l[b, t, i, j].
 *   - lengths[b] counts tokens, 1 <= lengths[b] <= N; edges t >= lengths[b]-1 are padding
 *     (the semiring identity, Sec. 6a / Fig. 3) and get marginal 0.
 *   - no start or end potentials: the first and last labels are summed over freely, so
 *     a single token gives A = log C.
 *   - -inf potentials are allowed (the semiring zero); an all -inf row of sums gives -inf.
 *
 * Arithmetic: float64 throughout, libm exp/log, no fast-math.  fp32 inputs are widened
 * exactly on read.  Viterbi compares float64 sums exactly.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_ARG -1
#define ORC_ERR_MEM -2

/* element (b,t,i,j) of the potentials, widened to double */
static inline double pot_at(const float* pf, const double* pd, int64_t N, int64_t C,
                            int64_t b, int64_t t, int64_t i, int64_t j) {
    int64_t idx = ((b * (N - 1) + t) * C + i) * C + j;
    return pd ? pd[idx] : (double)pf[idx];
}

/* log(sum_k exp(x[k])) with the usual max shift; all -inf gives -inf (Sec. 5.1, LSE). */
static double lse(const double* x, int64_t n) {
    double m = -INFINITY;
    for (int64_t k = 0; k < n; ++k)
        if (x[k] > m) m = x[k];
    if (m == -INFINITY) return -INFINITY;
    double s = 0.0;
    for (int64_t k = 0; k < n; ++k) s += exp(x[k] - m);
    return m + log(s);
}

static int check_args(const void* pf, const void* pd, const int32_t* lengths, int64_t B,
                      int64_t N, int64_t C) {
    if ((!pf && !pd) || B < 1 || N < 1 || C < 1) return ORC_ERR_ARG;
    if (lengths)
        for (int64_t b = 0; b < B; ++b)
            if (lengths[b] < 1 || lengths[b] > N) return ORC_ERR_ARG;
    return ORC_OK;
}

/*
 * Forward log-messages of one sequence (Sec. 5.2, the forward algorithm):
 *   alpha_0(i) = 0,  alpha_{t+1}(j) = LSE_i [alpha_t(i) + l[t,i,j]],  A = LSE_j alpha_{L-1}(j)
 * alpha is [L, C]; tmp is [C].  Returns A.
 */
static double fwd_seq(const float* pf, const double* pd, int64_t N, int64_t C, int64_t b,
                      int64_t L, double* alpha, double* tmp) {
    for (int64_t i = 0; i < C; ++i) alpha[i] = 0.0;
    for (int64_t t = 0; t + 1 < L; ++t)
        for (int64_t j = 0; j < C; ++j) {
            for (int64_t i = 0; i < C; ++i)
                tmp[i] = alpha[t * C + i] + pot_at(pf, pd, N, C, b, t, i, j);
            alpha[(t + 1) * C + j] = lse(tmp, C);
        }
    return lse(alpha + (L - 1) * C, C);
}

/*
 * Forward and backward log-messages of one sequence (the forward algorithm and its
 * reverse):  beta_{L-1}(j) = 0,  beta_t(i) = LSE_j [l[t,i,j] + beta_{t+1}(j)].
 * alpha and beta are [L, C]; tmp is [C].  Returns A.
 */
static double fwd_bwd_seq(const float* pf, const double* pd, int64_t N, int64_t C, int64_t b,
                          int64_t L, double* alpha, double* beta, double* tmp) {
    const double A = fwd_seq(pf, pd, N, C, b, L, alpha, tmp);
    for (int64_t j = 0; j < C; ++j) beta[(L - 1) * C + j] = 0.0;
    for (int64_t t = L - 2; t >= 0; --t)
        for (int64_t i = 0; i < C; ++i) {
            for (int64_t j = 0; j < C; ++j)
                tmp[j] = pot_at(pf, pd, N, C, b, t, i, j) + beta[(t + 1) * C + j];
            beta[t * C + i] = lse(tmp, C);
        }
    return A;
}

/* mu[t,i,j] = exp(alpha_t(i) + l[t,i,j] + beta_{t+1}(j) - A)  (Sec. 5.1: p(z_p=1) = dA/dl_p) */
static void edge_marginal(const float* pf, const double* pd, int64_t N, int64_t C, int64_t b,
                          int64_t t, const double* alpha, const double* beta, double logZ,
                          double* out) {
    for (int64_t i = 0; i < C; ++i)
        for (int64_t j = 0; j < C; ++j) {
            double v = 0.0;
            if (logZ != -INFINITY)
                v = exp(alpha[t * C + i] + pot_at(pf, pd, N, C, b, t, i, j) +
                        beta[(t + 1) * C + j] - logZ);
            out[i * C + j] = v;
        }
}

static int logpartition_impl(const float* pf, const double* pd, const int32_t* lengths,
                             int64_t B, int64_t N, int64_t C, double* logZ) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc) return rc;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t L = lengths ? lengths[b] : N;
        double* alpha = malloc(sizeof(double) * L * C);
        double* tmp = malloc(sizeof(double) * C);
        if (!alpha || !tmp) {
#pragma omp atomic write
            err = 1;
        } else {
            logZ[b] = fwd_seq(pf, pd, N, C, b, L, alpha, tmp);
        }
        free(alpha); free(tmp);
    }
    return err ? ORC_ERR_MEM : ORC_OK;
}

static int marginals_impl(const float* pf, const double* pd, const int32_t* lengths, int64_t B,
                          int64_t N, int64_t C, double* logZ, double* marg) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc) return rc;
    if (N == 1) return logpartition_impl(pf, pd, lengths, B, N, C, logZ);
    int err = 0;
    double* alpha = malloc(sizeof(double) * B * N * C);
    double* beta = malloc(sizeof(double) * B * N * C);
    if (!alpha || !beta) { free(alpha); free(beta); return ORC_ERR_MEM; }
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t L = lengths ? lengths[b] : N;
        double* tmp = malloc(sizeof(double) * C);
        if (!tmp) {
#pragma omp atomic write
            err = 1;
        } else {
            logZ[b] = fwd_bwd_seq(pf, pd, N, C, b, L, alpha + b * N * C, beta + b * N * C, tmp);
        }
        free(tmp);
    }
    if (!err) {
#pragma omp parallel for collapse(2) schedule(static)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t t = 0; t < N - 1; ++t) {
                int64_t L = lengths ? lengths[b] : N;
                double* out = marg + (b * (N - 1) + t) * C * C;
                if (t + 1 < L)
                    edge_marginal(pf, pd, N, C, b, t, alpha + b * N * C, beta + b * N * C,
                                  logZ[b], out);
                else
                    memset(out, 0, sizeof(double) * C * C);
            }
    }
    free(alpha); free(beta);
    return err ? ORC_ERR_MEM : ORC_OK;
}

/*
 * Viterbi DP, the (max, +) instance (Sec. 5.1 A*, Sec. 5.2, Table 2 "Max"):
 *   delta_0(i) = 0,  delta_{t+1}(j) = max_i [delta_t(i) + l[t,i,j]],
 *   bp_{t+1}(j) = the smallest i that attains the max;
 *   score = max_j delta_{L-1}(j), z_{L-1} = the smallest j that attains it,
 *   z_t = bp_{t+1}(z_{t+1});  path[n] = -1 for n >= L.
 */
static int viterbi_impl(const float* pf, const double* pd, const int32_t* lengths, int64_t B,
                        int64_t N, int64_t C, int32_t* path, double* score) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc) return rc;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t L = lengths ? lengths[b] : N;
        double* delta = malloc(sizeof(double) * L * C);
        int32_t* bp = malloc(sizeof(int32_t) * L * C);
        if (!delta || !bp) {
#pragma omp atomic write
            err = 1;
            free(delta); free(bp);
            continue;
        }
        for (int64_t i = 0; i < C; ++i) delta[i] = 0.0;
        for (int64_t t = 0; t + 1 < L; ++t)
            for (int64_t j = 0; j < C; ++j) {
                double best = delta[t * C] + pot_at(pf, pd, N, C, b, t, 0, j);
                int32_t arg = 0;
                for (int64_t i = 1; i < C; ++i) {
                    double v = delta[t * C + i] + pot_at(pf, pd, N, C, b, t, i, j);
                    if (v > best) { best = v; arg = (int32_t)i; }
                }
                delta[(t + 1) * C + j] = best;
                bp[(t + 1) * C + j] = arg;
            }
        double best = delta[(L - 1) * C];
        int32_t z = 0;
        for (int64_t j = 1; j < C; ++j)
            if (delta[(L - 1) * C + j] > best) { best = delta[(L - 1) * C + j]; z = (int32_t)j; }
        score[b] = best;
        int32_t* p = path + b * N;
        for (int64_t n = L; n < N; ++n) p[n] = -1;
        p[L - 1] = z;
        for (int64_t t = L - 2; t >= 0; --t) {
            z = bp[(t + 1) * C + z];
            p[t] = z;
        }
        free(delta); free(bp);
    }
    return err ? ORC_ERR_MEM : ORC_OK;
}

/*
 * Entropy of p(z) = exp(sum_t l[t,z_t,z_{t+1}] - A) for each sequence.  A chain is a
 * Markov chain under p, so by the chain rule of entropy
 *   H = H(z_0) + sum_{t < L-1} H(z_{t+1} | z_t),
 *   H(z_0) = -sum_i m_0(i) log m_0(i),   m_t(i) = sum_j mu[t,i,j]  (node marginals),
 *   H(z_{t+1} | z_t) = -sum_{i,j} mu[t,i,j] log(mu[t,i,j] / m_t(i)),   0 log 0 = 0,
 * with mu the edge marginals above.  One token: H = log C (a free label).  A sequence with
 * no finite path has all marginals 0 and gets H = 0.
 */
static int entropy_impl(const float* pf, const double* pd, const int32_t* lengths, int64_t B,
                        int64_t N, int64_t C, double* H) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc) return rc;
    if (N == 1) {
        for (int64_t b = 0; b < B; ++b) H[b] = log((double)C);
        return ORC_OK;
    }
    double* logZ = malloc(sizeof(double) * B);
    double* marg = malloc(sizeof(double) * B * (N - 1) * C * C);
    if (!logZ || !marg) { free(logZ); free(marg); return ORC_ERR_MEM; }
    rc = marginals_impl(pf, pd, lengths, B, N, C, logZ, marg);
    if (rc == ORC_OK) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t b = 0; b < B; ++b) {
            int64_t L = lengths ? lengths[b] : N;
            if (L == 1) { H[b] = log((double)C); continue; }
            double h = 0.0;
            for (int64_t t = 0; t + 1 < L; ++t) {
                const double* mu = marg + (b * (N - 1) + t) * C * C;
                for (int64_t i = 0; i < C; ++i) {
                    double m = 0.0;
                    for (int64_t j = 0; j < C; ++j) m += mu[i * C + j];
                    if (m <= 0.0) continue;
                    if (t == 0) h -= m * log(m);
                    for (int64_t j = 0; j < C; ++j)
                        if (mu[i * C + j] > 0.0) h -= mu[i * C + j] * log(mu[i * C + j] / m);
                }
            }
            H[b] = h;
        }
    }
    free(logZ); free(marg);
    return rc;
}

/*
 * log p(z) = sum_{t < L-1} l[t, z_t, z_{t+1}] - A for the label sequence labels[b, :L]
 * (Sec. 5.1, the CRF probability of one structure); entries n >= L are ignored.  A label
 * outside [0, C) is an argument error.
 */
static int log_density_impl(const float* pf, const double* pd, const int32_t* lengths,
                            const int32_t* labels, int64_t B, int64_t N, int64_t C,
                            double* out) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc) return rc;
    if (!labels) return ORC_ERR_ARG;
    for (int64_t b = 0; b < B; ++b) {
        int64_t L = lengths ? lengths[b] : N;
        for (int64_t n = 0; n < L; ++n)
            if (labels[b * N + n] < 0 || labels[b * N + n] >= C) return ORC_ERR_ARG;
    }
    double* logZ = malloc(sizeof(double) * B);
    if (!logZ) return ORC_ERR_MEM;
    rc = logpartition_impl(pf, pd, lengths, B, N, C, logZ);
    if (rc == ORC_OK)
        for (int64_t b = 0; b < B; ++b) {
            int64_t L = lengths ? lengths[b] : N;
            const int32_t* z = labels + b * N;
            double s = 0.0;
            for (int64_t t = 0; t + 1 < L; ++t) s += pot_at(pf, pd, N, C, b, t, z[t], z[t + 1]);
            out[b] = s - logZ[b];
        }
    free(logZ);
    return rc;
}

/*
 * Forward filtering, backward sampling (the "Sample" semiring of Table 2 draws from the
 * same distribution): with edge marginals mu and node marginals m,
 *   z_{L-1} ~ m_{L-1}(j) = sum_i mu[L-2, i, j],
 *   z_t | z_{t+1} = j ~ p(z_t = i | z_{t+1} = j) = mu[t, i, j] / m_{t+1}(j),  t = L-2..0
 * (the Markov property of the chain).  One token: z_0 uniform over the C labels.  Each
 * draw takes the caller's uniform u in [0, 1) by inverse CDF: the smallest k whose
 * inclusive prefix sum of the weights exceeds u * total (all-zero weights: k = 0).
 * uniforms and paths are [S, B, N]; paths get -1 past each length.  margin[s*B + b]
 * receives the smallest distance of u * total from an edge of the chosen bin, relative to
 * the total, over that sequence's draws (how close the draw came to a different label).
 */
static int draw(const double* w, int64_t C, double u, double* margin) {
    double tot = 0.0;
    for (int64_t k = 0; k < C; ++k) tot += w[k];
    if (!(tot > 0.0)) { *margin = INFINITY; return 0; }
    const double x = u * tot;
    double cum = 0.0;
    for (int64_t k = 0; k < C; ++k) {
        const double lo = cum;
        cum += w[k];
        if (cum > x || k == C - 1) {
            const double d = fmin(x - lo, cum - x) / tot;
            *margin = d;
            return (int)k;
        }
    }
    *margin = INFINITY;
    return 0;
}

static int sample_impl(const float* pf, const int32_t* lengths, const float* uniforms,
                       int64_t S, int64_t B, int64_t N, int64_t C, int32_t* paths,
                       double* margin) {
    int rc = check_args(pf, NULL, lengths, B, N, C);
    if (rc) return rc;
    if (!uniforms || S < 1) return ORC_ERR_ARG;
    double* logZ = malloc(sizeof(double) * B);
    double* marg = malloc(sizeof(double) * B * (N > 1 ? N - 1 : 1) * C * C);
    double* w = malloc(sizeof(double) * C);
    if (!logZ || !marg || !w) { free(logZ); free(marg); free(w); return ORC_ERR_MEM; }
    if (N > 1) rc = marginals_impl(pf, NULL, lengths, B, N, C, logZ, marg);
    if (rc == ORC_OK)
        for (int64_t s = 0; s < S; ++s)
            for (int64_t b = 0; b < B; ++b) {
                const int64_t L = lengths ? lengths[b] : N;
                const float* u = uniforms + (s * B + b) * N;
                int32_t* z = paths + (s * B + b) * N;
                double mg = INFINITY, d;
                for (int64_t n = L; n < N; ++n) z[n] = -1;
                if (L == 1) {
                    for (int64_t k = 0; k < C; ++k) w[k] = 1.0;
                } else {
                    const double* mu = marg + (b * (N - 1) + (L - 2)) * C * C;
                    for (int64_t j = 0; j < C; ++j) {
                        w[j] = 0.0;
                        for (int64_t i = 0; i < C; ++i) w[j] += mu[i * C + j];
                    }
                }
                z[L - 1] = draw(w, C, (double)u[L - 1], &d);
                mg = fmin(mg, d);
                for (int64_t t = L - 2; t >= 0; --t) {
                    const double* mu = marg + (b * (N - 1) + t) * C * C;
                    for (int64_t i = 0; i < C; ++i) w[i] = mu[i * C + z[t + 1]];
                    z[t] = draw(w, C, (double)u[t], &d);
                    mg = fmin(mg, d);
                }
                if (margin) margin[s * B + b] = mg;
            }
    free(logZ); free(marg); free(w);
    return rc;
}

/*
 * Semi-Markov CRF (Table 1, "Semi-Markov": segment labels, parts N K C^2, segmental
 * forward-backward).  A sequence of L tokens has E = L-1 steps t = 0..E-1 (the chain's
 * edges).  A segmentation covers the steps with consecutive segments of lengths 1..K;
 * segment m spans steps [s_m, s_m + k_m) and carries label y_m, and y_0 is a free initial
 * label (the chain's z_0).  Its score is sum_m sp[s_m, k_m - 1, y_{m-1}, y_m] with
 * sp [B, N-1, K, C, C].  With K = 1 this is the linear chain exactly.
 *   alpha_0(i) = 0,  alpha_e(j) = LSE over k <= min(K, e), i of alpha_{e-k}(i) + sp[e-k, k-1, i, j],
 *   A = LSE_j alpha_E(j)  (E = 0: log C),
 *   beta_E(j) = 0,   beta_e(i) = LSE over k <= min(K, E-e), j of sp[e, k-1, i, j] + beta_{e+k}(j),
 *   mu[e, k-1, i, j] = exp(alpha_e(i) + sp[e, k-1, i, j] + beta_{e+k}(j) - A)  (dA/dsp, Sec.
 *   5.1), and 0 where e + k > E.
 * Viterbi: V the same recursion in (max, +); the last label is the lowest j maximising
 * V_E(j); going back from a segment end e with label j it takes, among the (k, i) with
 * V_{e-k}(i) + sp[e-k, k-1, i, j] = V_e(j), the smallest k and then the lowest i.
 * Outputs path[n] for n < L: path[0] = y_0 and path[t+1] = the label of the segment that
 * covers step t; seglen[t] = k where a segment of length k starts at step t, else 0; both
 * -1 past the sequence.
 */
static inline double sp_at(const float* pf, const double* pd, int64_t N, int64_t K, int64_t C,
                           int64_t b, int64_t t, int64_t k, int64_t i, int64_t j) {
    int64_t idx = (((b * (N - 1) + t) * K + k) * C + i) * C + j;
    return pd ? pd[idx] : (double)pf[idx];
}

/* alpha [E+1, C] and beta [E+1, C] of one sequence with E steps; tmp [K*C].  Returns A. */
static double semi_fwd_bwd(const float* pf, const double* pd, int64_t N, int64_t K, int64_t C,
                           int64_t b, int64_t E, double* alpha, double* beta, double* tmp) {
    for (int64_t i = 0; i < C; ++i) alpha[i] = 0.0;
    for (int64_t e = 1; e <= E; ++e)
        for (int64_t j = 0; j < C; ++j) {
            int64_t n = 0;
            for (int64_t k = 1; k <= K && k <= e; ++k)
                for (int64_t i = 0; i < C; ++i)
                    tmp[n++] = alpha[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k - 1, i, j);
            alpha[e * C + j] = lse(tmp, n);
        }
    for (int64_t j = 0; j < C; ++j) beta[E * C + j] = 0.0;
    for (int64_t e = E - 1; e >= 0; --e)
        for (int64_t i = 0; i < C; ++i) {
            int64_t n = 0;
            for (int64_t k = 1; k <= K && e + k <= E; ++k)
                for (int64_t j = 0; j < C; ++j)
                    tmp[n++] = sp_at(pf, pd, N, K, C, b, e, k - 1, i, j) + beta[(e + k) * C + j];
            beta[e * C + i] = lse(tmp, n);
        }
    return E == 0 ? log((double)C) : lse(alpha + E * C, C);
}

static int semi_marginals_impl(const float* pf, const double* pd, const int32_t* lengths,
                               int64_t B, int64_t N, int64_t K, int64_t C, double* logZ,
                               double* marg) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc || K < 1) return rc ? rc : ORC_ERR_ARG;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        const int64_t E = (lengths ? lengths[b] : N) - 1;
        double* alpha = malloc(sizeof(double) * (E + 1) * C);
        double* beta = malloc(sizeof(double) * (E + 1) * C);
        double* tmp = malloc(sizeof(double) * K * C);
        if (!alpha || !beta || !tmp) {
#pragma omp atomic write
            err = 1;
            free(alpha); free(beta); free(tmp);
            continue;
        }
        const double A = semi_fwd_bwd(pf, pd, N, K, C, b, E, alpha, beta, tmp);
        logZ[b] = A;
        if (marg)
            for (int64_t e = 0; e < N - 1; ++e)
                for (int64_t k = 1; k <= K; ++k)
                    for (int64_t i = 0; i < C; ++i)
                        for (int64_t j = 0; j < C; ++j) {
                            double v = 0.0;
                            if (e + k <= E && A != -INFINITY)
                                v = exp(alpha[e * C + i] + sp_at(pf, pd, N, K, C, b, e, k - 1, i, j)
                                        + beta[(e + k) * C + j] - A);
                            marg[((((b * (N - 1) + e) * K) + k - 1) * C + i) * C + j] = v;
                        }
        free(alpha); free(beta); free(tmp);
    }
    return err ? ORC_ERR_MEM : ORC_OK;
}

static int semi_viterbi_impl(const float* pf, const double* pd, const int32_t* lengths,
                             int64_t B, int64_t N, int64_t K, int64_t C, int32_t* path,
                             int32_t* seglen, double* score) {
    int rc = check_args(pf, pd, lengths, B, N, C);
    if (rc || K < 1) return rc ? rc : ORC_ERR_ARG;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        const int64_t E = (lengths ? lengths[b] : N) - 1;
        double* V = malloc(sizeof(double) * (E + 1) * C);
        if (!V) {
#pragma omp atomic write
            err = 1;
            continue;
        }
        for (int64_t i = 0; i < C; ++i) V[i] = 0.0;
        for (int64_t e = 1; e <= E; ++e)
            for (int64_t j = 0; j < C; ++j) {
                double best = -INFINITY;
                for (int64_t k = 1; k <= K && k <= e; ++k)
                    for (int64_t i = 0; i < C; ++i) {
                        double v = V[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k - 1, i, j);
                        if (v > best) best = v;
                    }
                V[e * C + j] = best;
            }
        int32_t j = 0;
        for (int64_t c = 1; c < C; ++c)
            if (V[E * C + c] > V[E * C + j]) j = (int32_t)c;
        score[b] = V[E * C + j];
        int32_t* p = path + b * N;
        int32_t* g = seglen + b * (N - 1);
        for (int64_t n = E + 1; n < N; ++n) p[n] = -1;
        for (int64_t t = 0; t < N - 1; ++t) g[t] = t < E ? 0 : -1;
        /* walk back over the segments: the smallest k, then the lowest i, that attains V */
        int64_t e = E;
        while (e > 0) {
            int64_t kb = 1;
            int32_t ib = 0;
            int found = 0;
            for (int64_t k = 1; k <= K && k <= e && !found; ++k)
                for (int64_t i = 0; i < C && !found; ++i)
                    if (V[(e - k) * C + i] + sp_at(pf, pd, N, K, C, b, e - k, k - 1, i, j) ==
                        V[e * C + j]) {
                        kb = k;
                        ib = (int32_t)i;
                        found = 1;
                    }
            for (int64_t t = e - kb; t < e; ++t) p[t + 1] = j;
            g[e - kb] = (int32_t)kb;
            j = ib;
            e -= kb;
        }
        p[0] = j;
        free(V);
    }
    return err ? ORC_ERR_MEM : ORC_OK;
}

/* ---------------- exported entry points ---------------- */

/* OpenMP threads a parallel region of the oracle may use */
int orc_max_threads(void) { return omp_get_max_threads(); }

/* fp32 potentials, widened exactly */
int orc_logpartition(const float* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                     double* logZ) {
    return logpartition_impl(pot, NULL, lengths, B, N, C, logZ);
}
int orc_marginals(const float* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                  double* logZ, double* marg) {
    return marginals_impl(pot, NULL, lengths, B, N, C, logZ, marg);
}
int orc_viterbi(const float* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                int32_t* path, double* score) {
    return viterbi_impl(pot, NULL, lengths, B, N, C, path, score);
}

int orc_entropy(const float* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                double* H) {
    return entropy_impl(pot, NULL, lengths, B, N, C, H);
}
int orc_log_density(const float* pot, const int32_t* lengths, const int32_t* labels, int64_t B,
                    int64_t N, int64_t C, double* out) {
    return log_density_impl(pot, NULL, lengths, labels, B, N, C, out);
}

int orc_sample(const float* pot, const int32_t* lengths, const float* uniforms, int64_t S,
               int64_t B, int64_t N, int64_t C, int32_t* paths, double* margin) {
    return sample_impl(pot, lengths, uniforms, S, B, N, C, paths, margin);
}

/* float64 potentials (used by the finite-difference pins) */
int orc_logpartition_f64(const double* pot, const int32_t* lengths, int64_t B, int64_t N,
                         int64_t C, double* logZ) {
    return logpartition_impl(NULL, pot, lengths, B, N, C, logZ);
}
int orc_marginals_f64(const double* pot, const int32_t* lengths, int64_t B, int64_t N,
                      int64_t C, double* logZ, double* marg) {
    return marginals_impl(NULL, pot, lengths, B, N, C, logZ, marg);
}
int orc_viterbi_f64(const double* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                    int32_t* path, double* score) {
    return viterbi_impl(NULL, pot, lengths, B, N, C, path, score);
}

/*
 * Marginals of edges t0 <= t < t1 of sequence b only (fp32 potentials), for sampled
 * comparisons at sizes where the full float64 marginal tensor is too large to keep.
 * out is [(t1-t0), C, C]; edges at or past the sequence's last edge get 0.
 * logZ_out (nullable) receives A for sequence b.
 */
int orc_marginals_seq(const float* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                      int64_t b, int64_t t0, int64_t t1, double* out, double* logZ_out) {
    if (!pot || b < 0 || b >= B || t0 < 0 || t1 < t0 || t1 > N - 1 || C < 1) return ORC_ERR_ARG;
    int64_t L = lengths ? lengths[b] : N;
    if (L < 1 || L > N) return ORC_ERR_ARG;
    double* alpha = malloc(sizeof(double) * L * C);
    double* beta = malloc(sizeof(double) * L * C);
    double* tmp = malloc(sizeof(double) * C);
    if (!alpha || !beta || !tmp) { free(alpha); free(beta); free(tmp); return ORC_ERR_MEM; }
    double logZ = fwd_bwd_seq(pot, NULL, N, C, b, L, alpha, beta, tmp);
    if (logZ_out) *logZ_out = logZ;
#pragma omp parallel for schedule(static)
    for (int64_t t = t0; t < t1; ++t) {
        double* o = out + (t - t0) * C * C;
        if (t + 1 < L)
            edge_marginal(pot, NULL, N, C, b, t, alpha, beta, logZ, o);
        else
            memset(o, 0, sizeof(double) * C * C);
    }
    free(alpha); free(beta); free(tmp);
    return ORC_OK;
}

/*
 * Streamed marginals, for sizes where the float64 tensor [B, N-1, C, C] is too large to
 * hold at once.  orc_messages runs the forward and backward recursions of every sequence
 * once (the same fwd_bwd_seq as orc_marginals): alpha and beta are [B, N, C] (rows at or
 * past a sequence's length are left unwritten), logZ is [B].  orc_edge_marginals then
 * forms the marginals of edges t0 <= t < t1 of sequence b from them with the same
 * edge_marginal as orc_marginals, so the two agree bitwise; out is [(t1-t0), C, C] and
 * edges at or past the sequence's last edge are 0.
 */
int orc_messages(const float* pot, const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                 double* alpha, double* beta, double* logZ) {
    int rc = check_args(pot, NULL, lengths, B, N, C);
    if (rc) return rc;
    if (!alpha || !beta || !logZ) return ORC_ERR_ARG;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        int64_t L = lengths ? lengths[b] : N;
        double* tmp = malloc(sizeof(double) * C);
        if (!tmp) {
#pragma omp atomic write
            err = 1;
        } else {
            logZ[b] = fwd_bwd_seq(pot, NULL, N, C, b, L, alpha + b * N * C, beta + b * N * C, tmp);
        }
        free(tmp);
    }
    return err ? ORC_ERR_MEM : ORC_OK;
}

int orc_edge_marginals(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                       int64_t C, const double* alpha, const double* beta, const double* logZ,
                       int64_t b, int64_t t0, int64_t t1, double* out) {
    if (!pot || !alpha || !beta || !logZ || !out || b < 0 || b >= B || t0 < 0 || t1 < t0 ||
        t1 > N - 1 || C < 1)
        return ORC_ERR_ARG;
    int64_t L = lengths ? lengths[b] : N;
    if (L < 1 || L > N) return ORC_ERR_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t t = t0; t < t1; ++t) {
        double* o = out + (t - t0) * C * C;
        if (t + 1 < L)
            edge_marginal(pot, NULL, N, C, b, t, alpha + b * N * C, beta + b * N * C, logZ[b], o);
        else
            memset(o, 0, sizeof(double) * C * C);
    }
    return ORC_OK;
}

/* semi-Markov CRF: sp [B, N-1, K, C, C] (fp32 widened exactly, or float64) */
int orc_semi_marginals(const float* sp, const int32_t* lengths, int64_t B, int64_t N, int64_t K,
                       int64_t C, double* logZ, double* marg) {
    return semi_marginals_impl(sp, NULL, lengths, B, N, K, C, logZ, marg);
}
int orc_semi_marginals_f64(const double* sp, const int32_t* lengths, int64_t B, int64_t N,
                           int64_t K, int64_t C, double* logZ, double* marg) {
    return semi_marginals_impl(NULL, sp, lengths, B, N, K, C, logZ, marg);
}
int orc_semi_viterbi(const float* sp, const int32_t* lengths, int64_t B, int64_t N, int64_t K,
                     int64_t C, int32_t* path, int32_t* seglen, double* score) {
    return semi_viterbi_impl(sp, NULL, lengths, B, N, K, C, path, seglen, score);
}
