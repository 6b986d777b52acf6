/*
 * ga_oracle.c -- CPU oracle for RITA group attention (test infrastructure).
 *
 * This file is test infrastructure.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg load it; the GPU library never does.  It shares
 * no code with the GPU path.
 *
 * Plain, slow, fp64 C written from the paper's definitions:
 *   - grouping: Lloyd K-means on the keys, "a few" iterations (Section 4.4),
 *     with the squared distance expanded as |c|^2 - 2 v.c (the |v|^2 term is
 *     the same for every centre and drops out of the argmin);
 *   - embedding aggregation: per-group SUM of the value vectors (Section 4.2,
 *     Algorithm 1, embedding-aggregation loop);
 *   - group softmax (Eq. 3) and output combine (Algorithm 1);
 *   - the adaptive scheduler's merge plan (Section 5.1: Lemma 1 turns the
 *     error bound eps into a distance threshold, the simplified rule of Eq. 5
 *     marks mergeable groups).
 *
 * Readings where the paper is silent:
 *   init     C0_j = k_{floor(j*n/N)} (strided), or a caller-given fp32 init.
 *   iters    T = number of (assign, update) rounds, no convergence test.
 *   R        R = round_dt(C): identity for fp32 inputs, round-to-nearest-even
 *            to bfloat16 for bf16 inputs; R is the representative key used
 *            both for assignment and for the attention scores.
 *   score    nrm_j = sum_c r_jc*r_jc and dot_ij = sum_c k_ic*r_jc as fp64 fma
 *            chains in the order c = 0..d-1 starting from 0, and
 *            s_ij = fma(-2, dot_ij, nrm_j).  a_i = lowest j with minimal s_ij.
 *   update   count_j = #{i: a_i = j}; S_j = sum over members in ascending i
 *            (fp64); C_j = (float)(S_j / count_j); an empty group keeps C_j.
 *   softmax  p_ij = scale * (q_i . r_j); the max m_i is taken over non-empty
 *            groups only and subtracted (exact in real arithmetic); groups with
 *            count 0 contribute nothing; o_i = sum_j e_ij vsum_j / s_i with
 *            s_i = sum_j count_j e_ij (no count factor in the numerator, since
 *            vsum is already a sum over the group's members).
 *
 * Layout: every tensor is dense row-major, [B, H, n, d] / [B, H, N, d] /
 * [B, H, n] / [B, H, N].  Inputs arrive as doubles holding the exact values of
 * the bf16 / fp32 inputs.  dtype: 0 = fp32, 1 = bf16.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

/* Round a float to the nearest bfloat16 (ties to even), returned as a float. */
static float oracle_round_bf16(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) { /* inf / nan: truncate */
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u += 0x7fffu + lsb;
        u &= 0xffff0000u;
    }
    float y;
    memcpy(&y, &u, 4);
    return y;
}

static double round_dt(float c, int dtype) {
    return dtype == ORACLE_BF16 ? (double)oracle_round_bf16(c) : (double)c;
}

/* Exactness check of one fp64 addition a + b (Knuth's TwoSum error term). */
static int add_inexact(double a, double b, double s) {
    double bb = s - a;
    double err = (a - (s - bb)) + (b - bb);
    return err != 0.0;
}

int ga_oracle_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
    return omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}

/* Canonical squared-norm of a representative: fma chain over c = 0..d-1. */
static double canon_nrm(const double *r, int d) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc = fma(r[c], r[c], acc);
    return acc;
}

/* Canonical score of key k against representative r with norm nrm. */
static double canon_score(const double *k, const double *r, double nrm, int d) {
    double dot = 0.0;
    for (int c = 0; c < d; ++c) dot = fma(k[c], r[c], dot);
    return fma(-2.0, dot, nrm);
}

/*
 * One (b, h) slice of the grouping.
 *   K      [n][d] doubles;   C [N][d] floats (in: C0, out: C^T)
 *   belong [n], count [N]
 *   trace_belong [iters][n], trace_margin [iters][n], trace_centroid
 *   [iters][N][d] (C^1..C^T) may be NULL; the strides between iterations are
 *   given so the caller can interleave slices.
 */
static int64_t cluster_slice(int n, int d, int dtype, const double *K, int N, int iters,
                             float *C, int32_t *belong, int32_t *count,
                             int32_t *trace_belong, double *trace_margin, float *trace_centroid,
                             int64_t tb_stride, int64_t tc_stride) {
    double *R = (double *)malloc(sizeof(double) * (size_t)N * d);
    double *nrm = (double *)malloc(sizeof(double) * (size_t)N);
    double *S = (double *)malloc(sizeof(double) * (size_t)N * d);
    int64_t inexact = 0;

    for (int t = 0; t < iters; ++t) {
        /* representatives of the previous centroids */
        for (int j = 0; j < N; ++j) {
            for (int c = 0; c < d; ++c) R[(size_t)j * d + c] = round_dt(C[(size_t)j * d + c], dtype);
            nrm[j] = canon_nrm(R + (size_t)j * d, d);
        }
        /* assignment: lowest index among exact minima of the canonical score */
        for (int i = 0; i < n; ++i) {
            const double *k = K + (size_t)i * d;
            double best = INFINITY, second = INFINITY;
            int bj = 0;
            for (int j = 0; j < N; ++j) {
                double s = canon_score(k, R + (size_t)j * d, nrm[j], d);
                if (s < best) {
                    second = best;
                    best = s;
                    bj = j;
                } else if (s < second) {
                    second = s;
                }
            }
            belong[i] = bj;
            if (trace_belong) trace_belong[t * tb_stride + i] = bj;
            if (trace_margin) trace_margin[t * tb_stride + i] = second - best;
        }
        /* update: counts and fp64 member sums in ascending key order */
        memset(S, 0, sizeof(double) * (size_t)N * d);
        for (int j = 0; j < N; ++j) count[j] = 0;
        for (int i = 0; i < n; ++i) {
            int j = belong[i];
            count[j] += 1;
            double *Sj = S + (size_t)j * d;
            const double *k = K + (size_t)i * d;
            for (int c = 0; c < d; ++c) {
                double s = Sj[c] + k[c];
                inexact += add_inexact(Sj[c], k[c], s);
                Sj[c] = s;
            }
        }
        for (int j = 0; j < N; ++j) {
            if (count[j] == 0) continue; /* empty group keeps its centroid */
            for (int c = 0; c < d; ++c)
                C[(size_t)j * d + c] = (float)(S[(size_t)j * d + c] / (double)count[j]);
        }
        if (trace_centroid)
            memcpy(trace_centroid + t * tc_stride, C, sizeof(float) * (size_t)N * d);
    }
    free(R);
    free(nrm);
    free(S);
    return inexact;
}

/*
 * Grouping of every (b, h) slice.  Returns the number of inexact fp64
 * additions seen in the centroid sums (0 means every sum was exact, so any
 * summation order gives the same bits).
 */
int64_t ga_oracle_cluster(int B, int H, int n, int d, int dtype, const double *K, int N,
                          int iters, const float *init_or_null, int32_t *belong,
                          int32_t *count, float *centroid, int32_t *trace_belong,
                          double *trace_margin, float *trace_centroid) {
    const int64_t BH = (int64_t)B * H;
    int64_t inexact = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : inexact)
    for (int64_t u = 0; u < BH; ++u) {
        const double *Ku = K + u * (int64_t)n * d;
        float *Cu = centroid + u * (int64_t)N * d;
        for (int j = 0; j < N; ++j) {
            if (init_or_null) {
                memcpy(Cu + (size_t)j * d, init_or_null + u * (int64_t)N * d + (size_t)j * d,
                       sizeof(float) * (size_t)d);
            } else {
                int64_t src = ((int64_t)j * n) / N;
                for (int c = 0; c < d; ++c) Cu[(size_t)j * d + c] = (float)Ku[src * d + c];
            }
        }
        inexact += cluster_slice(n, d, dtype, Ku, N, iters, Cu, belong + u * (int64_t)n,
                                 count + u * (int64_t)N,
                                 trace_belong ? trace_belong + u * (int64_t)n : NULL,
                                 trace_margin ? trace_margin + u * (int64_t)n : NULL,
                                 trace_centroid ? trace_centroid + u * (int64_t)N * d : NULL,
                                 BH * n, BH * N * d);
    }
    return inexact;
}

/*
 * Embedding aggregation: vsum_j = sum of v_i over the members of group j, in
 * ascending i, fp64.  Entries of belong outside [0, N) are ignored.
 */
int64_t ga_oracle_aggregate(int B, int H, int n, int d, const double *V, const int32_t *belong,
                            int N, double *vsum) {
    const int64_t BH = (int64_t)B * H;
    int64_t inexact = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : inexact)
    for (int64_t u = 0; u < BH; ++u) {
        double *Su = vsum + u * (int64_t)N * d;
        memset(Su, 0, sizeof(double) * (size_t)N * d);
        for (int i = 0; i < n; ++i) {
            int j = belong[u * (int64_t)n + i];
            if (j < 0 || j >= N) continue;
            const double *v = V + (u * (int64_t)n + i) * d;
            for (int c = 0; c < d; ++c) {
                double s = Su[(size_t)j * d + c] + v[c];
                inexact += add_inexact(Su[(size_t)j * d + c], v[c], s);
                Su[(size_t)j * d + c] = s;
            }
        }
    }
    return inexact;
}

/*
 * Group softmax and combine for every query.  Representatives are
 * round_dt(centroid).  A slice whose groups are all empty yields zeros.
 * O is [B, H, n, d] doubles.
 */
void ga_oracle_attend(int B, int H, int n, int d, int dtype, const double *Q,
                      const float *centroid, const int32_t *count, const double *vsum, int N,
                      double scale, double *O) {
    const int64_t BH = (int64_t)B * H;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t u = 0; u < BH; ++u) {
        double *R = (double *)malloc(sizeof(double) * (size_t)N * d);
        double *p = (double *)malloc(sizeof(double) * (size_t)N);
        const int32_t *cnt = count + u * (int64_t)N;
        const double *vs = vsum + u * (int64_t)N * d;
        for (int64_t x = 0; x < (int64_t)N * d; ++x) R[x] = round_dt(centroid[u * (int64_t)N * d + x], dtype);
        for (int i = 0; i < n; ++i) {
            const double *q = Q + (u * (int64_t)n + i) * d;
            double *o = O + (u * (int64_t)n + i) * d;
            double m = -INFINITY;
            for (int j = 0; j < N; ++j) {
                double dot = 0.0;
                for (int c = 0; c < d; ++c) dot += q[c] * R[(size_t)j * d + c];
                p[j] = scale * dot;
                if (cnt[j] > 0 && p[j] > m) m = p[j];
            }
            for (int c = 0; c < d; ++c) o[c] = 0.0;
            if (m == -INFINITY) continue; /* no non-empty group */
            double s = 0.0;
            for (int j = 0; j < N; ++j) {
                if (cnt[j] <= 0) continue;
                double e = exp(p[j] - m);
                s += (double)cnt[j] * e;
                for (int c = 0; c < d; ++c) o[c] += e * vs[(size_t)j * d + c];
            }
            for (int c = 0; c < d; ++c) o[c] /= s;
        }
        free(R);
        free(p);
    }
}

/* Squared Euclidean distance of x and y as an fp64 fma chain over c = 0..d-1
 * from 0; every difference is exact in fp64 (bf16 / fp32 operands). */
static double canon_dist2(const double *x, const double *y, int d) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) {
        const double t = x[c] - y[c];
        acc = fma(t, t, acc);
    }
    return acc;
}

/*
 * Merge plan of the adaptive scheduler (Section 5.1) for every (b, h) slice.
 *   Lemma 1: if every key lies within dthr of its group's representative and
 *     dthr <= ln(eps) / (2 R'), the restored attention is within a factor eps
 *     of the exact one; R' bounds the (scaled) query norms, which is what the
 *     proof uses: R' = |scale| max_i |q_i|.  dthr = log_eps / (2 R') (+inf if
 *     R' = 0).
 *   Lemma 2 / Eq. 5 (simplified rule): the groups are halved into
 *     S1 = [0, ceil(N/2)) and S2 = [ceil(N/2), N); a group j of S2 is marked
 *     when some i of S1 has |c_i - c_j| + rad_i <= dthr and
 *     |c_j - c_i| + rad_j <= dthr / 2, where c is the group centroid and
 *     rad_g = max over the members x of g of |x - c_g|.
 * Readings: only non-empty groups take part (an empty group has radius 0, is
 * never marked and is never a partner); partner_j = the lowest such i (-1 if
 * none, and -1 for every group of S1); merges = number of marked groups.
 * Evaluation: squared distances by canon_dist2, radius = sqrt of the largest
 * squared member distance, qmax = sqrt of the largest squared query norm,
 * R' = |scale| * qmax, dthr = log_eps / (2 * R'), sums in fp64.
 *   Q, K [B,H,n,d] doubles; belong [B,H,n]; centroid [B,H,N,d] floats;
 *   count [B,H,N].  Out: radius [B,H,N], dthr [B,H], partner [B,H,N],
 *   merges [B,H].
 */
void ga_oracle_merge_plan(int B, int H, int n, int d, const double *Q, const double *K,
                          const int32_t *belong, const float *centroid, const int32_t *count, int N,
                          double scale, double log_eps, double *radius, double *dthr,
                          int32_t *partner, int32_t *merges) {
    const int64_t BH = (int64_t)B * H;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t u = 0; u < BH; ++u) {
        double *C = (double *)malloc(sizeof(double) * (size_t)N * d);
        double *rad2 = (double *)calloc((size_t)N, sizeof(double));
        const int32_t *cnt = count + u * (int64_t)N;
        for (int64_t x = 0; x < (int64_t)N * d; ++x) C[x] = (double)centroid[u * (int64_t)N * d + x];
        double qmax2 = 0.0;
        for (int i = 0; i < n; ++i) {
            const double *q = Q + (u * (int64_t)n + i) * d;
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc = fma(q[c], q[c], acc);
            if (acc > qmax2) qmax2 = acc;
            const int g = belong[u * (int64_t)n + i];
            if (g < 0 || g >= N) continue;
            const double r2 = canon_dist2(K + (u * (int64_t)n + i) * d, C + (size_t)g * d, d);
            if (r2 > rad2[g]) rad2[g] = r2;
        }
        const double rprime = fabs(scale) * sqrt(qmax2);
        const double t = log_eps / (2.0 * rprime);
        dthr[u] = t;
        int32_t marked = 0;
        const int half = (N + 1) / 2;
        for (int j = 0; j < N; ++j) radius[u * (int64_t)N + j] = sqrt(rad2[j]);
        for (int j = 0; j < N; ++j) {
            int32_t pj = -1;
            if (j >= half && cnt[j] > 0) {
                const double rj = sqrt(rad2[j]);
                for (int i = 0; i < half; ++i) {
                    if (cnt[i] <= 0) continue;
                    const double dij = sqrt(canon_dist2(C + (size_t)i * d, C + (size_t)j * d, d));
                    if (dij + sqrt(rad2[i]) <= t && dij + rj <= 0.5 * t) {
                        pj = i;
                        break;
                    }
                }
            }
            partner[u * (int64_t)N + j] = pj;
            marked += pj >= 0;
        }
        merges[u] = marked;
        free(C);
        free(rad2);
    }
}
