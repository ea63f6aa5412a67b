/*
 * kmeans_oracle.c -- plain, slow fp64 CPU oracle of exact k-means (Lloyd).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It shares no code with the
 * HIP path: no headers, helpers or tables.
 *
 * What it computes (paper Section 5, "Flash-KMeans clean-start workload"):
 * one Lloyd iteration is an assignment step, which finds for every point the
 * centroid at the smallest squared Euclidean distance (an arg-min over the K
 * centroids), followed by a centroid update, which reduces the points of each
 * cluster into a per-cluster sum and count and divides.  The method is exact
 * k-means, so this file writes the textbook definition out directly:
 *
 *   d_ik      = sum_j (x_ij - c_kj)^2            direct form, j ascending, fp64
 *   idx_i     = smallest k with d_ik minimal     (ties -> lowest index)
 *   min_dist_i= d_i,idx_i
 *   gap_i     = second smallest d_ik over k != idx_i, minus min_dist_i
 *   n_k       = #{i : idx_i = k},  S_k = sum_{i: idx_i = k} x_i  (i ascending)
 *   c'_k      = S_k / n_k if n_k > 0, else c_k   (an empty cluster keeps its centroid)
 *   J_t       = sum_i min_dist_i                 (i ascending, fp64)
 *
 * Points are read as stored (fp32, bf16 or fp16 bits) and widened exactly to
 * fp64; centroids are passed in fp64.  B independent instances are laid out
 * back to back ([B,N,D] points, [B,K,D] centroids).
 *
 * Readings where the paper is silent: ties go to the lowest index; an empty
 * cluster keeps its previous centroid; J_t is the objective of the assignment
 * made under C_t, before that iteration's update.
 *
 * Values that are not finite (the paper does not treat them): a point with a
 * NaN or infinite coordinate is left unassigned (idx -1, min_dist and gap
 * NaN); a centroid with one is never chosen, and a point with no centroid
 * left is unassigned too.  The update counts and sums only points whose idx
 * is in [0, K); J_t sums the assigned points' min_dist.
 *
 * KNN search (the same distance with a top-k instead of an arg-min; the paper
 * lists KNN build and search beside KMeans in Section 6 and reports recall
 * 1.0): for query q and database rows r_j,
 *
 *   e_j       = sum_l (q_l - r_jl)^2             direct form, l ascending, fp64
 *   nbr       = the k smallest e_j in increasing order, ties -> lowest j
 *   next_dist = the (k+1)-th smallest e_j (+inf when k == N)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F16 = 2 };
enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_ENOMEM = -2 };

/* bfloat16: the upper half of an IEEE binary32. */
static double widen_bf16(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double widen_f16(uint16_t h) {
    int s = h >> 15, e = (h >> 10) & 0x1f, m = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);                 /* subnormal: m * 2^-14 * 2^-10 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + m), e - 25);     /* (1 + m/1024) * 2^(e-15) */
    return s ? -v : v;
}

static double widen_one(const void* src, int dtype, int64_t i) {
    if (dtype == ORC_F32) return (double)((const float*)src)[i];
    if (dtype == ORC_BF16) return widen_bf16(((const uint16_t*)src)[i]);
    return widen_f16(((const uint16_t*)src)[i]);
}

static int dtype_ok(int dtype) { return dtype == ORC_F32 || dtype == ORC_BF16 || dtype == ORC_F16; }

/* Exact widening of n stored values to fp64. */
int oracle_widen(const void* src, int dtype, int64_t n, double* dst) {
    if (!src || !dst || n < 0 || !dtype_ok(dtype)) return ORC_EINVAL;
    for (int64_t i = 0; i < n; ++i) dst[i] = widen_one(src, dtype, i);
    return ORC_OK;
}

static int all_finite(const double* v, int64_t n) {
    for (int64_t j = 0; j < n; ++j)
        if (!isfinite(v[j])) return 0;
    return 1;
}

/* Assignment step for B instances.  gap may be NULL; for K == 1 (one usable
 * centroid) it is +inf. */
int oracle_assign(const void* X, int dtype, const double* C, int64_t B, int64_t N,
                  int64_t D, int64_t K, int32_t* idx, double* min_dist, double* gap) {
    if (!X || !C || !idx || !min_dist || !dtype_ok(dtype) || B < 1 || N < 0 || D < 1 || K < 1)
        return ORC_EINVAL;
    char* usable = (char*)malloc((size_t)K);
    if (!usable) return ORC_ENOMEM;
    int err = ORC_OK;
    for (int64_t b = 0; b < B; ++b) {
        const double* Cb = C + b * K * D;
        for (int64_t k = 0; k < K; ++k) usable[k] = (char)all_finite(Cb + k * D, D);
#pragma omp parallel
        {
            double* x = (double*)malloc((size_t)D * sizeof(double));
            if (!x) {
#pragma omp atomic write
                err = ORC_ENOMEM;
            }
#pragma omp for schedule(static)
            for (int64_t i = 0; i < N; ++i) {
                if (!x) continue;
                const int64_t row = b * N + i;
                for (int64_t j = 0; j < D; ++j) x[j] = widen_one(X, dtype, row * D + j);
                double best = INFINITY, second = INFINITY;
                int64_t arg = -1;
                const int point_ok = all_finite(x, D);
                for (int64_t k = 0; k < K && point_ok; ++k) {
                    if (!usable[k]) continue;
                    const double* c = Cb + k * D;
                    double d = 0.0;
                    for (int64_t j = 0; j < D; ++j) {
                        const double t = x[j] - c[j];
                        d += t * t;
                    }
                    if (arg < 0 || d < best) {
                        second = best;
                        best = d;
                        arg = k;
                    } else if (d < second) {
                        second = d;
                    }
                }
                idx[row] = (int32_t)arg;
                min_dist[row] = arg < 0 ? NAN : best;
                if (gap) gap[row] = arg < 0 ? NAN : second - best;
            }
            free(x);
        }
    }
    free(usable);
    return err;
}

/* Update step: per-cluster counts and means over the points with idx in
 * [0, K); empty clusters keep C_prev. */
int oracle_update(const void* X, int dtype, const int32_t* idx, const double* C_prev,
                  int64_t B, int64_t N, int64_t D, int64_t K, double* C_out, int64_t* counts) {
    if (!X || !idx || !C_prev || !C_out || !counts || !dtype_ok(dtype) || B < 1 || N < 0 ||
        D < 1 || K < 1)
        return ORC_EINVAL;
    double* S = (double*)calloc((size_t)(K * D), sizeof(double));
    if (!S) return ORC_ENOMEM;
    int err = ORC_OK;
    for (int64_t b = 0; b < B && err == ORC_OK; ++b) {
        memset(S, 0, (size_t)(K * D) * sizeof(double));
        int64_t* n = counts + b * K;
        for (int64_t k = 0; k < K; ++k) n[k] = 0;
        for (int64_t i = 0; i < N; ++i) {
            const int64_t row = b * N + i;
            const int32_t k = idx[row];
            if (k < 0 || k >= K) continue;
            n[k] += 1;
            for (int64_t j = 0; j < D; ++j) S[k * D + j] += widen_one(X, dtype, row * D + j);
        }
        for (int64_t k = 0; k < K; ++k) {
            double* out = C_out + (b * K + k) * D;
            const double* prev = C_prev + (b * K + k) * D;
            for (int64_t j = 0; j < D; ++j)
                out[j] = n[k] > 0 ? S[k * D + j] / (double)n[k] : prev[j];
        }
    }
    free(S);
    return err;
}

/*
 * T Lloyd iterations from C0.  Outputs: C_T (C_out), and idx, min_dist and
 * counts of the last iteration; objective[b*iters + t] = J_t of instance b.
 */
int oracle_lloyd(const void* X, int dtype, const double* C0, int64_t B, int64_t N, int64_t D,
                 int64_t K, int iters, double* C_out, int32_t* idx, double* min_dist,
                 int64_t* counts, double* objective) {
    if (!C0 || !C_out || iters < 1) return ORC_EINVAL;
    double* C = (double*)malloc((size_t)(B * K * D) * sizeof(double));
    if (!C) return ORC_ENOMEM;
    memcpy(C, C0, (size_t)(B * K * D) * sizeof(double));
    int err = ORC_OK;
    for (int t = 0; t < iters && err == ORC_OK; ++t) {
        err = oracle_assign(X, dtype, C, B, N, D, K, idx, min_dist, NULL);
        if (err) break;
        if (objective)
            for (int64_t b = 0; b < B; ++b) {
                double J = 0.0;
                for (int64_t i = 0; i < N; ++i)
                    if (idx[b * N + i] >= 0) J += min_dist[b * N + i];
                objective[b * iters + t] = J;
            }
        err = oracle_update(X, dtype, idx, C, B, N, D, K, C_out, counts);
        memcpy(C, C_out, (size_t)(B * K * D) * sizeof(double));
    }
    free(C);
    return err;
}

/*
 * KNN search for B instances: queries Q [B,M,D] and database R [B,N,D], both
 * stored in `dtype`.  nbr_idx / nbr_dist [B,M,k]; next_dist [B,M] may be NULL.
 * Each query keeps its k + 1 smallest distances by insertion into a list
 * ordered by (distance, index).
 */
int oracle_knn(const void* Q, const void* R, int dtype, int64_t B, int64_t M, int64_t N,
               int64_t D, int64_t k, int32_t* nbr_idx, double* nbr_dist, double* next_dist) {
    if (!Q || !R || !nbr_idx || !nbr_dist || !dtype_ok(dtype) || B < 1 || M < 0 || N < 1 ||
        D < 1 || k < 1 || k > N)
        return ORC_EINVAL;
    double* rw = (double*)malloc((size_t)(N * D) * sizeof(double));
    if (!rw) return ORC_ENOMEM;
    int err = ORC_OK;
    for (int64_t b = 0; b < B && err == ORC_OK; ++b) {
        for (int64_t j = 0; j < N * D; ++j) rw[j] = widen_one(R, dtype, b * N * D + j);
#pragma omp parallel
        {
            double* q = (double*)malloc((size_t)D * sizeof(double));
            double* ld = (double*)malloc((size_t)(k + 1) * sizeof(double));
            int64_t* li = (int64_t*)malloc((size_t)(k + 1) * sizeof(int64_t));
            if (!q || !ld || !li) {
#pragma omp atomic write
                err = ORC_ENOMEM;
            }
#pragma omp for schedule(static)
            for (int64_t i = 0; i < M; ++i) {
                if (!q || !ld || !li) continue;
                const int64_t row = b * M + i;
                for (int64_t l = 0; l < D; ++l) q[l] = widen_one(Q, dtype, row * D + l);
                int64_t n = 0;  /* entries in the list, at most k + 1 */
                for (int64_t j = 0; j < N; ++j) {
                    const double* r = rw + j * D;
                    double e = 0.0;
                    for (int64_t l = 0; l < D; ++l) {
                        const double t = q[l] - r[l];
                        e += t * t;
                    }
                    /* j ascending: an equal distance goes after the entries already there */
                    if (n == k + 1 && !(e < ld[k])) continue;
                    int64_t pos = n < k + 1 ? n : k;
                    while (pos > 0 && e < ld[pos - 1]) {
                        ld[pos] = ld[pos - 1];
                        li[pos] = li[pos - 1];
                        --pos;
                    }
                    ld[pos] = e;
                    li[pos] = j;
                    if (n < k + 1) ++n;
                }
                for (int64_t t = 0; t < k; ++t) {
                    nbr_idx[row * k + t] = (int32_t)li[t];
                    nbr_dist[row * k + t] = ld[t];
                }
                if (next_dist) next_dist[row] = n > k ? ld[k] : INFINITY;
            }
            free(q);
            free(ld);
            free(li);
        }
    }
    free(rw);
    return err;
}
