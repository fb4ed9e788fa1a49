/*
 * CPU oracle for the per-token topic draw -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * use this file.  It shares no code, header or constant with the HIP library.
 *
 * What it computes is the plain definition of the draw (Section 2 of the
 * paper, Algorithm 1 with the search of Algorithms 2/3), in fp64:
 *   a_k  = theta[d][k] * phi[w][k]       exact in fp64 for fp32 inputs
 *   S_k  = a_0 + ... + a_k               sequential fp64 sum (Algorithm 1)
 *   stop = u * S_{K-1}                   scaled uniform (Algorithms 2/3)
 *   z    = min { k : stop < S_k }        strict "<", smallest index on ties
 *   z    = K - 1 if no k qualifies       what the linear and binary searches
 *                                        return when the loop runs off the end
 * in_band marks tokens where |stop - S_k| <= band_rel * S_{K-1} for some k:
 * there an fp32 evaluation of the same definition may legitimately land on a
 * neighbouring topic.
 *
 * It also counts a set of draws (oracle_counts): the per-document and
 * per-word topic counts that the update of theta and phi consumes once every
 * z has been drawn (Section 1: draw z for each word, then update theta and
 * phi; Section 2: the uncollapsed sampler).  Integer work, exact.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads for the following draws (n >= 1); the arithmetic is unchanged. */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* S[k] = sum_{i<=k} theta[d][i] * phi[w][i], sequential, fp64. */
void oracle_prefix(const float *theta_row, const float *phi_row, int32_t K,
                   double *S)
{
    double run = 0.0;
    for (int32_t k = 0; k < K; ++k) {
        run += (double)theta_row[k] * (double)phi_row[k];
        S[k] = run;
    }
}

/* The smallest k with stop < S[k]; K - 1 if there is none. */
int32_t oracle_search(const double *S, int32_t K, double stop)
{
    for (int32_t k = 0; k < K; ++k)
        if (stop < S[k])
            return k;
    return K - 1;
}

/*
 * z[n] for every token.  theta is [M][K] and phi is [V][K], row-major.
 * in_band may be NULL; otherwise it receives 1 for tokens inside the
 * rounding band and 0 elsewhere.  Returns 0, or -1 if scratch allocation
 * failed.  Ids are not range-checked: callers pass valid ids.
 */
int oracle_draw(const float *theta, const float *phi, const int32_t *doc_id,
                const int32_t *word_id, const float *u, int64_t N, int32_t K,
                int32_t *z, uint8_t *in_band, double band_rel)
{
    int failed = 0;
#pragma omp parallel
    {
        double *S = (double *)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
        if (!S) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            if (!S)
                continue;
            const float *th = theta + (int64_t)doc_id[n] * K;
            const float *ph = phi + (int64_t)word_id[n] * K;
            oracle_prefix(th, ph, K, S);
            const double total = S[K - 1];
            const double stop = (double)u[n] * total;
            z[n] = oracle_search(S, K, stop);
            if (in_band) {
                uint8_t band = 0;
                for (int32_t k = 0; k < K; ++k)
                    if (fabs(stop - S[k]) <= band_rel * total) {
                        band = 1;
                        break;
                    }
                in_band[n] = band;
            }
        }
        free(S);
    }
    return failed ? -1 : 0;
}

/*
 * Topic counts of the draws z[0..N): every token n with 0 <= doc_id[n] < M,
 * 0 <= word_id[n] < V and 0 <= z[n] < K adds one to ndk[doc_id[n]][z[n]] and
 * one to nwk[word_id[n]][z[n]]; tokens with an id or topic out of range are
 * not counted.  ndk is [M][K] and nwk is [V][K] (word-major, the layout of
 * phi), row-major int32, and are overwritten (zeroed first).  One sequential
 * pass in token order.  Returns the number of tokens counted.
 */
int64_t oracle_counts(const int32_t *doc_id, const int32_t *word_id,
                      const int32_t *z, int64_t N, int32_t M, int32_t V,
                      int32_t K, int32_t *ndk, int32_t *nwk)
{
    memset(ndk, 0, sizeof(int32_t) * (size_t)M * (size_t)K);
    memset(nwk, 0, sizeof(int32_t) * (size_t)V * (size_t)K);
    int64_t counted = 0;
    for (int64_t n = 0; n < N; ++n) {
        const int32_t d = doc_id[n], w = word_id[n], k = z[n];
        if (d < 0 || d >= M || w < 0 || w >= V || k < 0 || k >= K)
            continue;
        ndk[(int64_t)d * K + k] += 1;
        nwk[(int64_t)w * K + k] += 1;
        ++counted;
    }
    return counted;
}
