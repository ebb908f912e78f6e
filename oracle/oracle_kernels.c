/*
 * CPU oracle for the tensor kernels whose schedules are tuned.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or constant with the HIP library and must never be reached from the
 * product path.
 *
 * The paper (Section 1 and Definition 1) treats a kernel as operations on
 * tensors indexed by linear combinations of naturals; the evaluation tunes
 * ONNX models whose hot kernels are conv2d and matmul/dense (Section 3, RQ6).
 * The paper does not spell out their semantics, so the reading taken here is
 * the ONNX / TVM "conv2d_nchw" definition:
 *
 *   P = floor((H + 2*pad - R) / stride) + 1,  Q = floor((W + 2*pad - S) / stride) + 1
 *   y[n,k,p,q] = sum_{c<C} sum_{r<R} sum_{s<S}
 *                x[n, c, p*stride - pad + r, q*stride - pad + s] * w[k,c,r,s]
 *
 * with out-of-range input positions contributing zero (cross-correlation, no
 * flip, dilation 1, one group, no bias), and for matmul
 *
 *   C[i,j] = sum_{l<K} A[i,l] * B[l,j]     (row-major, C overwritten).
 *
 * Every product of two fp32 values is exact in fp64, and the sums are taken
 * in fp64 in the plain loop order below, so the result is the exact value up
 * to fp64 rounding of at most C*R*S (or K) terms.
 *
 * Build: gcc -O3 -fopenmp -fPIC -shared (no fast-math).
 */
#include <stdint.h>
#include <stdlib.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)

static int conv_dims(const int64_t *sh, int64_t *P, int64_t *Q) {
    int64_t N = sh[0], C = sh[1], H = sh[2], W = sh[3], K = sh[4], R = sh[5], S = sh[6],
            st = sh[7], pd = sh[8];
    if (N < 0 || C < 0 || H < 0 || W < 0 || K < 0 || R < 1 || S < 1 || st < 1 || pd < 0)
        return ORACLE_EINVAL;
    if (H + 2 * pd < R || W + 2 * pd < S) return ORACLE_EINVAL;
    *P = (H + 2 * pd - R) / st + 1;
    *Q = (W + 2 * pd - S) / st + 1;
    return ORACLE_OK;
}

/* Output spatial size; returns ORACLE_EINVAL for a shape with no output. */
int oracle_conv2d_out(const int64_t *shape9, int64_t *P, int64_t *Q) {
    return conv_dims(shape9, P, Q);
}

/* Full direct convolution.  x: [N,C,H,W] fp32, w: [K,C,R,S] fp32,
 * y: [N,K,P,Q] fp64 (overwritten).  Parallel over the (n,k) output planes. */
int oracle_conv2d_f64(const float *x, const float *w, double *y, const int64_t *shape9) {
    int64_t P, Q;
    if (conv_dims(shape9, &P, &Q) != ORACLE_OK) return ORACLE_EINVAL;
    const int64_t N = shape9[0], C = shape9[1], H = shape9[2], W = shape9[3], K = shape9[4],
                  R = shape9[5], S = shape9[6], st = shape9[7], pd = shape9[8];
    int64_t nk;
#pragma omp parallel for schedule(dynamic, 1)
    for (nk = 0; nk < N * K; ++nk) {
        const int64_t n = nk / K, k = nk % K;
        double *yp = y + nk * P * Q;
        for (int64_t i = 0; i < P * Q; ++i) yp[i] = 0.0;
        for (int64_t c = 0; c < C; ++c) {
            const float *xp = x + (n * C + c) * H * W;
            for (int64_t r = 0; r < R; ++r) {
                for (int64_t s = 0; s < S; ++s) {
                    const double wv = (double)w[((k * C + c) * R + r) * S + s];
                    for (int64_t p = 0; p < P; ++p) {
                        const int64_t iy = p * st - pd + r;
                        if (iy < 0 || iy >= H) continue;
                        for (int64_t q = 0; q < Q; ++q) {
                            const int64_t ix = q * st - pd + s;
                            if (ix < 0 || ix >= W) continue;
                            yp[p * Q + q] += (double)xp[iy * W + ix] * wv;
                        }
                    }
                }
            }
        }
    }
    return ORACLE_OK;
}

/* The same sum, one output at a time, for a list of flat output indices
 * (idx = ((n*K + k)*P + p)*Q + q).  Used to check very large outputs on a
 * sample of positions. */
int oracle_conv2d_f64_points(const float *x, const float *w, const int64_t *shape9,
                             const int64_t *idx, int64_t npts, double *out) {
    int64_t P, Q;
    if (conv_dims(shape9, &P, &Q) != ORACLE_OK) return ORACLE_EINVAL;
    const int64_t N = shape9[0], C = shape9[1], H = shape9[2], W = shape9[3], K = shape9[4],
                  R = shape9[5], S = shape9[6], st = shape9[7], pd = shape9[8];
    int64_t t;
    for (t = 0; t < npts; ++t)
        if (idx[t] < 0 || idx[t] >= N * K * P * Q) return ORACLE_EINVAL;
#pragma omp parallel for schedule(static)
    for (t = 0; t < npts; ++t) {
        int64_t f = idx[t];
        const int64_t q = f % Q; f /= Q;
        const int64_t p = f % P; f /= P;
        const int64_t k = f % K;
        const int64_t n = f / K;
        double acc = 0.0;
        for (int64_t c = 0; c < C; ++c)
            for (int64_t r = 0; r < R; ++r) {
                const int64_t iy = p * st - pd + r;
                if (iy < 0 || iy >= H) continue;
                for (int64_t s = 0; s < S; ++s) {
                    const int64_t ix = q * st - pd + s;
                    if (ix < 0 || ix >= W) continue;
                    acc += (double)x[((n * C + c) * H + iy) * W + ix] *
                           (double)w[((k * C + c) * R + r) * S + s];
                }
            }
        out[t] = acc;
    }
    return ORACLE_OK;
}

/* C[M,N] = A[M,K] * B[K,N], all row-major; inputs fp32, output fp64. */
int oracle_matmul_f64(const float *A, const float *B, double *Cm, int64_t M, int64_t N,
                      int64_t K) {
    if (M < 0 || N < 0 || K < 0) return ORACLE_EINVAL;
    int64_t i;
#pragma omp parallel for schedule(dynamic, 1)
    for (i = 0; i < M; ++i) {
        double *cp = Cm + i * N;
        for (int64_t j = 0; j < N; ++j) cp[j] = 0.0;
        for (int64_t l = 0; l < K; ++l) {
            const double a = (double)A[i * K + l];
            const float *bp = B + l * N;
            for (int64_t j = 0; j < N; ++j) cp[j] += a * (double)bp[j];
        }
    }
    return ORACLE_OK;
}

/* Matmul outputs at flat indices idx = i*N + j. */
int oracle_matmul_f64_points(const float *A, const float *B, int64_t M, int64_t N, int64_t K,
                             const int64_t *idx, int64_t npts, double *out) {
    if (M < 0 || N < 0 || K < 0) return ORACLE_EINVAL;
    int64_t t;
    for (t = 0; t < npts; ++t)
        if (idx[t] < 0 || idx[t] >= M * N) return ORACLE_EINVAL;
#pragma omp parallel for schedule(static)
    for (t = 0; t < npts; ++t) {
        const int64_t i = idx[t] / N, j = idx[t] % N;
        double acc = 0.0;
        for (int64_t l = 0; l < K; ++l) acc += (double)A[i * K + l] * (double)B[l * N + j];
        out[t] = acc;
    }
    return ORACLE_OK;
}

/* Number of OpenMP threads a parallel region of this library would use. */
int oracle_num_threads(void) {
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
