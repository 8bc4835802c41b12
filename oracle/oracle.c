/*
 * Plain CPU oracle for the three convolution passes of a 2-D convolutional
 * layer (Dryden et al., "Improving Strong-Scaling of CNN Training by
 * Exploiting Finer-Grained Parallelism", Sec. II-A, Eqs. (1)-(3)).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the GPU path.
 *
 * Notation (paper -> here): N samples, C channels, F filters -> K,
 * filter K x K -> R x S, stride S -> stride, padding P -> pad.
 *
 * The paper states Eqs. (1)-(3) for stride 1 and output-preserving padding
 * and notes that neither assumption matters to the method.  The general form
 * used here is the one those equations reduce to at stride 1,
 * pad = floor(K/2):
 *
 *   y [n,k,p,q] = sum_c sum_r sum_s  X(n,c, p*stride-pad+r, q*stride-pad+s) * w[k,c,r,s]
 *   dx[n,c,i,j] = sum_k sum_r sum_s  DY(n,k, (i+pad-r)/stride, (j+pad-s)/stride) * w[k,c,r,s]
 *                 (a term exists only where both divisions are exact)
 *   dw[k,c,r,s] = sum_n sum_p sum_q  dy[n,k,p,q] * X(n,c, p*stride-pad+r, q*stride-pad+s)
 *
 * X and DY read zero outside the tensor (Sec. II-A leaves subscripts outside
 * the tensor to the padding).  There is no filter flip (Eq. (1) pairs x at
 * offset +a with w at a+O) and no bias.
 *
 * Arithmetic: inputs are fp32 arrays (bf16 inputs arrive already widened,
 * exactly, to fp32).  Every product of two such values is exact in fp64, and
 * each output is accumulated in one fp64 variable in a fixed order -- (c,r,s)
 * for y, (k,r,s) for dx, (n,p,q) for dw -- and returned in fp64.  The caller
 * rounds to fp32.  OpenMP splits only the outermost independent output loops,
 * so results do not depend on the thread count.
 *
 * All tensors are dense, row-major: x [N][C][Hi][Wi], w [K][C][R][S],
 * y and dy [N][K][Ho][Wo], dx [N][C][Hi][Wi], dw [K][C][R][S].
 */
#include <stdint.h>
#include <stddef.h>
#include <omp.h>

typedef int64_t i64;

static double x_at(const float* x, i64 C, i64 Hi, i64 Wi, i64 n, i64 c, i64 i, i64 j)
{
    if (i < 0 || i >= Hi || j < 0 || j >= Wi) return 0.0;  /* zero padding */
    return (double)x[((n * C + c) * Hi + i) * Wi + j];
}

/* One output of Eq. (1), generalised to stride/pad. */
static double fwd_one(const float* x, const float* w, i64 C, i64 Hi, i64 Wi,
                      i64 R, i64 S, i64 stride, i64 pad,
                      i64 n, i64 k, i64 p, i64 q)
{
    double acc = 0.0;
    for (i64 c = 0; c < C; ++c)
        for (i64 r = 0; r < R; ++r)
            for (i64 s = 0; s < S; ++s)
                acc += x_at(x, C, Hi, Wi, n, c, p * stride - pad + r, q * stride - pad + s)
                     * (double)w[((k * C + c) * R + r) * S + s];
    return acc;
}

/* One output of Eq. (3): gather form of the input gradient. */
static double bwd_data_one(const float* dy, const float* w, i64 C, i64 K,
                           i64 Ho, i64 Wo, i64 R, i64 S, i64 stride, i64 pad,
                           i64 n, i64 c, i64 i, i64 j)
{
    double acc = 0.0;
    for (i64 k = 0; k < K; ++k)
        for (i64 r = 0; r < R; ++r)
            for (i64 s = 0; s < S; ++s) {
                i64 ti = i + pad - r, tj = j + pad - s;
                if (ti < 0 || tj < 0) continue;
                if (ti % stride != 0 || tj % stride != 0) continue;
                i64 p = ti / stride, q = tj / stride;
                if (p >= Ho || q >= Wo) continue;
                acc += (double)dy[((n * K + k) * Ho + p) * Wo + q]
                     * (double)w[((k * C + c) * R + r) * S + s];
            }
    return acc;
}

/* One output of Eq. (2): the weight gradient summed over samples and pixels. */
static double bwd_filter_one(const float* x, const float* dy, i64 N, i64 C, i64 K,
                             i64 Hi, i64 Wi, i64 Ho, i64 Wo, i64 stride, i64 pad,
                             i64 k, i64 c, i64 r, i64 s)
{
    double acc = 0.0;
    for (i64 n = 0; n < N; ++n)
        for (i64 p = 0; p < Ho; ++p)
            for (i64 q = 0; q < Wo; ++q)
                acc += (double)dy[((n * K + k) * Ho + p) * Wo + q]
                     * x_at(x, C, Hi, Wi, n, c, p * stride - pad + r, q * stride - pad + s);
    return acc;
}

/* ---------------- whole-tensor entry points ---------------- */

void oracle_conv_fwd(i64 N, i64 C, i64 K, i64 Hi, i64 Wi, i64 Ho, i64 Wo,
                     i64 R, i64 S, i64 stride, i64 pad,
                     const float* x, const float* w, double* y)
{
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (i64 n = 0; n < N; ++n)
        for (i64 k = 0; k < K; ++k)
            for (i64 p = 0; p < Ho; ++p)
                for (i64 q = 0; q < Wo; ++q)
                    y[((n * K + k) * Ho + p) * Wo + q] =
                        fwd_one(x, w, C, Hi, Wi, R, S, stride, pad, n, k, p, q);
}

void oracle_conv_bwd_data(i64 N, i64 C, i64 K, i64 Hi, i64 Wi, i64 Ho, i64 Wo,
                          i64 R, i64 S, i64 stride, i64 pad,
                          const float* dy, const float* w, double* dx)
{
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (i64 n = 0; n < N; ++n)
        for (i64 c = 0; c < C; ++c)
            for (i64 i = 0; i < Hi; ++i)
                for (i64 j = 0; j < Wi; ++j)
                    dx[((n * C + c) * Hi + i) * Wi + j] =
                        bwd_data_one(dy, w, C, K, Ho, Wo, R, S, stride, pad, n, c, i, j);
}

void oracle_conv_bwd_filter(i64 N, i64 C, i64 K, i64 Hi, i64 Wi, i64 Ho, i64 Wo,
                            i64 R, i64 S, i64 stride, i64 pad,
                            const float* x, const float* dy, double* dw)
{
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (i64 k = 0; k < K; ++k)
        for (i64 c = 0; c < C; ++c)
            for (i64 r = 0; r < R; ++r)
                for (i64 s = 0; s < S; ++s)
                    dw[((k * C + c) * R + r) * S + s] =
                        bwd_filter_one(x, dy, N, C, K, Hi, Wi, Ho, Wo, stride, pad, k, c, r, s);
}

/* ---------------- sampled entry points ----------------
 * idx[t] is the flat row-major index of the t-th requested output element in
 * the corresponding output tensor; out[t] receives its fp64 value.  Used where
 * the full output would take the oracle too long. */

void oracle_conv_fwd_points(i64 N, i64 C, i64 K, i64 Hi, i64 Wi, i64 Ho, i64 Wo,
                            i64 R, i64 S, i64 stride, i64 pad,
                            const float* x, const float* w,
                            const i64* idx, i64 count, double* out)
{
    (void)N;
    #pragma omp parallel for schedule(dynamic)
    for (i64 t = 0; t < count; ++t) {
        i64 f = idx[t];
        i64 q = f % Wo; f /= Wo;
        i64 p = f % Ho; f /= Ho;
        i64 k = f % K;  f /= K;
        out[t] = fwd_one(x, w, C, Hi, Wi, R, S, stride, pad, f, k, p, q);
    }
}

void oracle_conv_bwd_data_points(i64 N, i64 C, i64 K, i64 Hi, i64 Wi, i64 Ho, i64 Wo,
                                 i64 R, i64 S, i64 stride, i64 pad,
                                 const float* dy, const float* w,
                                 const i64* idx, i64 count, double* out)
{
    (void)N;
    #pragma omp parallel for schedule(dynamic)
    for (i64 t = 0; t < count; ++t) {
        i64 f = idx[t];
        i64 j = f % Wi; f /= Wi;
        i64 i = f % Hi; f /= Hi;
        i64 c = f % C;  f /= C;
        out[t] = bwd_data_one(dy, w, C, K, Ho, Wo, R, S, stride, pad, f, c, i, j);
    }
}

void oracle_conv_bwd_filter_points(i64 N, i64 C, i64 K, i64 Hi, i64 Wi, i64 Ho, i64 Wo,
                                   i64 R, i64 S, i64 stride, i64 pad,
                                   const float* x, const float* dy,
                                   const i64* idx, i64 count, double* out)
{
    #pragma omp parallel for schedule(dynamic)
    for (i64 t = 0; t < count; ++t) {
        i64 f = idx[t];
        i64 s = f % S; f /= S;
        i64 r = f % R; f /= R;
        i64 c = f % C; f /= C;
        out[t] = bwd_filter_one(x, dy, N, C, K, Hi, Wi, Ho, Wo, stride, pad, f, c, r, s);
    }
}

/* Threads the OpenMP loops above use (for reporting timings). */
int oracle_num_threads(void) { return omp_get_max_threads(); }

/* Run the loops above on n threads from now on (timing at one thread). */
void oracle_set_num_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
