/*
 * Runs the oracle's whole-tensor and sampled-point entry points over seeded
 * random small layers (strides 1-3, pads 0-2, filters 1-5, R != S) under
 * AddressSanitizer / UndefinedBehaviorSanitizer, and checks that every
 * sampled point equals the whole-tensor value.  Exit 0 on success.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef int64_t i64;
void oracle_conv_fwd(i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, const float*, const float*, double*);
void oracle_conv_bwd_data(i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, const float*, const float*, double*);
void oracle_conv_bwd_filter(i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, const float*, const float*, double*);
void oracle_conv_fwd_points(i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, const float*, const float*,
                            const i64*, i64, double*);
void oracle_conv_bwd_data_points(i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, const float*,
                                 const float*, const i64*, i64, double*);
void oracle_conv_bwd_filter_points(i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, i64, const float*,
                                   const float*, const i64*, i64, double*);

static uint64_t rs = 0x2545f4914f6cdd1dull;
static i64 rnd(i64 n) { rs ^= rs << 13; rs ^= rs >> 7; rs ^= rs << 17; return (i64)(rs % (uint64_t)n); }
static float* fill(i64 n) { float* a = malloc((size_t)n * sizeof(float)); for (i64 i = 0; i < n; ++i) a[i] = (float)(rnd(2001) - 1000) / 1000.0f; return a; }

static int check(const double* whole, i64 n, const double* pts, const i64* idx, i64 m)
{
    for (i64 t = 0; t < m; ++t) if (idx[t] >= n || pts[t] != whole[idx[t]]) return 1;
    return 0;
}

int main(void)
{
    int bad = 0, runs = 0;
    for (int it = 0; it < 300; ++it) {
        const i64 N = 1 + rnd(2), C = 1 + rnd(3), K = 1 + rnd(3), H = 3 + rnd(7), W = 3 + rnd(7);
        const i64 R = 1 + rnd(5), S = rnd(3) ? R : 1 + rnd(5), st = 1 + rnd(3), pad = rnd(3);
        const i64 Ho = (H + 2 * pad - R) / st + 1, Wo = (W + 2 * pad - S) / st + 1;
        if (H + 2 * pad < R || W + 2 * pad < S || Ho < 1 || Wo < 1) continue;
        float* x = fill(N * C * H * W), * w = fill(K * C * R * S), * dy = fill(N * K * Ho * Wo);
        double* y = malloc(sizeof(double) * N * K * Ho * Wo), * dx = malloc(sizeof(double) * N * C * H * W);
        double* dw = malloc(sizeof(double) * K * C * R * S);
        oracle_conv_fwd(N, C, K, H, W, Ho, Wo, R, S, st, pad, x, w, y);
        oracle_conv_bwd_data(N, C, K, H, W, Ho, Wo, R, S, st, pad, dy, w, dx);
        oracle_conv_bwd_filter(N, C, K, H, W, Ho, Wo, R, S, st, pad, x, dy, dw);
        i64 idx[16];
        double pts[16];
        const i64 sizes[3] = {N * K * Ho * Wo, N * C * H * W, K * C * R * S};
        for (int k = 0; k < 3; ++k) {
            for (int t = 0; t < 16; ++t) idx[t] = t == 0 ? 0 : t == 1 ? sizes[k] - 1 : rnd(sizes[k]);
            if (k == 0) { oracle_conv_fwd_points(N, C, K, H, W, Ho, Wo, R, S, st, pad, x, w, idx, 16, pts); bad |= check(y, sizes[0], pts, idx, 16); }
            if (k == 1) { oracle_conv_bwd_data_points(N, C, K, H, W, Ho, Wo, R, S, st, pad, dy, w, idx, 16, pts); bad |= check(dx, sizes[1], pts, idx, 16); }
            if (k == 2) { oracle_conv_bwd_filter_points(N, C, K, H, W, Ho, Wo, R, S, st, pad, x, dy, idx, 16, pts); bad |= check(dw, sizes[2], pts, idx, 16); }
        }
        free(x); free(w); free(dy); free(y); free(dx); free(dw);
        ++runs;
    }
    printf("oracle checks: %d layers, %s\n", runs, bad ? "MISMATCH" : "ok");
    return bad || runs == 0;
}
