// Weight gradient on a padded tile (Eq. (2) of Sec. II-A restricted to the
// tile, Sec. III-A) as a GEMM whose reduction runs over output pixels:
//
//   dw[o][ci, r, s] = sum_{pixels} dy[o][pixel] * x[ci][pixel shifted by (r, s)]
//
// NCHW keeps both operands contiguous along the reduction (pixels), so no
// transpose is needed.  The pixel range of a tile is split into chunks of
// output rows; each workgroup reduces one chunk into a partial dw slice in
// the workspace, and a second kernel adds the partials in chunk order (fixed
// order, no atomics: deterministic).  Only the interior of the dy tile is
// read -- the weight gradient needs no dy halo (Sec. III-A).
//
// bf16: v_mfma_f32_32x32x16_bf16, a k-step of 16 pixels (8 per half-wave).
//       Four waves = 2 blocks of 32 filters x 2 blocks of 32 channels; each
//       wave accumulates its 32 x 32 block at every tap (r, s) of its filter
//       rows.  The 8 pixels a lane feeds for tap s start s elements into the
//       staged x row: two aligned 16-byte LDS reads give a 16-element window
//       from which every shift is cut with byte-align operations.
// fp32: v_mfma_f32_32x32x2_f32, a k-step of 2 pixels (one per half-wave);
//       columns are the flattened (ci, r, s) index in blocks of 32, and each
//       lane reads its own single x value.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.h"

namespace dc {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

static constexpr int kThreads = 256;
static constexpr int kBQ = 64;          // output columns staged per step
static constexpr int kTargetWGs = 256;  // workgroups aimed for per launch (one per CU)

union Pack8 {
    uint4 v;
    uint32_t d[4];
    uint16_t h[8];
    bf16x8 b;
};

// ---------------------------------------------------------------- planning

struct WgradGrid {
    int gy, gz;               // tap-row groups / column groups, filter/channel superblocks
    int chunks_per_tile, rows_per_chunk;
    int TRB;                  // bf16: filter rows per workgroup
};

static int bf16_trb(int S) { return std::max(1, 9 / S); }

static bool wgrad_grid(int dtype, int ntiles, int N, int C, int K, int R, int S, int Hot,
                       WgradGrid* g) {
    if (dtype == 1) {
        if (S > 7) return false;
        g->TRB = std::min(bf16_trb(S), R);
        g->gy = (R + g->TRB - 1) / g->TRB;
        g->gz = ((K + 63) / 64) * ((C + 63) / 64);
    } else {
        const int NCB = (C * R * S + 31) / 32;
        g->TRB = R;
        g->gy = (NCB + 7) / 8;   // 4 waves x 2 column blocks per workgroup
        g->gz = (K + 63) / 64;
    }
    const int rows = N * Hot;
    int want = std::max(1, kTargetWGs / (g->gy * g->gz));
    int cpt = std::max(1, std::min(rows, (want + ntiles - 1) / ntiles));
    g->rows_per_chunk = (rows + cpt - 1) / cpt;
    g->chunks_per_tile = (rows + g->rows_per_chunk - 1) / g->rows_per_chunk;
    return true;
}

size_t wgrad_workspace_bytes(int dtype, int ntiles, int N, int C, int K, int R, int S,
                             int Hot, int Wot) {
    (void)Wot;
    WgradGrid g;
    if (!wgrad_grid(dtype, ntiles, N, C, K, R, S, Hot, &g)) return 0;
    return size_t(ntiles) * g.chunks_per_tile * size_t(K) * C * R * S * sizeof(float);
}

__host__ __device__ inline int bf16_xwp(int istr, int S) {
    int xw = (kBQ - 1) * istr + S;
    xw = xw > kBQ + 8 ? xw : kBQ + 8;
    return (xw + 7) / 8 * 8;
}
// stride between channel planes (elements): an odd number of 16-byte units
__host__ __device__ inline int odd16(int elems) {
    int u = (elems + 7) / 8;
    if ((u & 1) == 0) ++u;
    return u * 8;
}
static constexpr int kDyP = 72;   // staged dy row pitch (bf16): 9 x 16 bytes

bool wgrad_plan(WgradArgs& a, int dtype) {
    WgradGrid g;
    if (!wgrad_grid(dtype, a.ntiles, a.Nn, a.C, a.K, a.R, a.S, a.Hot, &g)) return false;
    a.TRB = g.TRB;
    a.chunks_per_tile = g.chunks_per_tile;
    a.rows_per_chunk = g.rows_per_chunk;
    a.nchunks = a.ntiles * g.chunks_per_tile;
    if (dtype == 1) {
        const int plane = odd16(a.TRB * bf16_xwp(a.istr, a.S));
        a.lds_bytes = (64 * kDyP + 64 * plane) * 2;
    } else {
        const int XW = (kBQ - 1) * a.istr + a.S;
        // channels a workgroup's 256 flattened columns can touch
        const int span = std::min(a.C, 256 / (a.R * a.S) + 2);
        a.lds_bytes = (64 * (kBQ + 1) + span * a.R * XW) * 4;
    }
    return a.lds_bytes <= device_lds_limit();
}

// ---------------------------------------------------------------- bf16

template <int SS, int TRB>
__global__ __launch_bounds__(kThreads) void wgrad_bf16_kernel(WgradArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int XWP = bf16_xwp(a.istr, SS);
    const int PLANE = odd16(a.TRB * XWP);   // a.TRB <= TRB rows are staged
    uint16_t* dyl = reinterpret_cast<uint16_t*>(smem);   // [64 o][kDyP]
    uint16_t* xl = dyl + 64 * kDyP;                      // [64 ci][TRB rows][XWP]

    const int chunk = blockIdx.x;
    const int tile = chunk / a.chunks_per_tile;
    const int row_b = (chunk - tile * a.chunks_per_tile) * a.rows_per_chunk;
    const int row_e = min(row_b + a.rows_per_chunk, a.Nn * a.Hot);
    const int r0 = blockIdx.y * a.TRB;
    const int nTR = min(a.TRB, a.R - r0);
    const int ncsb = (a.C + 63) / 64;
    const int o0 = (blockIdx.z / ncsb) * 64, c0 = (blockIdx.z % ncsb) * 64;

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int ow = wave & 1, cw = wave >> 1;

    const uint16_t* xt = static_cast<const uint16_t*>(a.x) + tile * a.x_tile;
    const uint16_t* dyt = static_cast<const uint16_t*>(a.dy) + tile * a.dy_tile;
    const int64_t xplane = int64_t(a.x_rows) * a.x_pitch;
    const int dy_rows = a.Hot + 2 * a.dy_off;
    const int64_t dyplane = int64_t(dy_rows) * a.dy_pitch;

    floatx16 acc[TRB][SS];
#pragma unroll
    for (int i = 0; i < TRB; ++i)
#pragma unroll
        for (int j = 0; j < SS; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    const int ncb = (a.Wot + kBQ - 1) / kBQ;
    const int XW = (kBQ - 1) * a.istr + SS;
    for (int f = row_b; f < row_e; ++f) {
        const int n = f / a.Hot, p = f - n * a.Hot;
        for (int cb = 0; cb < ncb; ++cb) {
            const int q0 = cb * kBQ;
            __syncthreads();
            // dy row segment: [64 o][kBQ], zero beyond the tile
            for (int e = tid; e < 64 * kBQ; e += kThreads) {
                const int q = e % kBQ, ol = e / kBQ;
                const int o = o0 + ol;
                uint16_t v = 0;
                if (o < a.K && q0 + q < a.Wot)
                    v = dyt[(int64_t(n) * a.K + o) * dyplane + int64_t(p + a.dy_off) * a.dy_pitch +
                            a.dy_off + q0 + q];
                dyl[ol * kDyP + q] = v;
            }
            // x rows p*istr + r + base_r for this group's filter rows
            for (int e = tid; e < 64 * a.TRB * XWP; e += kThreads) {
                const int xc = e % XWP;
                const int rest = e / XWP;
                const int tr = rest % a.TRB, cl = rest / a.TRB;
                const int ci = c0 + cl;
                const int gr = p * a.istr + a.base_r + r0 + tr;
                const int gc = q0 * a.istr + a.base_c + xc;
                uint16_t v = 0;
                if (ci < a.C && tr < nTR && xc < XW && gr < a.x_rows && gc < a.x_cols)
                    v = xt[(int64_t(n) * a.C + ci) * xplane + int64_t(gr) * a.x_pitch + gc];
                xl[cl * PLANE + tr * XWP + xc] = v;
            }
            __syncthreads();

            const int qmax = min(kBQ, a.Wot - q0);
            for (int kq = 0; kq < qmax; kq += 16) {
                const int qc = kq + 8 * hi;   // first of this half-wave's 8 pixels
                Pack8 A;
                A.v = *reinterpret_cast<const uint4*>(dyl + (ow * 32 + l32) * kDyP + qc);
                const uint16_t* xrow0 = xl + (cw * 32 + l32) * PLANE;
#pragma unroll
                for (int tr = 0; tr < TRB; ++tr) {
                    if (tr >= nTR) continue;
                    const uint16_t* xr = xrow0 + tr * XWP;
                    if (a.istr == 1) {
                        Pack8 lo, hh;
                        lo.v = *reinterpret_cast<const uint4*>(xr + qc);
                        hh.v = *reinterpret_cast<const uint4*>(xr + qc + 8);
                        const uint32_t d[8] = {lo.d[0], lo.d[1], lo.d[2], lo.d[3],
                                               hh.d[0], hh.d[1], hh.d[2], hh.d[3]};
#pragma unroll
                        for (int s = 0; s < SS; ++s) {
                            Pack8 B;
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                if ((s & 1) == 0)
                                    B.d[i] = d[s / 2 + i];
                                else
                                    B.d[i] = __builtin_amdgcn_alignbyte(d[s / 2 + i + 1], d[s / 2 + i], 2);
                            }
                            acc[tr][s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A.b, B.b, acc[tr][s], 0, 0, 0);
                        }
                    } else {
#pragma unroll
                        for (int s = 0; s < SS; ++s) {
                            Pack8 B;
#pragma unroll
                            for (int j = 0; j < 8; ++j) B.h[j] = xr[(qc + j) * a.istr + s];
                            acc[tr][s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A.b, B.b, acc[tr][s], 0, 0, 0);
                        }
                    }
                }
            }
        }
    }

    // partial slice: rows = filters, columns = channels (D layout of the 32x32 tile)
    float* part = a.part + int64_t(chunk) * a.K * a.C * a.R * a.S;
    const int ci = c0 + cw * 32 + l32;
    if (ci >= a.C) return;
#pragma unroll
    for (int tr = 0; tr < TRB; ++tr) {
        if (tr >= nTR) continue;
#pragma unroll
        for (int s = 0; s < SS; ++s)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int o = o0 + ow * 32 + 8 * (i / 4) + 4 * hi + (i % 4);
                if (o < a.K)
                    part[((int64_t(o) * a.C + ci) * a.R + r0 + tr) * a.S + s] = acc[tr][s][i];
            }
    }
}

// ---------------------------------------------------------------- fp32

template <int NBW>
__global__ __launch_bounds__(kThreads) void wgrad_f32_kernel(WgradArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int DYP = kBQ + 1;
    float* dyl = reinterpret_cast<float*>(smem);   // [64 o][DYP]
    float* xl = dyl + 64 * DYP;                    // [span ci][R][XW]
    const int XW = (kBQ - 1) * a.istr + a.S;
    const int RS = a.R * a.S, CRS = a.C * RS;
    const int NCB = (CRS + 31) / 32;

    const int chunk = blockIdx.x;
    const int tile = chunk / a.chunks_per_tile;
    const int row_b = (chunk - tile * a.chunks_per_tile) * a.rows_per_chunk;
    const int row_e = min(row_b + a.rows_per_chunk, a.Nn * a.Hot);
    const int o0 = blockIdx.z * 64;
    const int NOB = min(2, (a.K - o0 + 31) / 32);

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int cbw = (blockIdx.y * 4 + wave) * NBW;      // this wave's first column block
    const int col_lo = blockIdx.y * 4 * NBW * 32;        // workgroup's first flattened column
    const int col_hi = min(CRS, col_lo + 4 * NBW * 32) - 1;
    const int ci_lo = col_lo / RS, ci_hi = col_hi / RS;
    const int span = ci_hi - ci_lo + 1;

    // this lane's (ci, r, s) for each of its column blocks
    int xoff[NBW];
    bool valid[NBW];
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
        const int fcol = (cbw + j) * 32 + l32;
        valid[j] = fcol < CRS;
        const int ci = valid[j] ? fcol / RS : ci_lo;
        const int rs = valid[j] ? fcol - ci * RS : 0;
        const int r = rs / a.S, s = rs - r * a.S;
        xoff[j] = ((ci - ci_lo) * a.R + r) * XW + s;
    }
    const bool wave_active = cbw < NCB;

    const float* xt = static_cast<const float*>(a.x) + tile * a.x_tile;
    const float* dyt = static_cast<const float*>(a.dy) + tile * a.dy_tile;
    const int64_t xplane = int64_t(a.x_rows) * a.x_pitch;
    const int dy_rows = a.Hot + 2 * a.dy_off;
    const int64_t dyplane = int64_t(dy_rows) * a.dy_pitch;

    floatx16 acc[2][NBW];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NBW; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    const int ncb = (a.Wot + kBQ - 1) / kBQ;
    for (int f = row_b; f < row_e; ++f) {
        const int n = f / a.Hot, p = f - n * a.Hot;
        for (int cb = 0; cb < ncb; ++cb) {
            const int q0 = cb * kBQ;
            __syncthreads();
            for (int e = tid; e < 64 * kBQ; e += kThreads) {
                const int q = e % kBQ, ol = e / kBQ;
                const int o = o0 + ol;
                float v = 0.f;
                if (o < a.K && q0 + q < a.Wot)
                    v = dyt[(int64_t(n) * a.K + o) * dyplane + int64_t(p + a.dy_off) * a.dy_pitch +
                            a.dy_off + q0 + q];
                dyl[ol * DYP + q] = v;
            }
            for (int e = tid; e < span * a.R * XW; e += kThreads) {
                const int xc = e % XW;
                const int rest = e / XW;
                const int r = rest % a.R, cl = rest / a.R;
                const int gr = p * a.istr + a.base_r + r;
                const int gc = q0 * a.istr + a.base_c + xc;
                float v = 0.f;
                if (gr < a.x_rows && gc < a.x_cols)
                    v = xt[(int64_t(n) * a.C + ci_lo + cl) * xplane + int64_t(gr) * a.x_pitch + gc];
                xl[e] = v;
            }
            __syncthreads();
            if (!wave_active) continue;
            const int qmax = min(kBQ, a.Wot - q0);
            // k-step: half-wave 0 takes pixel kk, half-wave 1 pixel kk+32
            for (int kk = 0; kk < 32; ++kk) {
                const int q = kk + 32 * hi;
                if (kk >= qmax) break;   // uniform: kk < 32 <= ... both halves share kk
                float A[2], B[NBW];
#pragma unroll
                for (int ob = 0; ob < 2; ++ob) A[ob] = dyl[(ob * 32 + l32) * DYP + q];
#pragma unroll
                for (int j = 0; j < NBW; ++j) B[j] = valid[j] ? xl[xoff[j] + q * a.istr] : 0.f;
#pragma unroll
                for (int ob = 0; ob < 2; ++ob) {
                    if (ob >= NOB) continue;
#pragma unroll
                    for (int j = 0; j < NBW; ++j)
                        acc[ob][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(A[ob], B[j], acc[ob][j], 0, 0, 0);
                }
            }
        }
    }

    if (!wave_active) return;
    float* part = a.part + int64_t(chunk) * a.K * CRS;
#pragma unroll
    for (int ob = 0; ob < 2; ++ob) {
        if (ob >= NOB) continue;
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
            if (!valid[j]) continue;
            const int fcol = (cbw + j) * 32 + l32;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int o = o0 + ob * 32 + 8 * (i / 4) + 4 * hi + (i % 4);
                if (o < a.K) part[int64_t(o) * CRS + fcol] = acc[ob][j][i];
            }
        }
    }
}

// ---------------------------------------------------------------- reduction

// dw[e] = (accumulate ? dw[e] : 0) + sum_{c = 0..nchunks-1} part[c][e], in chunk order.
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ part,
                                                           float* __restrict__ dw, int64_t E,
                                                           int nchunks, int accumulate) {
    const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (e >= E) return;
    float s = 0.f;
    for (int c = 0; c < nchunks; ++c) s += part[int64_t(c) * E + e];
    dw[e] = accumulate ? dw[e] + s : s;
}

template <typename K>
static hipError_t set_lds(K kernel, int bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

template <int SS>
static hipError_t launch_bf16(const WgradArgs& a, dim3 grid, hipStream_t s) {
    constexpr int TRB = SS == 1 ? 9 : (9 / SS > 0 ? 9 / SS : 1);
    hipError_t e = set_lds(wgrad_bf16_kernel<SS, TRB>, a.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wgrad_bf16_kernel<SS, TRB>), grid, dim3(kThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& a, int dtype, hipStream_t s) {
    WgradGrid g;
    wgrad_grid(dtype, a.ntiles, a.Nn, a.C, a.K, a.R, a.S, a.Hot, &g);
    dim3 grid(a.nchunks, g.gy, g.gz);
    hipError_t e = hipSuccess;
    if (dtype == 1) {
        switch (a.S) {
            case 1: e = launch_bf16<1>(a, grid, s); break;
            case 2: e = launch_bf16<2>(a, grid, s); break;
            case 3: e = launch_bf16<3>(a, grid, s); break;
            case 4: e = launch_bf16<4>(a, grid, s); break;
            case 5: e = launch_bf16<5>(a, grid, s); break;
            case 6: e = launch_bf16<6>(a, grid, s); break;
            case 7: e = launch_bf16<7>(a, grid, s); break;
            default: return hipErrorInvalidValue;
        }
    } else {
        e = set_lds(wgrad_f32_kernel<2>, a.lds_bytes);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(wgrad_f32_kernel<2>, grid, dim3(kThreads), a.lds_bytes, s, a);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    const int64_t E = int64_t(a.K) * a.C * a.R * a.S;
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(unsigned((E + 255) / 256)), dim3(256), 0, s,
                       a.part, a.dw, E, a.nchunks, a.accumulate);
    return hipGetLastError();
}

}  // namespace dc
