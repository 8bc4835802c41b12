// Forward / backward-data convolution, bf16, stride-1 input walk: the weights
// stay in registers (Eqs. (1) and (3) of Sec. II-A on a tile, Sec. III-A).
//
//   out[o][pixel] = sum_{tap, ci} W[o][tap, ci] * in[ci][pixel + tap]
//
// Each wave keeps the whole weight operand of its OB output channels as
// v_mfma_f32_32x32x16_bf16 A-fragments in VGPRs (OB x taps x Cin values,
// loaded once per workgroup), so the k-loop reads only the input operand
// from LDS: one 16-byte read feeds OB/32 MFMAs.
//
// A workgroup (4 waves) walks down a 64-column strip of one sample, two
// output rows per step; wave w computes row w/2, pixels 32*(w%2)..+31.  Input
// rows are kept in an LDS ring, channel-innermost ([row][pixel][channel],
// odd 16-byte pixel stride), so the 8 channels of a pixel are one aligned
// read.  Each step loads the two new input rows with 16-byte global loads
// (8 channels x 8 pixels per thread), transposes them in registers and
// stores them while the previous rows run on the matrix cores.
#include <hip/hip_runtime.h>

#include "bf16util.h"
#include "kernels.h"

namespace dc {

static constexpr int kWThreads = 256;

// 8x8 transpose of 16-bit elements: in[c] holds 8 pixels of channel c,
// out[p] receives the 8 channels of pixel p.
__device__ __forceinline__ void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
    const uint32_t* s = reinterpret_cast<const uint32_t*>(in);
    uint32_t* d = reinterpret_cast<uint32_t*>(out);
#pragma unroll
    for (int m = 0; m < 4; ++m)        // pixel pair (2m, 2m+1)
#pragma unroll
        for (int j = 0; j < 4; ++j) {  // channel pair (2j, 2j+1)
            const uint32_t lo = s[(2 * j) * 4 + m], hi = s[(2 * j + 1) * 4 + m];
            d[(2 * m) * 4 + j] = (lo & 0xffffu) | (hi << 16);
            d[(2 * m + 1) * 4 + j] = (lo >> 16) | (hi & 0xffff0000u);
        }
}

template <int NOB, int TR, int TS, int CG, int MINWG>
__global__ __launch_bounds__(kWThreads, MINWG) void igemm_wreg_kernel(IgemmArgs a) {
    constexpr int KS = TR * TS * CG;          // 16-wide k-steps: (tap, 16-channel group)
    constexpr int CIN = CG * 16;
    constexpr int PS = 8 * ((CIN / 8) | 1);   // ring pixel stride (elements)
    constexpr int RPX8 = (64 + TS - 1 + 7) / 8;
    constexpr int NRING = TR + 3;
    constexpr int ROWSZ = RPX8 * 8 * PS;
    constexpr int OBT = NOB * 32;
    constexpr int NCG8 = CIN / 8;
    constexpr int BLK_ROW = NCG8 * RPX8;      // 8x8 staging blocks per ring row
    constexpr int BPT = (2 * BLK_ROW + kWThreads - 1) / kWThreads;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int vb = c % a.nvb; c /= a.nvb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int u0 = seg * a.rows_per_seg;
    const int u_end = min(u0 + a.rows_per_seg, a.Uo);
    const int v0 = vb * 64;
    const int o0 = blockIdx.y * OBT;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;

    // ---- weights -> A-fragments in VGPRs, in three LDS passes:
    //  1. the workgroup's block of w, copied in its natural order with
    //     coalesced 16-byte loads: rows of `rowlen` elements
    //       forward:       row = output channel o  -> w[o][0..Cin)[R][S]
    //       backward-data: row = reduction channel -> w[ci][o0..o0+nO)[R][S]
    //  2. the fragment image [KS][2][OBT][8]: 8 reduction channels of one
    //     (output channel, tap) per 16-byte entry, zero where o >= Cout;
    //  3. each wave reads its OB/32 x KS fragments.
    const int T = a.R * a.S;
    const int nO = min(OBT, a.Cout - o0);               // valid output channels here
    const int nrow = a.wmode ? CIN : nO;
    const int rowlen = a.wmode ? nO * T : CIN * T;
    const int pitch = rowlen + ((6 - rowlen % 4) % 4);   // pitch % 4 == 2: odd dword stride
    const int nat_elems = nrow * pitch;
    uint16_t* nat = lds;                                 // [nrow][pitch]
    uint16_t* img = lds + ((nat_elems + 7) & ~7);        // [KS][2][OBT][8]
    {
        const uint16_t* w = static_cast<const uint16_t*>(a.w);
        const int64_t row_stride = a.wmode ? int64_t(a.Cout) * T : int64_t(CIN) * T;
        const int64_t col0 = a.wmode ? int64_t(o0) * T : int64_t(o0) * CIN * T;
        const bool vec = (rowlen % 8 == 0) && (row_stride % 8 == 0) && (col0 % 8 == 0);
        if (vec) {
            const int vpr = rowlen / 8, nv = nrow * vpr;
            for (int base = 0; base < nv; base += 8 * kWThreads) {
                uint4 buf[8];
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                    int v = base + b * kWThreads + tid;
                    v = v < nv ? v : nv - 1;
                    const int row = v / vpr, cv = v - row * vpr;
                    buf[b] = *reinterpret_cast<const uint4*>(w + col0 + row * row_stride + cv * 8);
                }
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                    const int v = base + b * kWThreads + tid;
                    if (v < nv) {
                        const int row = v / vpr, cv = v - row * vpr;
                        uint32_t* dst = reinterpret_cast<uint32_t*>(nat + row * pitch + cv * 8);
                        dst[0] = buf[b].x; dst[1] = buf[b].y; dst[2] = buf[b].z; dst[3] = buf[b].w;
                    }
                }
            }
        } else {
            for (int e = tid; e < nrow * rowlen; e += kWThreads) {
                const int row = e / rowlen, cl = e - row * rowlen;
                nat[row * pitch + cl] = w[col0 + row * row_stride + cl];
            }
        }
    }
    __syncthreads();
    for (int u = tid; u < KS * 2 * OBT; u += kWThreads) {
        const int ol = u % OBT, kh = u / OBT;
        const int h2 = kh & 1, k = kh >> 1;
        const int t = k / CG, cgi = k - t * CG;
        const int tr = t / TS, ts = t - tr * TS;
        const int tn = (a.wr0 + a.wrstep * tr) * a.S + (a.ws0 + a.wsstep * ts);   // tap in w
        const int ci0 = cgi * 16 + 8 * h2;
        Pack8 pk;
        if (ol < nO) {
            const int base = a.wmode ? ci0 * pitch + ol * T + tn : ol * pitch + ci0 * T + tn;
            const int step = a.wmode ? pitch : T;
#pragma unroll
            for (int j = 0; j < 8; ++j) pk.h[j] = nat[base + j * step];
        } else {
            pk.v = make_uint4(0, 0, 0, 0);
        }
        *reinterpret_cast<uint4*>(img + u * 8) = pk.v;
    }
    __syncthreads();
    bf16x8 Wf[NOB][KS];
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int k = 0; k < KS; ++k)
            Wf[ob][k] = *reinterpret_cast<const bf16x8*>(img + ((k * 2 + hi) * OBT + ob * 32 + l32) * 8);
    __syncthreads();   // the image space becomes the input ring

    // ---- input ring
    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const uint16_t* in = static_cast<const uint16_t*>(a.in) + tile * a.in_tile +
                         int64_t(n) * a.Cin * plane;
    const int xr0 = u0 + a.base_r;   // input row of ring row 0 (stride-1 walk)
    const int xc0 = v0 + a.base_c;   // input column of staged pixel 0 (a multiple of 8)
    uint4 stg[BPT][8];

    auto load_rows = [&](int m0, int nrow) {   // ring rows m0 .. m0+nrow-1 -> registers
#pragma unroll
        for (int b = 0; b < BPT; ++b) {
            const int blk = tid + b * kWThreads;
            if (blk < nrow * BLK_ROW) {
                const int m = m0 + blk / BLK_ROW, rb = blk % BLK_ROW;
                const int cg8 = rb % NCG8, pg = rb / NCG8;
                // Unconditional 16-byte loads from clamped addresses: a row or
                // column outside the tile only ever feeds output pixels that
                // are not stored, so its values need no masking.
                const int gr = min(max(xr0 + m, 0), a.in_rows - 1);
                const int gc = min(xc0 + pg * 8, a.in_pitch - 8);
                const uint16_t* src = in + int64_t(gr) * a.in_pitch + gc + (cg8 * 8) * plane;
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    stg[b][j] = *reinterpret_cast<const uint4*>(src + j * plane);
            }
        }
    };
    auto store_rows = [&](int m0, int nrow) {
#pragma unroll
        for (int b = 0; b < BPT; ++b) {
            const int blk = tid + b * kWThreads;
            if (blk < nrow * BLK_ROW) {
                const int m = m0 + blk / BLK_ROW, rb = blk % BLK_ROW;
                const int cg8 = rb % NCG8, pg = rb / NCG8;
                uint4 t[8];
                transpose8x8(stg[b], t);
                uint16_t* dst = lds + (m % NRING) * ROWSZ + (pg * 8) * PS + cg8 * 8;
#pragma unroll
                for (int p = 0; p < 8; ++p) *reinterpret_cast<uint4*>(dst + p * PS) = t[p];
            }
        }
    };

    // prologue: ring rows 0 .. TR (the inputs of the first two output rows)
    for (int m = 0; m <= TR; m += 2) {
        const int nr = min(2, TR + 1 - m);
        load_rows(m, nr);
        store_rows(m, nr);
    }
    __syncthreads();

    float* out = a.out + tile * a.out_tile + int64_t(n) * a.Cout * a.out_rows * a.out_cols;
    const int wrow = wave >> 1;
    const int px = (wave & 1) * 32 + l32;
    const int nsteps = (u_end - u0 + 1) / 2;
    for (int i = 0; i < nsteps; ++i) {
        const bool more = i + 1 < nsteps;
        if (more) load_rows(2 * i + TR + 1, 2);

        floatx16 acc[NOB];
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[ob][e] = 0.f;
        const int slot0 = (2 * i + wrow) % NRING;
#pragma unroll
        for (int k = 0; k < KS; ++k) {
            const int t = k / CG, cgi = k % CG;
            const int tr = t / TS, ts = t % TS;
            int slot = slot0 + tr;
            if (slot >= NRING) slot -= NRING;
            const bf16x8 B = *reinterpret_cast<const bf16x8*>(
                lds + slot * ROWSZ + (px + ts) * PS + cgi * 16 + 8 * hi);
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob)
                acc[ob] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Wf[ob][k], B, acc[ob], 0, 0, 0);
        }

        // D layout: value e of lane l is output channel 8*(e/4) + 4*(l/32) + e%4, pixel l%32
        const int u = u0 + 2 * i + wrow;
        const int v = v0 + px;
        if (u < u_end && v < a.Vo) {
            float* orow = out + int64_t(u * a.ostr + a.oph_r) * a.out_cols + v * a.ostr + a.oph_c;
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int o = o0 + ob * 32 + 8 * (e / 4) + 4 * hi + (e % 4);
                    if (o < a.Cout) orow[int64_t(o) * a.out_rows * a.out_cols] = acc[ob][e];
                }
        }
        if (more) store_rows(2 * i + TR + 1, 2);
        __syncthreads();
    }
}

// ---------------------------------------------------------------- planning

static bool wreg_shape(int NOB, int TR, int TS, int CG) {
    // instantiated shapes (see launch_igemm_wreg)
    const int shapes[][4] = {{2, 3, 3, 4}, {1, 3, 3, 4}, {1, 5, 5, 2}, {2, 1, 1, 16},
                             {2, 1, 1, 4}, {1, 3, 4, 4}, {1, 4, 3, 4}, {1, 4, 4, 4}, {2, 3, 3, 2},
                             {1, 3, 3, 2}};
    for (auto& s : shapes)
        if (s[0] == NOB && s[1] == TR && s[2] == TS && s[3] == CG) return true;
    return false;
}

static int wreg_lds(int NOB, int TR, int TS, int CG, int nO, int T, int wmode) {
    const int CIN = CG * 16, PS = 8 * ((CIN / 8) | 1), RPX8 = (64 + TS - 1 + 7) / 8;
    const int ring = (TR + 3) * RPX8 * 8 * PS * 2;
    const int nrow = wmode ? CIN : nO, rowlen = wmode ? nO * T : CIN * T;
    const int pitch = rowlen + ((6 - rowlen % 4) % 4);
    const int nat = ((nrow * pitch + 7) & ~7) * 2;
    const int image = TR * TS * CG * 2 * NOB * 32 * 16;
    return ring > nat + image ? ring : nat + image;
}

bool igemm_wreg_plan(IgemmArgs& a) {
    if (a.istr != 1 || a.Cin % 16 != 0 || a.Tr < 1 || a.Ts < 1) return false;
    if (a.base_c % 8 != 0 || a.in_pitch % 8 != 0) return false;   // 16-byte aligned row loads
    const int NOB = a.Cout <= 32 ? 1 : 2;
    const int CG = a.Cin / 16;
    if (!wreg_shape(NOB, a.Tr, a.Ts, CG)) return false;
    const int lds = wreg_lds(NOB, a.Tr, a.Ts, CG, a.Cout < NOB * 32 ? a.Cout : NOB * 32, a.R * a.S,
                             a.wmode);
    if (lds > device_lds_limit()) return false;
    a.OB = NOB * 32;
    a.nvb = (a.Vo + 63) / 64;
    const int strips = a.ntiles * a.Nn * a.nvb * ((a.Cout + a.OB - 1) / a.OB);
    const int want = 256;
    int nseg = (want + strips - 1) / strips;
    nseg = nseg < 1 ? 1 : nseg;
    int rps = (a.Uo + nseg - 1) / nseg;
    rps = (rps + 1) & ~1;   // whole steps of two rows
    if (rps < 2) rps = 2;
    a.rows_per_seg = rps;
    a.nseg = (a.Uo + rps - 1) / rps;
    a.lds_bytes = lds;
    a.kind = 1;
    return true;
}

template <int NOB, int TR, int TS, int CG, int MINWG>
static hipError_t launch_one(const IgemmArgs& a, hipStream_t s) {
    auto k = igemm_wreg_kernel<NOB, TR, TS, CG, MINWG>;
    if (a.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    dim3 grid(a.ntiles * a.Nn * a.nvb * a.nseg, (a.Cout + a.OB - 1) / a.OB);
    hipLaunchKernelGGL(k, grid, dim3(kWThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_igemm_wreg(const IgemmArgs& a, hipStream_t s) {
    const int NOB = a.OB / 32, CG = a.Cin / 16;
#define DC_WREG(nob, tr, ts, cg) \
    if (NOB == nob && a.Tr == tr && a.Ts == ts && CG == cg) \
        return launch_one<nob, tr, ts, cg, 1>(a, s);
    DC_WREG(2, 3, 3, 4)
    DC_WREG(1, 3, 3, 4)
    DC_WREG(1, 5, 5, 2)
    DC_WREG(2, 1, 1, 16)
    DC_WREG(2, 1, 1, 4)
    DC_WREG(1, 3, 4, 4)
    DC_WREG(1, 4, 3, 4)
    DC_WREG(1, 4, 4, 4)
    DC_WREG(2, 3, 3, 2)
    DC_WREG(1, 3, 3, 2)
#undef DC_WREG
    return hipErrorInvalidValue;
}

}  // namespace dc
