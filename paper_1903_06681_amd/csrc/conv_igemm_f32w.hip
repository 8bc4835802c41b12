// Forward / backward-data convolution, fp32, stride-1 input walk, weights in
// registers (Eqs. (1) and (3) of Sec. II-A on a tile, Sec. III-A).
//
//   out[o][pixel] = sum_{tap, ci} W[o][tap, ci] * in[ci][pixel + tap]
//
// v_mfma_f32_32x32x2_f32: a k-step is two reduction values; lane l feeds row
// (output channel) / column (pixel) l % 32 with reduction value l / 32.  The
// reduction is ordered (tap, channel pair): k-step j = t * CIN/2 + cp takes
// channels 2cp and 2cp+1 of tap t, so the lane's channel is 2cp + l/32 and
// the B operand of every k-step is one 4-byte LDS read at a per-lane base plus
// a compile-time offset.  Each lane keeps its A values (one per k-step) in
// registers for the whole launch.
//
// The kernel is compiled for a channel capacity CC (a class: multiples of 4
// up to 32, and 18, the mesh layer's count) and runs any channel count
// C <= CC: channels C .. CC-1 get zero weights and zero-filled ring rows, so
// they add nothing (at most three per k-step group; none for C = CC).
//
// A workgroup (4 waves) walks down a 64-column strip of one sample, two
// output rows per step (wave w: row w / 2, pixels 32 * (w % 2) .. + 31); input
// rows live in an LDS ring stored channel-major ([row][channel][column]).
// Each step loads the two new input rows with 16-byte loads from clamped
// addresses (out-of-tile values only feed outputs that are never stored) and
// writes them to the ring after the step's MFMAs.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "bf16util.h"
#include "kernels.h"

namespace dc {

namespace {

constexpr int kF32WThreads = 256;
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int TS>
struct F32WGeom {
    static constexpr int XW = 64 + TS - 1;                 // staged columns
    static constexpr int XWP = (XW + 3) / 4 * 4 + 4;       // row pitch (floats): 16-byte units, odd-ish
    static constexpr int V4 = XWP / 4;                     // 16-byte units per staged row
};

}  // namespace

template <int CIN, int TR, int TS>   // CIN: the channel capacity, a.Cin <= CIN
__global__ __launch_bounds__(kF32WThreads, 1) void igemm_f32w_kernel(IgemmArgs a) {
    using G = F32WGeom<TS>;
    constexpr int T = TR * TS;
    constexpr int NJ = T * CIN / 2;                          // k-steps
    constexpr int NRING = TR + 3;
    constexpr int ROW = CIN * G::XWP;                        // floats per ring row
    constexpr int UNITS = 2 * CIN * G::V4;                   // 16-byte units per step (two rows)
    constexpr int UPT = (UNITS + kF32WThreads - 1) / kF32WThreads;
    constexpr int PF = 8;                                    // B reads in flight ahead of the MFMAs
    extern __shared__ __align__(16) unsigned char smem[];
    float* ring = reinterpret_cast<float*>(smem);

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int vb = c % a.nvb; c /= a.nvb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int u0 = seg * a.rows_per_seg;
    const int u_end = min(u0 + a.rows_per_seg, a.Uo);
    const int v0 = vb * 64;
    const int o0 = blockIdx.y * 32;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int wrow = wave >> 1, pb = wave & 1;

    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const int cin = a.Cin;
    const float* in = static_cast<const float*>(a.in) + tile * a.in_tile + int64_t(n) * cin * plane;
    const int xr0 = u0 + a.base_r;   // input row of ring row 0
    const int xc0 = v0 + a.base_c;   // input column of staged column 0 (a multiple of 4)

    // ---- A values: k-step j = t * CIN/2 + cp, channel 2cp + hi, tap t
    float A[NJ];
    {
        const float* w = static_cast<const float*>(a.w);
        const int o = o0 + l32;
        const bool ok = o < a.Cout;
        const int64_t wo = int64_t(ok ? o : 0) * a.w_os;
        static_for<0, NJ>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            constexpr int t = j / (CIN / 2), cp = j % (CIN / 2), tr = t / TS, ts = t % TS;
            const int ci = 2 * cp + hi;
            const bool oki = ok && ci < cin;
            const float v = w[wo + (oki ? ci : 0) * a.w_cs + (a.wr0 + a.wrstep * tr) * a.S + (a.ws0 + a.wsstep * ts)];
            A[j] = oki ? v : 0.f;
        });
    }

    // ---- staging: unit u of a step = (row q of the two, channel ci, 16-byte column group g)
    f32x4 stg[UPT];
    auto load_rows = [&](int m0) {   // ring rows m0, m0+1 -> registers
        static_for<0, UPT>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int u = min(tid + k * kF32WThreads, UNITS - 1);
            const int q = u / (CIN * G::V4), rem = u % (CIN * G::V4);
            const int ci = rem / G::V4, g = rem % G::V4;
            const int gr = min(max(xr0 + m0 + q, 0), a.in_rows - 1);
            const int gc = min(xc0 + 4 * g, a.in_pitch - 4);
            stg[k] = ci < cin ? *reinterpret_cast<const f32x4*>(in + ci * plane + int64_t(gr) * a.in_pitch + gc)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
        });
    };
    auto store_rows = [&](int m0) {
        static_for<0, UPT>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int u = min(tid + k * kF32WThreads, UNITS - 1);   // duplicates repeat the last unit
            const int q = u / (CIN * G::V4), rem = u % (CIN * G::V4);
            const int ci = rem / G::V4, g = rem % G::V4;
            *reinterpret_cast<f32x4*>(ring + ((m0 + q) % NRING) * ROW + ci * G::XWP + 4 * g) = stg[k];
        });
    };

    // ring rows 0 .. TR (the inputs of the first two output rows)
    for (int m = 0; m <= TR; m += 2) {
        load_rows(m);
        store_rows(m);
    }
    __syncthreads();

    const int px = pb * 32 + l32;
    const int v = v0 + px;
    const int64_t oplane = int64_t(a.out_rows) * a.out_cols;
    float* const out = a.out + tile * a.out_tile + (int64_t(n) * a.Cout + o0 + 4 * hi) * oplane +
                       int64_t(v) * a.ostr + a.oph_c;
    const int lbase = hi * G::XWP + px;   // this lane's B offset inside a ring row
    const int nsteps = (u_end - u0 + 1) / 2;
    for (int i = 0; i < nsteps; ++i) {
        load_rows(2 * i + TR + 1);
        const float* rows[TR];
#pragma unroll
        for (int tr = 0; tr < TR; ++tr) rows[tr] = ring + ((2 * i + wrow + tr) % NRING) * ROW + lbase;
        auto readB = [&](auto jc) {
            constexpr int j = decltype(jc)::value;
            constexpr int t = j / (CIN / 2), cp = j % (CIN / 2);
            return rows[t / TS][2 * cp * G::XWP + (t % TS)];
        };
        floatx16 acc;
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] = 0.f;
        float Bq[PF];
        static_for<0, (PF < NJ ? PF : NJ)>([&](auto jc) { Bq[decltype(jc)::value] = readB(jc); });
        static_for<0, NJ>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            const float b = Bq[j % PF];
            if constexpr (j + PF < NJ) Bq[j % PF] = readB(std::integral_constant<int, j + PF>{});
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(A[j], b, acc, 0, 0, 0);
        });
        // D layout: value e of lane l is output channel 8*(e/4) + 4*(l/32) + e%4, pixel l%32
        const int u = u0 + 2 * i + wrow;
        if (u < u_end && v < a.Vo) {
            float* orow = out + int64_t(u * a.ostr + a.oph_r) * a.out_cols;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int oc = 8 * (e / 4) + (e % 4);
                if (o0 + 4 * hi + oc < a.Cout) __builtin_nontemporal_store(acc[e], orow + int64_t(oc) * oplane);
            }
        }
        store_rows(2 * i + TR + 1);
        __syncthreads();
    }
}

// ---------------------------------------------------------------- planning

// Channel capacity class of a layer with C input channels (0: none): the
// smallest of 4, 8, .., 32 that holds C, and 18 for the mesh layer's 17-18.
static int f32w_class(int C) {
    if (C < 1 || C > 32) return 0;
    if (C == 17 || C == 18) return 18;
    return (C + 3) / 4 * 4;
}
// filters the kernel is instantiated for: 3x3 and 1x1
static bool f32w_filter(int TR, int TS) { return (TR == 3 && TS == 3) || (TR == 1 && TS == 1); }

static int f32w_lds(int CIN, int TR, int TS) {
    const int XW = 64 + TS - 1, XWP = (XW + 3) / 4 * 4 + 4;
    return (TR + 3) * CIN * XWP * 4;
}

bool igemm_f32w_plan(IgemmArgs& a) {
    if (a.istr != 1 || a.Tr < 1 || a.Ts < 1) return false;
    if (a.base_c % 4 != 0 || a.in_pitch % 4 != 0) return false;   // 16-byte aligned row loads
    const int cc = f32w_class(a.Cin);
    if (cc == 0 || !f32w_filter(a.Tr, a.Ts)) return false;
    const int lds = f32w_lds(cc, a.Tr, a.Ts);
    if (lds > device_lds_limit()) return false;
    a.OB = 32;
    a.nvb = (a.Vo + 63) / 64;
    const int strips = a.ntiles * a.Nn * a.nvb * ((a.Cout + 31) / 32);
    const int want = 256;
    int nseg = (want + strips - 1) / strips;
    nseg = nseg < 1 ? 1 : nseg;
    int rps = (a.Uo + nseg - 1) / nseg;
    rps = (rps + 1) & ~1;   // whole steps of two rows
    if (rps < 2) rps = 2;
    a.rows_per_seg = rps;
    a.nseg = (a.Uo + rps - 1) / rps;
    a.lds_bytes = lds;
    a.kind = 2;
    return true;
}

template <int CIN, int TR, int TS>
static hipError_t launch_f32w(const IgemmArgs& a, hipStream_t s) {
    auto k = igemm_f32w_kernel<CIN, TR, TS>;
    if (a.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    dim3 grid(a.ntiles * a.Nn * a.nvb * a.nseg, (a.Cout + 31) / 32);
    hipLaunchKernelGGL(k, grid, dim3(kF32WThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_igemm_f32w(const IgemmArgs& a, hipStream_t s) {
    const int cc = f32w_class(a.Cin);
#define DC_F32W(cin, tr, ts) \
    if (cc == cin && a.Tr == tr && a.Ts == ts) return launch_f32w<cin, tr, ts>(a, s);
    DC_F32W(4, 3, 3) DC_F32W(8, 3, 3) DC_F32W(12, 3, 3) DC_F32W(16, 3, 3) DC_F32W(18, 3, 3)
    DC_F32W(20, 3, 3) DC_F32W(24, 3, 3) DC_F32W(28, 3, 3) DC_F32W(32, 3, 3)
    DC_F32W(4, 1, 1) DC_F32W(8, 1, 1) DC_F32W(12, 1, 1) DC_F32W(16, 1, 1) DC_F32W(18, 1, 1)
    DC_F32W(20, 1, 1) DC_F32W(24, 1, 1) DC_F32W(28, 1, 1) DC_F32W(32, 1, 1)
#undef DC_F32W
    return hipErrorInvalidValue;
}

}  // namespace dc
