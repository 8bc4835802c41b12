// Forward and backward-data convolution on a padded tile as an implicit GEMM
// on gfx950 matrix cores (Eqs. (1) and (3) of Sec. II-A on the tile of
// Sec. III-A).
//
//   D[o][pixel] = sum_{kg} A[o][kg] * B[kg][pixel],  kg = (tap, input channel)
//
// A is the weight tensor, B the implicit im2col view of the padded input
// tile.  A workgroup of 4 waves computes OB output channels x (4 rows x 64
// columns) of output pixels; wave w owns output row w, as OB/32 x 2 MFMA
// 32x32 tiles.  The input channels are walked in chunks of CC: each chunk
// stages the weights [tap, 8-channel group][o][8] and the input patch
// (rows x cols x channels, channel-innermost) in LDS, then runs the MFMA loop.
//
// bf16: v_mfma_f32_32x32x16_bf16.  A k-step of 16 = two groups of 8 channels
//       (one per half-wave), each group at its own tap; the 8 channels of a
//       pixel are one 16-byte LDS read.  The NCHW -> channel-innermost
//       transpose happens while staging.
// fp32: v_mfma_f32_32x32x2_f32.  A k-step of 2 = one (tap, channel) per
//       half-wave; a lane reads one float, so the patch stays channel-major.
// Accumulation is fp32 in both; outputs are fp32 stores of 32 consecutive
// pixels per half-wave (128-byte segments).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "bf16util.h"
#include "kernels.h"

namespace dc {


static constexpr int kThreads = 256;
static constexpr int kBH = 4;    // output rows per workgroup (one per wave)
static constexpr int kBW = 64;   // output columns per workgroup (two 32-pixel MFMA tiles)
// Staging batches: items per thread whose loads are all issued before the
// first is waited for (bf16 items are 8 loads each; larger fp32 batches
// measured slower)
static constexpr int kUB = 4, kUF = 8;
static constexpr int kRWord3c = 0x00020000;   // buffer resource word 3 (gfx9 family: raw access)
static constexpr int kOOBc = 0x7fffffff;      // byte offset past every buffer here: the load returns 0

// Pixel stride (bf16 elements) of the channel-innermost patch: an odd number
// of 16-byte units, so 16 consecutive lanes reading 16 B each hit distinct
// bank groups.
__host__ __device__ inline int bf16_pixel_stride(int CC) { return 8 * ((CC / 8) | 1); }

// fp32 patch plane stride (floats): rows*cols rounded up to 32 mod 64, so the
// two half-waves (adjacent channels, same pixels) use disjoint banks.
__host__ __device__ inline int f32_plane_stride(int p) {
    int r = p % 64;
    return r <= 32 ? p + (32 - r) : p + (96 - r);
}

// Pixels of a workgroup's input patch: kBH x kBW output block, or in frame
// mode the larger of that and its transpose (column segments).
__host__ __device__ inline int patch_pixels(const IgemmArgs& a) {
    const int rm = ((kBH - 1) * a.istr + a.Tr) * ((kBW - 1) * a.istr + a.Ts);
    const int cm = ((kBW - 1) * a.istr + a.Tr) * ((kBH - 1) * a.istr + a.Ts);
    return a.frame && cm > rm ? cm : rm;
}


// Output block of this workgroup: kBH rows x kBW columns from (u0, v0), with
// stores limited to rows < uend and columns < vend.  Whole tile: blocks in
// row-major order over Uo x Vo.  Frame mode: blocks of the segments in turn,
// each a rectangle of the output (the boundary band of a tile); the blocks of
// a column segment (cm) are kBW rows x kBH columns, wave w then owning output
// column w and its MFMA pixels running down the rows.
__device__ __forceinline__ void block_origin(const IgemmArgs& a, int& u0, int& v0, int& uend, int& vend,
                                             bool& cm) {
    cm = false;
    if (a.frame) {
        int sg = 0;
        while (sg + 1 < a.fseg && int(blockIdx.x) >= a.fblk[sg + 1]) ++sg;
        const int local = blockIdx.x - a.fblk[sg];
        cm = a.fcm[sg] != 0;   // column segment: blocks of kBW rows x kBH columns
        const int bw = cm ? kBH : kBW, bh = cm ? kBW : kBH;
        const int nvb = (a.fnv[sg] + bw - 1) / bw;
        const int vb = local % nvb, ub = local / nvb;
        u0 = a.fu0[sg] + ub * bh;
        v0 = a.fv0[sg] + vb * bw;
        uend = a.fu0[sg] + a.fnu[sg];
        vend = a.fv0[sg] + a.fnv[sg];
    } else {
        const int nvb = (a.Vo + kBW - 1) / kBW;
        const int vb = blockIdx.x % nvb, ub = blockIdx.x / nvb;
        u0 = ub * kBH;
        v0 = vb * kBW;
        uend = a.Uo;
        vend = a.Vo;
    }
}

// RB: the sample's input and the weights are under 2^31 bytes, so the staging
// gathers are buffer loads (an element outside the tensors is an offset past
// the buffer's end, which reads zero): no branches, a thread's batch of loads
// in flight together.  Otherwise the plain loop (one load round trip per item).
template <int OB, bool RB>
__global__ __launch_bounds__(kThreads) void igemm_bf16_kernel(IgemmArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int NOB = OB / 32;
    int u0, v0, uend, vend;
    bool cm;
    block_origin(a, u0, v0, uend, vend, cm);
    const int CC = a.CC, CCG = CC / 8;
    const int Tt = a.Tr * a.Ts;
    const int G = Tt * CCG;
    const int PR = ((cm ? kBW : kBH) - 1) * a.istr + a.Tr;
    const int PC = ((cm ? kBH : kBW) - 1) * a.istr + a.Ts;
    const int PS = bf16_pixel_stride(CC);
    uint16_t* wl = reinterpret_cast<uint16_t*>(smem);   // [G][OB][8]
    uint16_t* pl = wl + G * OB * 8;                      // [PR][PC][PS]

    const int o0 = blockIdx.y * OB;
    const int tile = blockIdx.z / a.Nn, n = blockIdx.z % a.Nn;

    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const uint16_t* in = static_cast<const uint16_t*>(a.in) + tile * a.in_tile +
                         int64_t(n) * a.Cin * plane;
    const uint16_t* w = static_cast<const uint16_t*>(a.w);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int row_in0 = u0 * a.istr + a.base_r;
    const int col_in0 = v0 * a.istr + a.base_c;

    floatx16 acc[NOB][2];
#pragma unroll
    for (int i = 0; i < NOB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(in), 0, RB ? int(a.Cin * plane * 2) : 0, kRWord3c);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(w), 0, RB ? a.wK * a.wC * a.R * a.S * 2 : 0, kRWord3c);
    for (int c0 = 0; c0 < a.Cin; c0 += CC) {
        __syncthreads();
        // weights: one 8-channel vector per (group, output channel)
        auto w_item = [&](int e, int j) -> int64_t {   // element offset of element j of item e, or -1
            const int g = e / OB, ol = e - g * OB;
            const int t = g / CCG, cb = g - t * CCG;
            const int tr = t / a.Ts, ts = t - tr * a.Ts;
            const int o = o0 + ol, ci = c0 + cb * 8 + j;
            const int wr = a.wr0 + a.wrstep * tr, ws = a.ws0 + a.wsstep * ts;
            return (o < a.Cout && ci < a.Cin) ? o * a.w_os + ci * a.w_cs + wr * a.S + ws : -1;
        };
        // input patch, transposed to channel-innermost
        auto p_item = [&](int e, int64_t& pix, int& cbase, int& slot) {   // pix < 0: outside the tile
            const int pc = e % PC;
            const int rest = e / PC;
            const int cg = rest % CCG, pr = rest / CCG;
            const int gr = row_in0 + pr, gc = col_in0 + pc;
            const bool ok = gr >= 0 && gr < a.in_rows && gc >= 0 && gc < a.in_cols;
            pix = ok ? int64_t(gr) * a.in_pitch + gc : -1;
            cbase = c0 + cg * 8;
            slot = (pr * PC + pc) * PS + cg * 8;
        };
        if constexpr (RB) {
            const int nw = G * OB, np = PR * CCG * PC;
            for (int e0 = tid; e0 < nw; e0 += kThreads * kUB) {
                Pack8 v[kUB];
#pragma unroll
                for (int q = 0; q < kUB; ++q) {
                    const int e = e0 + q * kThreads;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        // past the end: an out-of-range load, no memory access
                        const int64_t off = e < nw ? w_item(e, j) : -1;
                        v[q].h[j] = __builtin_amdgcn_raw_buffer_load_b16(rw, off >= 0 ? 2 * int(off) : kOOBc, 0, 0);
                    }
                }
#pragma unroll
                for (int q = 0; q < kUB; ++q)
                    if (e0 + q * kThreads < nw) *reinterpret_cast<uint4*>(wl + (e0 + q * kThreads) * 8) = v[q].v;
            }
            for (int e0 = tid; e0 < np; e0 += kThreads * kUB) {
                Pack8 v[kUB];
                int slot[kUB];
#pragma unroll
                for (int q = 0; q < kUB; ++q) {
                    const int e = e0 + q * kThreads;
                    int64_t pix = -1;   // past the end: out-of-range loads
                    int cbase = 0;
                    slot[q] = -1;
                    if (e < np) p_item(e, pix, cbase, slot[q]);
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int ci = cbase + j;
                        const int off = (pix >= 0 && ci < a.Cin) ? 2 * int(ci * plane + pix) : kOOBc;
                        v[q].h[j] = __builtin_amdgcn_raw_buffer_load_b16(rin, off, 0, 0);
                    }
                }
#pragma unroll
                for (int q = 0; q < kUB; ++q)
                    if (slot[q] >= 0) *reinterpret_cast<uint4*>(pl + slot[q]) = v[q].v;
            }
        } else {
            for (int e = tid; e < G * OB; e += kThreads) {
                Pack8 p;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int64_t off = w_item(e, j);
                    p.h[j] = off >= 0 ? w[off] : uint16_t(0);
                }
                *reinterpret_cast<uint4*>(wl + e * 8) = p.v;
            }
            for (int e = tid; e < PR * CCG * PC; e += kThreads) {
                int64_t pix;
                int cbase, slot;
                p_item(e, pix, cbase, slot);
                const uint16_t* src = in + pix;
                Pack8 p;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int ci = cbase + j;
                    p.h[j] = (pix >= 0 && ci < a.Cin) ? src[int64_t(ci) * plane] : uint16_t(0);
                }
                *reinterpret_cast<uint4*>(pl + slot) = p.v;
            }
        }
        __syncthreads();

        const int nk = (G + 1) / 2;
        for (int k = 0; k < nk; ++k) {
            const int g = 2 * k + hi;
            bf16x8 A[NOB], B[2];
            if (g < G) {
                const int t = g / CCG, cb = g - t * CCG;
                const int tr = t / a.Ts, ts = t - tr * a.Ts;
#pragma unroll
                for (int ob = 0; ob < NOB; ++ob)
                    A[ob] = *reinterpret_cast<const bf16x8*>(wl + (g * OB + ob * 32 + l32) * 8);
#pragma unroll
                for (int pb = 0; pb < 2; ++pb) {
                    const int pm = (pb * 32 + l32) * a.istr, pw = wave * a.istr;
                    const int prow = (cm ? pm : pw) + tr, pcol = (cm ? pw : pm) + ts;
                    B[pb] = *reinterpret_cast<const bf16x8*>(pl + (prow * PC + pcol) * PS + cb * 8);
                }
            } else {
#pragma unroll
                for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
                    for (int j = 0; j < 8; ++j) A[ob][j] = __bf16(0.f);
#pragma unroll
                for (int pb = 0; pb < 2; ++pb)
#pragma unroll
                    for (int j = 0; j < 8; ++j) B[pb][j] = __bf16(0.f);
            }
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
                for (int pb = 0; pb < 2; ++pb)
                    acc[ob][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[ob], B[pb], acc[ob][pb], 0, 0, 0);
        }
    }

    // D layout of a 32x32 MFMA tile: value i of lane l is row 8*(i/4) + 4*(l/32) + i%4,
    // column l%32.  Rows are output channels, columns pixels.
    float* out = a.out + tile * a.out_tile + int64_t(n) * a.Cout * a.out_rows * a.out_cols;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
            const int u = cm ? u0 + pb * 32 + l32 : u0 + wave;
            const int v = cm ? v0 + wave : v0 + pb * 32 + l32;
            if (u >= uend || v >= vend) continue;
            const int orow = u * a.ostr + a.oph_r;
            const int ocol = v * a.ostr + a.oph_c;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int o = o0 + ob * 32 + 8 * (i / 4) + 4 * hi + (i % 4);
                if (o < a.Cout)
                    out[(int64_t(o) * a.out_rows + orow) * a.out_cols + ocol] = acc[ob][pb][i];
            }
        }
}

template <int OB, bool RB>
__global__ __launch_bounds__(kThreads) void igemm_f32_kernel(IgemmArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int NOB = OB / 32;
    int u0, v0, uend, vend;
    bool cm;
    block_origin(a, u0, v0, uend, vend, cm);
    const int CC = a.CC;
    const int Tt = a.Tr * a.Ts;
    const int KG = Tt * CC;
    const int PR = ((cm ? kBW : kBH) - 1) * a.istr + a.Tr;
    const int PC = ((cm ? kBH : kBW) - 1) * a.istr + a.Ts;
    const int PLN = f32_plane_stride(patch_pixels(a));
    float* wl = reinterpret_cast<float*>(smem);   // [KG][OB]
    float* pl = wl + KG * OB;                     // [CC][PLN] with rows of PC

    const int o0 = blockIdx.y * OB;
    const int tile = blockIdx.z / a.Nn, n = blockIdx.z % a.Nn;

    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const float* in = static_cast<const float*>(a.in) + tile * a.in_tile +
                      int64_t(n) * a.Cin * plane;
    const float* w = static_cast<const float*>(a.w);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int row_in0 = u0 * a.istr + a.base_r;
    const int col_in0 = v0 * a.istr + a.base_c;

    floatx16 acc[NOB][2];
#pragma unroll
    for (int i = 0; i < NOB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(in), 0, RB ? int(a.Cin * plane * 4) : 0, kRWord3c);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(w), 0, RB ? a.wK * a.wC * a.R * a.S * 4 : 0, kRWord3c);
    for (int c0 = 0; c0 < a.Cin; c0 += CC) {
        __syncthreads();
        auto w_item = [&](int e) -> int64_t {   // element offset of weight item e, or -1
            const int kg = e / OB, ol = e - kg * OB;
            const int t = kg / CC, cl = kg - t * CC;
            const int tr = t / a.Ts, ts = t - tr * a.Ts;
            const int o = o0 + ol, ci = c0 + cl;
            const int wr = a.wr0 + a.wrstep * tr, ws = a.ws0 + a.wsstep * ts;
            return (o < a.Cout && ci < a.Cin) ? o * a.w_os + ci * a.w_cs + wr * a.S + ws : -1;
        };
        auto p_item = [&](int e, int& slot) -> int64_t {   // element offset of patch item e, or -1
            const int pc = e % PC;
            const int rest = e / PC;
            const int pr = rest % PR, cl = rest / PR;
            const int gr = row_in0 + pr, gc = col_in0 + pc, ci = c0 + cl;
            const bool ok = gr >= 0 && gr < a.in_rows && gc >= 0 && gc < a.in_cols && ci < a.Cin;
            slot = cl * PLN + pr * PC + pc;
            return ok ? ci * plane + int64_t(gr) * a.in_pitch + gc : -1;
        };
        if constexpr (RB) {
            const int nw = KG * OB, np = CC * PR * PC;
            for (int e0 = tid; e0 < nw; e0 += kThreads * kUF) {
                float v[kUF];
#pragma unroll
                for (int q = 0; q < kUF; ++q) {
                    // past the end: an out-of-range load, no memory access
                    const int64_t off = e0 + q * kThreads < nw ? w_item(e0 + q * kThreads) : -1;
                    v[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                        rw, off >= 0 ? 4 * int(off) : kOOBc, 0, 0));
                }
#pragma unroll
                for (int q = 0; q < kUF; ++q)
                    if (e0 + q * kThreads < nw) wl[e0 + q * kThreads] = v[q];
            }
            for (int e0 = tid; e0 < np; e0 += kThreads * kUF) {
                float v[kUF];
                int slot[kUF];
#pragma unroll
                for (int q = 0; q < kUF; ++q) {
                    const int e = e0 + q * kThreads;
                    int64_t off = -1;   // past the end: an out-of-range load, no memory access
                    slot[q] = -1;
                    if (e < np) off = p_item(e, slot[q]);
                    v[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                        rin, off >= 0 ? 4 * int(off) : kOOBc, 0, 0));
                }
#pragma unroll
                for (int q = 0; q < kUF; ++q)
                    if (slot[q] >= 0) pl[slot[q]] = v[q];
            }
        } else {
            for (int e = tid; e < KG * OB; e += kThreads) {
                const int64_t off = w_item(e);
                wl[e] = off >= 0 ? w[off] : 0.f;
            }
            for (int e = tid; e < CC * PR * PC; e += kThreads) {
                int slot;
                const int64_t off = p_item(e, slot);
                pl[slot] = off >= 0 ? in[off] : 0.f;
            }
        }
        __syncthreads();

        // k-steps: (tap t, channel pair c2) with t-major order, channels 2 c2
        // (lanes 0-31) and 2 c2 + 1 (lanes 32-63); CC is even, so a step's
        // two channels share the tap.  The tap and its (tr, ts) advance
        // incrementally, four steps per pass so that their operand reads can
        // be issued ahead of the MFMAs.
        const int CCH = CC / 2, nk = Tt * CCH;
        int c2 = 0, t = 0, tr = 0, ts = 0;
        auto kstep = [&]() __attribute__((always_inline)) {
            const int cl = 2 * c2 + hi, kg = t * CC + cl;
            float A[NOB], B[2];
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob) A[ob] = wl[kg * OB + ob * 32 + l32];
#pragma unroll
            for (int pb = 0; pb < 2; ++pb) {
                const int pm = (pb * 32 + l32) * a.istr, pw = wave * a.istr;
                const int prow = (cm ? pm : pw) + tr, pcol = (cm ? pw : pm) + ts;
                B[pb] = pl[cl * PLN + prow * PC + pcol];
            }
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
                for (int pb = 0; pb < 2; ++pb)
                    acc[ob][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(A[ob], B[pb], acc[ob][pb], 0, 0, 0);
            const bool wrap = ++c2 == CCH;
            c2 = wrap ? 0 : c2;
            t += wrap ? 1 : 0;
            const bool rwrap = wrap && ++ts == a.Ts;
            ts = rwrap ? 0 : ts;
            tr += rwrap ? 1 : 0;
        };
        int k = 0;
        for (; k + 4 <= nk; k += 4) { kstep(); kstep(); kstep(); kstep(); }
        for (; k < nk; ++k) kstep();
    }

    float* out = a.out + tile * a.out_tile + int64_t(n) * a.Cout * a.out_rows * a.out_cols;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
            const int u = cm ? u0 + pb * 32 + l32 : u0 + wave;
            const int v = cm ? v0 + wave : v0 + pb * 32 + l32;
            if (u >= uend || v >= vend) continue;
            const int orow = u * a.ostr + a.oph_r;
            const int ocol = v * a.ostr + a.oph_c;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int o = o0 + ob * 32 + 8 * (i / 4) + 4 * hi + (i % 4);
                if (o < a.Cout)
                    out[(int64_t(o) * a.out_rows + orow) * a.out_cols + ocol] = acc[ob][pb][i];
            }
        }
}

static int lds_bytes_for(const IgemmArgs& a, int dtype, int CC, int OB) {
    const int Tt = a.Tr * a.Ts;
    if (dtype == 1) {
        const int G = Tt * (CC / 8);
        return G * OB * 16 + patch_pixels(a) * bf16_pixel_stride(CC) * 2;
    }
    return (Tt * CC * OB + CC * f32_plane_stride(patch_pixels(a))) * 4;
}

void igemm_set_frame(IgemmArgs& a, const int bands[4]) {
    a.frame = 1;
    a.fseg = 0;
    const int top = std::min(bands[0], a.Uo), bot = std::min(bands[1], a.Uo - top);
    const int mid = a.Uo - top - bot;
    const int left = std::min(bands[2], a.Vo), right = std::min(bands[3], a.Vo - left);
    auto add = [&](int u0, int nu, int v0, int nv, int cm) {
        if (nu <= 0 || nv <= 0) return;
        const int k = a.fseg++;
        a.fu0[k] = u0; a.fnu[k] = nu; a.fv0[k] = v0; a.fnv[k] = nv; a.fcm[k] = cm;
    };
    add(0, top, 0, a.Vo, 0);                 // rows above the interior, full width
    add(a.Uo - bot, bot, 0, a.Vo, 0);        // rows below
    add(top, mid, 0, left, 1);               // columns left of the interior
    add(top, mid, a.Vo - right, right, 1);   // columns right
    a.fblk[0] = 0;
    for (int k = 0; k < a.fseg; ++k) {
        const int bh = a.fcm[k] ? kBW : kBH, bw = a.fcm[k] ? kBH : kBW;
        a.fblk[k + 1] = a.fblk[k] + ((a.fnu[k] + bh - 1) / bh) * ((a.fnv[k] + bw - 1) / bw);
    }
}

bool igemm_plan(IgemmArgs& a, int dtype) {
    a.kind = 0;
    // a merged-phase backward-data request runs on the register-weight kernel or not at all
    if (a.bp) return dtype == 1 && igemm_wreg_plan(a);
    // a frame runs on the frame kernel, else on the chunked kernel (the strip
    // kernels cover whole tiles)
    if (a.frame && igemm_frame_plan(a, dtype)) return true;
    if (!a.frame) {
        if (dtype == 1 && igemm_roll_plan(a)) return true;
        if (dtype == 1 && igemm_wreg_plan(a)) return true;
        if (dtype == 0 && igemm_f32w_plan(a)) return true;
    }
    a.OB = a.Cout <= 32 ? 32 : 64;
    // channel-chunk candidates, widest first: the channel count itself (rounded
    // to the k-granularity) when it is small, then powers of two
    const int gran = dtype == 1 ? 8 : 2;
    const int maxcc = dtype == 1 ? 64 : 32;
    const int cin_r = (a.Cin + gran - 1) / gran * gran;
    int cands[8], nc = 0;
    cands[nc++] = std::min(cin_r, maxcc);
    for (int c = maxcc; c >= gran; c /= 2)
        if (c < cands[0]) cands[nc++] = c;
    // prefer two workgroups per CU (<= 80 KB of LDS), else the device limit;
    // a grid of at most one workgroup per CU takes the widest chunk the
    // device allows (fewer chunks: fewer staging rounds and barriers)
    const int limit = device_lds_limit();
    const int64_t nwg = int64_t(a.frame ? a.fblk[a.fseg] : ((a.Vo + kBW - 1) / kBW) * ((a.Uo + kBH - 1) / kBH)) *
                        ((a.Cout + a.OB - 1) / a.OB) * a.ntiles * a.Nn;
    const int small = nwg <= device_cu_count() ? limit : std::min(80 * 1024, limit);
    for (int budget : {small, limit}) {
        for (int i = 0; i < nc; ++i) {
            const int b = lds_bytes_for(a, dtype, cands[i], a.OB);
            if (b <= budget) {
                a.CC = cands[i];
                a.lds_bytes = b;
                return true;
            }
        }
    }
    return false;
}

hipError_t launch_igemm(const IgemmArgs& a, int dtype, hipStream_t s) {
    if (a.kind == 1) return launch_igemm_wreg(a, s);
    if (a.kind == 2) return launch_igemm_f32w(a, s);
    if (a.kind == 3) return launch_igemm_roll(a, s);
    if (a.kind == 4) return launch_igemm_frame(a, dtype, s);
    const int nvb = (a.Vo + kBW - 1) / kBW, nub = (a.Uo + kBH - 1) / kBH;
    dim3 grid(a.frame ? a.fblk[a.fseg] : nvb * nub, (a.Cout + a.OB - 1) / a.OB, a.ntiles * a.Nn);
    if (grid.x == 0) return hipSuccess;   // an empty frame
    dim3 block(kThreads);
    // buffer loads when the sample's input and the weights are under 2^31 bytes
    const int64_t es = dtype == 1 ? 2 : 4;
    const bool rb = int64_t(a.Cin) * a.in_rows * a.in_pitch * es < kOOBc &&
                    int64_t(a.wK) * a.wC * a.R * a.S * es < kOOBc;
    const void* f;
    if (dtype == 1)
        f = a.OB == 32 ? (rb ? reinterpret_cast<const void*>(igemm_bf16_kernel<32, true>)
                             : reinterpret_cast<const void*>(igemm_bf16_kernel<32, false>))
                       : (rb ? reinterpret_cast<const void*>(igemm_bf16_kernel<64, true>)
                             : reinterpret_cast<const void*>(igemm_bf16_kernel<64, false>));
    else
        f = a.OB == 32 ? (rb ? reinterpret_cast<const void*>(igemm_f32_kernel<32, true>)
                             : reinterpret_cast<const void*>(igemm_f32_kernel<32, false>))
                       : (rb ? reinterpret_cast<const void*>(igemm_f32_kernel<64, true>)
                             : reinterpret_cast<const void*>(igemm_f32_kernel<64, false>));
    if (a.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    IgemmArgs ak = a;
    void* args[] = {&ak};
    return hipLaunchKernel(f, grid, block, args, a.lds_bytes, s);
}

}  // namespace dc
