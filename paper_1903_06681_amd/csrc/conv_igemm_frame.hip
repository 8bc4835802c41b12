// Boundary frame of a tile, bf16 (the outputs of Eqs. (1) / (3) whose window
// reads a halo margin; Sec. IV-A computes them after the exchange, the
// interior before it).
//
// The frame is a few output lines (the rows of the top and bottom bands, the
// columns of the left and right bands), each one output pixel wide.  A
// workgroup computes 32 consecutive outputs of one line for 32 output
// channels: one 32x32 MFMA tile, D[o][pixel] = sum_kg A[o][kg] B[kg][pixel]
// with kg = (tap, input channel) as in the whole-tile kernels.  The four
// waves split the reduction over kg (k-steps w, w+4, ...) and sum their tiles
// through LDS, so that a frame of ~1,000 pixels per image and 64 channels
// still spreads over a few hundred workgroups.
//
// Per channel chunk the weights of the block ([o][tap, 8-channel group][8])
// and the input window of the line piece (along x across x channels,
// channel-innermost) are gathered from NCHW with 2-byte buffer loads: an
// element outside the tensors (padding channels, rows or columns past the
// tile) is a load past the buffer's end, which returns zero, so the loads of
// a thread's batch carry no branches and are all issued before the first one
// is waited for, which is what a latency-bound launch of this size needs.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "bf16util.h"
#include "kernels.h"

namespace dc {

namespace {

constexpr int kThreads = 256;
constexpr int kPiece = 32;   // outputs of a line per workgroup (MFMA columns)
constexpr int kOB = 32;      // output channels per workgroup (MFMA rows)
constexpr int kWB = 9;       // weight items (8 loads each) per thread per batch
constexpr int kPB = 4;       // window items per thread per batch
constexpr int kWord3 = 0x00020000;   // buffer resource word 3 (gfx9 family: raw access)
constexpr int kOOB = 0x7fffffff;     // byte offset past every buffer here: the load returns 0
typedef unsigned f_v4u __attribute__((ext_vector_type(4)));

// Slots (16 bytes each) per output channel of the weight block: odd, so that
// 32 lanes reading one slot of consecutive channels hit distinct bank groups.
__host__ __device__ inline int frame_gp(int G) { return G | 1; }
// Window pixel stride (bf16 elements): an odd number of 16-byte units.
__host__ __device__ inline int frame_ps(int CC) { return 8 * ((CC / 8) | 1); }

// LDS elements of the weight block: the gathered [kOB][GP][8] layout or the
// raw rows (kOB rows of CC*Tt, or CC rows of kOB*Tt, plus 2 elements each),
// whichever is larger, rounded to 16 bytes
__host__ __device__ inline int frame_wl_elems(int Tt, int CC) {
    const int gathered = kOB * frame_gp(Tt * (CC / 8)) * 8;
    const int raw = kOB * CC * Tt + 2 * (kOB > CC ? kOB : CC);
    const int m = gathered > raw ? gathered : raw;
    return (m + 7) / 8 * 8;
}

int frame_lds(const IgemmArgs& a, int CC) {
    // window of a row line, of a column line: (along) x (across) pixels
    const int win = std::max((kPiece - 1 + a.Ts) * a.Tr, (kPiece - 1 + a.Tr) * a.Ts) * frame_ps(CC) * 2;
    // the reduction of the four waves' tiles reuses the space (16 KB)
    return std::max(frame_wl_elems(a.Tr * a.Ts, CC) * 2 + win, 4 * 1024 * 4);
}

}  // namespace

// TR, TS: filter taps (rows, columns) of the launch; CCG: 8-channel groups
// per chunk.  Non-zero values make every index division one by a constant
// and let the k-loop unroll; 0 takes the value from the arguments.  FULL:
// every channel chunk and output-channel block is whole (Cin a multiple of
// the chunk, Cout of 32) and the weight rows start on 16 bytes (C*R*S a
// multiple of 8): the block's weights are then copied as they lie in memory
// (rows of [ci][tap] per output channel in the forward layout, of [o][tap]
// per input channel in the backward-data layout) with 16-byte loads, and the
// A operand is gathered from LDS instead; a window load needs no channel
// check and the channel step of an item's 8 loads goes in the uniform offset.
template <int TR, int TS, int CCG_, bool FULL>
__global__ __launch_bounds__(kThreads) void igemm_frame_bf16_kernel(IgemmArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int Tr = TR > 0 ? TR : a.Tr, Ts = TS > 0 ? TS : a.Ts;
    const int CCG = CCG_ > 0 ? CCG_ : a.CC / 8, CC = CCG * 8;
    // segment, line and piece of this workgroup
    int sg = 0;
    while (sg + 1 < a.fseg && int(blockIdx.x) >= a.fblk[sg + 1]) ++sg;
    const bool cm = a.fcm[sg] != 0;   // a column of the left / right band
    const int len = cm ? a.fnu[sg] : a.fnv[sg];
    const int npc = (len + kPiece - 1) / kPiece;
    const int local = blockIdx.x - a.fblk[sg];
    const int line = local / npc, p0 = (local - line * npc) * kPiece;
    const int n_out = min(kPiece, len - p0);
    // first output pixel (u, v) of the piece; the line runs along v (rows of
    // the frame) or along u (columns)
    const int u = a.fu0[sg] + (cm ? p0 : line);
    const int v = a.fv0[sg] + (cm ? line : p0);

    // window extent along the line and across it
    const int PA = (kPiece - 1) + (cm ? Tr : Ts), TA = cm ? Ts : Tr;
    const int Tt = Tr * Ts, G = Tt * CCG, GP = frame_gp(G);
    const int PS = frame_ps(CC);
    // weights: [kOB][GP][8] (gathered) or raw rows of RSW elements (FULL)
    uint16_t* wl = reinterpret_cast<uint16_t*>(smem);
    uint16_t* pl = wl + frame_wl_elems(Tt, CC);          // [PA][TA][PS]
    // raw rows: nrow rows of L elements (8-element chunks), stride RSW
    const int L = a.wmode ? kOB * Tt : CC * Tt, nrow = a.wmode ? CC : kOB;
    const int RSW = L + 2;
    const int SO = a.wmode ? Tt : RSW, SC = a.wmode ? RSW : Tt;   // o, ci strides in the rows

    const int o0 = blockIdx.y * kOB;
    const int tile = blockIdx.z / a.Nn, n = blockIdx.z % a.Nn;
    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const uint16_t* in = static_cast<const uint16_t*>(a.in) + tile * a.in_tile + int64_t(n) * a.Cin * plane;
    const __amdgpu_buffer_rsrc_t rin =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(in), 0, int(a.Cin * plane * 2), kWord3);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.w), 0, a.wK * a.wC * a.R * a.S * 2, kWord3);
    const int w_os = int(a.w_os), w_cs = int(a.w_cs), iplane = int(plane);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int row0 = u + a.base_r, col0 = v + a.base_c;   // window origin (stride 1)

    floatx16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;

    const int nw = kOB * G, np = PA * TA * CCG;
    for (int c0 = 0; c0 < a.Cin; c0 += CC) {
        __syncthreads();
        if constexpr (FULL) {
            // 16-byte chunks of the raw rows: row (output channel o0 + row,
            // or input channel c0 + row), elements [8 c8, 8 c8 + 8) of it
            const int n8 = L / 8, nwc = nrow * n8;
            for (int e0 = tid; e0 < nwc; e0 += kThreads * kWB) {
                f_v4u v[kWB];
                int dst[kWB];
#pragma unroll
                for (int q = 0; q < kWB; ++q) {
                    const int e = e0 + q * kThreads;
                    const int ec = min(e, nwc - 1);
                    const int row = a.wmode ? ec / (kOB * Tt / 8) : ec / (CCG * Tt);
                    const int c8 = ec - row * n8;
                    const int gbase = a.wmode ? (c0 + row) * w_cs + o0 * Tt : (o0 + row) * w_os + c0 * Tt;
                    v[q] = __builtin_amdgcn_raw_buffer_load_b128(rw, 2 * (gbase + c8 * 8), 0, 0);
                    dst[q] = e < nwc ? row * RSW + c8 * 8 : -1;
                }
#pragma unroll
                for (int q = 0; q < kWB; ++q)
                    if (dst[q] >= 0) {
                        // rows start on 4 bytes (RSW / 2 odd: the operand
                        // gathers of 32 consecutive rows hit distinct banks)
                        uint32_t* d = reinterpret_cast<uint32_t*>(wl + dst[q]);
                        d[0] = v[q].x; d[1] = v[q].y; d[2] = v[q].z; d[3] = v[q].w;
                    }
            }
        } else {
            // gathered: item (output channel ol, group g = tap * CCG + cb), 8
            // input channels; in the forward layout a channel's taps and input
            // channels are contiguous (g runs fastest), in the backward-data
            // layout the output channels are (ol runs fastest)
            for (int e0 = tid; e0 < nw; e0 += kThreads * kWB) {
                Pack8 p[kWB];
                int slot[kWB];
#pragma unroll
                for (int q = 0; q < kWB; ++q) {
                    const int e = e0 + q * kThreads;
                    const int ec = min(e, nw - 1);
                    int ol, g;
                    if (a.wmode == 0) { ol = ec / G; g = ec - ol * G; }
                    else { g = ec / kOB; ol = ec - g * kOB; }
                    const int t = g / CCG, cb = g - t * CCG;
                    const int tr = t / Ts, ts = t - tr * Ts;
                    const int o = o0 + ol;
                    const int wr = a.wr0 + a.wrstep * tr, ws = a.ws0 + a.wsstep * ts;
                    const int base = o * w_os + wr * a.S + ws;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int ci = c0 + cb * 8 + j;
                        const int off = (o < a.Cout && ci < a.Cin) ? 2 * (base + ci * w_cs) : kOOB;
                        p[q].h[j] = __builtin_amdgcn_raw_buffer_load_b16(rw, off, 0, 0);
                    }
                    slot[q] = e < nw ? (ol * GP + g) * 8 : -1;
                }
#pragma unroll
                for (int q = 0; q < kWB; ++q)
                    if (slot[q] >= 0) *reinterpret_cast<uint4*>(wl + slot[q]) = p[q].v;
            }
        }
        // input window: item (along, across, channel group), 8 channels;
        // the memory-contiguous coordinate (input column) runs fastest
        for (int e0 = tid; e0 < np; e0 += kThreads * kPB) {
            Pack8 p[kPB];
            int slot[kPB];
#pragma unroll
            for (int q = 0; q < kPB; ++q) {
                const int e = e0 + q * kThreads;
                const int ec = min(e, np - 1);
                int al, ac, cg;
                if (!cm) { al = ec % PA; const int r = ec / PA; ac = r % TA; cg = r / TA; }
                else { ac = ec % TA; const int r = ec / TA; al = r % PA; cg = r / PA; }
                const int gr = row0 + (cm ? al : ac), gc = col0 + (cm ? ac : al);
                const bool ok = gr >= 0 && gr < a.in_rows && gc >= 0 && gc < a.in_cols;
                const int pix = gr * a.in_pitch + gc;
                if constexpr (FULL) {
                    // an element outside the tile: an offset past the buffer
                    // (whether or not the uniform offset counts in the check)
                    const int off = ok ? 2 * ((c0 + cg * 8) * iplane + pix) : kOOB;
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        p[q].h[j] = __builtin_amdgcn_raw_buffer_load_b16(rin, off, 2 * j * iplane, 0);
                } else {
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int ci = c0 + cg * 8 + j;
                        const int off = (ok && ci < a.Cin) ? 2 * (ci * iplane + pix) : kOOB;
                        p[q].h[j] = __builtin_amdgcn_raw_buffer_load_b16(rin, off, 0, 0);
                    }
                }
                slot[q] = e < np ? (al * TA + ac) * PS + cg * 8 : -1;
            }
#pragma unroll
            for (int q = 0; q < kPB; ++q)
                if (slot[q] >= 0) *reinterpret_cast<uint4*>(pl + slot[q]) = p[q].v;
        }
        __syncthreads();

        // k-steps of this wave: k = wave + 4 i, groups 2k (lanes 0-31) and
        // 2k+1 (lanes 32-63); a group past the last reads group 0 and
        // multiplies zeros
        const int nkw = ((G + 1) / 2 + 3) / 4;
        auto kstep = [&](int i) {
            const int g = 2 * (wave + 4 * i) + hi;
            const bool live = g < G;
            const int gg = live ? g : 0;
            const int t = gg / CCG, cb = gg - t * CCG;
            const int tr = t / Ts, ts = t - tr * Ts;
            Pack8 A, B;
            if constexpr (FULL) {
                const int tap = (a.wr0 + a.wrstep * tr) * a.S + (a.ws0 + a.wsstep * ts);
                const uint16_t* src = wl + l32 * SO + cb * 8 * SC + tap;
#pragma unroll
                for (int j = 0; j < 8; ++j) A.h[j] = src[j * SC];
            } else {
                A.v = *reinterpret_cast<const uint4*>(wl + (l32 * GP + gg) * 8);
            }
            const int al = l32 + (cm ? tr : ts), ac = cm ? ts : tr;
            B.v = *reinterpret_cast<const uint4*>(pl + (al * TA + ac) * PS + cb * 8);
            if (!live) A.v = make_uint4(0, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A.b, B.b, acc, 0, 0, 0);
        };
        if constexpr (TR > 0 && TS > 0 && CCG_ > 0) {
#pragma unroll
            for (int i = 0; i < nkw; ++i) kstep(i);
        } else {
            for (int i = 0; i < nkw; ++i) kstep(i);
        }
    }

    // sum the four waves' tiles: red[wave][value i][lane]
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int i = 0; i < 16; ++i) red[(wave * 16 + i) * 64 + lane] = acc[i];
    __syncthreads();
    // thread (q = wave, lane) sums values i = q + 4 m: output channel
    // 8 m + 4 (lane / 32) + q, pixel lane % 32 (MFMA D layout)
    float* out = a.out + tile * a.out_tile + int64_t(n) * a.Cout * a.out_rows * a.out_cols;
    if (l32 < n_out) {
        const int pu = cm ? u + l32 : u, pv = cm ? v : v + l32;
        const int orow = pu * a.ostr + a.oph_r, ocol = pv * a.ostr + a.oph_c;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int i = wave + 4 * m;
            const float s = red[(0 * 16 + i) * 64 + lane] + red[(1 * 16 + i) * 64 + lane] +
                            red[(2 * 16 + i) * 64 + lane] + red[(3 * 16 + i) * 64 + lane];
            const int o = o0 + 8 * m + 4 * hi + wave;
            if (o < a.Cout) out[(int64_t(o) * a.out_rows + orow) * a.out_cols + ocol] = s;
        }
    }
}

bool igemm_frame_plan(IgemmArgs& a) {
    if (!a.frame || a.istr != 1 || a.Tr * a.Ts == 0 || a.bp) return false;
    // byte offsets of the buffer loads are 32-bit
    if (int64_t(a.Cin) * a.in_rows * a.in_pitch * 2 >= kOOB ||
        int64_t(a.wK) * a.wC * a.R * a.S * 2 >= kOOB)
        return false;
    const int cin_r = (a.Cin + 7) / 8 * 8;
    const int limit = device_lds_limit();
    int cands[4] = {std::min(cin_r, 64), 32, 16, 8}, nc = 0;
    for (int i = 0; i < 4; ++i)
        if (i == 0 || cands[i] < cands[0]) cands[nc++] = cands[i];
    for (int budget : {std::min(80 * 1024, limit), limit}) {
        for (int i = 0; i < nc; ++i) {
            const int b = frame_lds(a, cands[i]);
            if (b <= budget) {
                a.CC = cands[i];
                a.lds_bytes = b;
                a.OB = kOB;
                a.kind = 4;
                // workgroups: one per (line, 32-output piece) of each segment
                a.fblk[0] = 0;
                for (int k = 0; k < a.fseg; ++k) {
                    const int lines = a.fcm[k] ? a.fnv[k] : a.fnu[k];
                    const int len = a.fcm[k] ? a.fnu[k] : a.fnv[k];
                    a.fblk[k + 1] = a.fblk[k] + lines * ((len + kPiece - 1) / kPiece);
                }
                return true;
            }
        }
    }
    return false;
}

template <int TR, int TS, int CCG, bool FULL>
static hipError_t launch_frame_f(const IgemmArgs& a, dim3 grid, hipStream_t s) {
    const void* f = reinterpret_cast<const void*>(igemm_frame_bf16_kernel<TR, TS, CCG, FULL>);
    if (a.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((igemm_frame_bf16_kernel<TR, TS, CCG, FULL>), grid, dim3(kThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

template <int TR, int TS, int CCG>
static hipError_t launch_frame_t(const IgemmArgs& a, dim3 grid, hipStream_t s) {
    if (a.Cin % a.CC == 0 && a.Cout % kOB == 0 && (int64_t(a.wC) * a.R * a.S) % 8 == 0)
        return launch_frame_f<TR, TS, CCG, true>(a, grid, s);
    return launch_frame_f<TR, TS, CCG, false>(a, grid, s);
}

template <int T>
static hipError_t launch_frame_taps(const IgemmArgs& a, dim3 grid, hipStream_t s) {
    switch (a.CC / 8) {
        case 8: return launch_frame_t<T, T, 8>(a, grid, s);
        case 4: return launch_frame_t<T, T, 4>(a, grid, s);
        case 2: return launch_frame_t<T, T, 2>(a, grid, s);
        case 1: return launch_frame_t<T, T, 1>(a, grid, s);
        default: return launch_frame_t<0, 0, 0>(a, grid, s);
    }
}

hipError_t launch_igemm_frame(const IgemmArgs& a, hipStream_t s) {
    dim3 grid(a.fblk[a.fseg], (a.Cout + kOB - 1) / kOB, a.ntiles * a.Nn);
    if (grid.x == 0) return hipSuccess;   // an empty frame
    if (a.Tr == 3 && a.Ts == 3) return launch_frame_taps<3>(a, grid, s);
    if (a.Tr == 5 && a.Ts == 5) return launch_frame_taps<5>(a, grid, s);
    if (a.Tr == 7 && a.Ts == 7) return launch_frame_taps<7>(a, grid, s);
    return launch_frame_t<0, 0, 0>(a, grid, s);
}

}  // namespace dc
