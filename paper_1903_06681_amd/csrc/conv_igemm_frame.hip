// Boundary frame of a tile, bf16 and fp32 (the outputs of Eqs. (1) / (3)
// whose window reads a halo margin; Sec. IV-A computes them after the
// exchange, the interior before it).
//
// The frame is a few output lines (the rows of the top and bottom bands, the
// columns of the left and right bands), each one output pixel wide.  A
// workgroup computes 32 consecutive outputs of one line for 32 output
// channels: one 32x32 MFMA tile, D[o][pixel] = sum_kg A[o][kg] B[kg][pixel]
// with kg = (tap, input channel) as in the whole-tile kernels.  Its waves
// (four for bf16, eight for fp32) split the reduction over kg and sum their
// tiles through LDS, so that a frame of ~1,000 pixels per image and 64
// channels still spreads over a few hundred workgroups.
//
// bf16: per channel chunk the weights of the block ([o][tap, 8-channel group][8])
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
// fp32: eight waves (two per SIMD: a frame of a small layer is few
// workgroups, whose staging is VALU work), and the elements per thread and
// batch of the weights and the window
constexpr int kWavesF = 8, kThreadsF = 64 * kWavesF;
constexpr int kWF = 20;
constexpr int kPF = 8;
// fp32 weight row stride (floats): one more than the 32 output channels, so
// that the stores of items along a weight row (different k, one channel)
// fall in different banks
constexpr int kWS = kOB + 1;
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

// fp32: weights [Tt * CC][kWS] and the larger window [CC][PA][TA] floats
int frame_lds_f32(const IgemmArgs& a, int CC) {
    const int Tt = a.Tr * a.Ts;
    const int win = std::max((kPiece - 1 + a.Ts) * a.Tr, (kPiece - 1 + a.Tr) * a.Ts) * CC;
    return std::max((Tt * CC * kWS + win) * 4, kWavesF * 4 * 1024);
}

int frame_lds(const IgemmArgs& a, int CC) {
    // window of a row line, of a column line: (along) x (across) pixels
    const int win = std::max((kPiece - 1 + a.Ts) * a.Tr, (kPiece - 1 + a.Tr) * a.Ts) * frame_ps(CC) * 2;
    // the reduction of the four waves' tiles reuses the space (16 KB)
    return std::max(frame_wl_elems(a.Tr * a.Ts, CC) * 2 + win, 4 * 1024 * 4);
}

}  // namespace

// Sums the NWV waves' tiles through LDS (red[wave][value i][lane], NWV * 4
// KB at the start of the workgroup's LDS, after a barrier) and stores the
// piece: thread (q = wave, lane) sums values i = q + NWV m, which are
// output channel 8 (i / 4) + 4 (lane / 32) + i % 4, pixel lane % 32 of the
// tile (MFMA D layout), in the order of the waves.
template <int NWV>
__device__ __forceinline__ void frame_sum_store(const IgemmArgs& a, const floatx16& acc, unsigned char* smem,
                                                int tile, int n, int o0, bool cm, int u, int v, int n_out) {
    static_assert(NWV == 4 || NWV == 8, "four or eight waves");
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    __syncthreads();
    float* red = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int i = 0; i < 16; ++i) red[(wave * 16 + i) * 64 + lane] = acc[i];
    __syncthreads();
    float* out = a.out + tile * a.out_tile + int64_t(n) * a.Cout * a.out_rows * a.out_cols;
    if (l32 < n_out) {
        const int pu = cm ? u + l32 : u, pv = cm ? v : v + l32;
        const int orow = pu * a.ostr + a.oph_r, ocol = pv * a.ostr + a.oph_c;
#pragma unroll
        for (int m = 0; m < 16 / NWV; ++m) {
            const int i = wave + NWV * m;
            float s = red[i * 64 + lane];
#pragma unroll
            for (int w = 1; w < NWV; ++w) s += red[(w * 16 + i) * 64 + lane];
            const int o = o0 + 8 * (i / 4) + 4 * hi + i % 4;
            if (o < a.Cout) out[(int64_t(o) * a.out_rows + orow) * a.out_cols + ocol] = s;
        }
    }
}

// n / d and n % d (0 <= n < 2^22, d >= 1) from a float reciprocal of d: the
// product is within one of the quotient, which one correction each way
// makes exact.
__device__ __forceinline__ int frame_divmod(int n, int d, float inv, int& r) {
    int q = int(float(n) * inv);
    r = n - q * d;
    const bool lo = r < 0;
    q -= lo ? 1 : 0;
    r += lo ? d : 0;
    const bool hi = r >= d;
    q += hi ? 1 : 0;
    r -= hi ? d : 0;
    return q;
}

// Segment, line and piece of this workgroup: the line's first output pixel
// (u, v), whether it is a column of the side bands (cm), outputs in the piece.
struct FramePiece {
    int u, v, n_out;
    bool cm;
};

__device__ __forceinline__ FramePiece frame_piece(const IgemmArgs& a) {
    int sg = 0;
    while (sg + 1 < a.fseg && int(blockIdx.x) >= a.fblk[sg + 1]) ++sg;
    FramePiece f;
    f.cm = a.fcm[sg] != 0;
    const int len = f.cm ? a.fnu[sg] : a.fnv[sg];
    const int npc = (len + kPiece - 1) / kPiece;
    const int local = blockIdx.x - a.fblk[sg];
    const int line = local / npc, p0 = (local - line * npc) * kPiece;
    f.n_out = min(kPiece, len - p0);
    f.u = a.fu0[sg] + (f.cm ? p0 : line);
    f.v = a.fv0[sg] + (f.cm ? line : p0);
    return f;
}

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
    const FramePiece fp = frame_piece(a);
    const bool cm = fp.cm;   // a column of the left / right band
    const int u = fp.u, v = fp.v, n_out = fp.n_out;

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

    frame_sum_store<4>(a, acc, smem, tile, n, o0, cm, u, v, n_out);
}

// fp32: v_mfma_f32_32x32x2_f32 (eight waves splitting the reduction), a
// k-step is one (tap, input channel) per half-wave: lanes 0-31 channel 2 c2, lanes 32-63 channel 2 c2 + 1 of one
// tap.  Per chunk of CC channels (even) the weights lie in LDS as
// [tap * CC + ci][32 output channels, padded to 33] and the window as
// [ci][along][across] floats; both are read one float per lane.  Weight items are
// taken in the tensor's own order (a row of the [K][C][R][S] tensor: taps
// and input channels of one output channel forward, taps and output
// channels of one input channel for the input gradient), so the loads are
// contiguous; the tap flip of Eq. (3) is applied when they are placed.
template <int TR, int TS>
__global__ __launch_bounds__(kThreadsF) void igemm_frame_f32_kernel(IgemmArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int Tr = TR > 0 ? TR : a.Tr, Ts = TS > 0 ? TS : a.Ts, Tt = Tr * Ts;
    const int CC = a.CC, CCH = CC / 2;
    const FramePiece fp = frame_piece(a);
    const bool cm = fp.cm;
    const int u = fp.u, v = fp.v, n_out = fp.n_out;
    const int PA = (kPiece - 1) + (cm ? Tr : Ts), TA = cm ? Ts : Tr;
    float* wl = reinterpret_cast<float*>(smem);   // [Tt * CC][kWS]
    float* pl = wl + Tt * CC * kWS;               // [CC][PA][TA]

    const int o0 = blockIdx.y * kOB;
    const int tile = blockIdx.z / a.Nn, n = blockIdx.z % a.Nn;
    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const float* in = static_cast<const float*>(a.in) + tile * a.in_tile + int64_t(n) * a.Cin * plane;
    const __amdgpu_buffer_rsrc_t rin =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(in), 0, int(a.Cin * plane * 4), kWord3);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.w), 0, a.wK * a.wC * a.R * a.S * 4, kWord3);
    const int w_os = int(a.w_os), w_cs = int(a.w_cs), iplane = int(plane);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int row0 = u + a.base_r, col0 = v + a.base_c;   // window origin (stride 1)

    floatx16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;

    // weight rows: forward, output channel ol with CC * Tt elements (ci, tap);
    // input gradient, input channel ci with kOB * Tt elements (o, tap)
    const int rowlen = (a.wmode ? kOB : CC) * Tt, nw = (a.wmode ? CC : kOB) * rowlen;
    const float rinv = 1.0f / float(rowlen);
    const int np = CC * PA * TA;
    for (int c0 = 0; c0 < a.Cin; c0 += CC) {
        __syncthreads();
        // one batch of weight and one of window elements per pass, all loads
        // of the pass issued before its first store
        const int nbw = (nw + kThreadsF * kWF - 1) / (kThreadsF * kWF);
        const int nbp = (np + kThreadsF * kPF - 1) / (kThreadsF * kPF);
        for (int b = 0; b < nbw || b < nbp; ++b) {
            float wv[kWF], pv[kPF];
            int ws_[kWF], ps_[kPF];
            if (b < nbw) {
                const int e0 = tid + b * kThreadsF * kWF;
#pragma unroll
                for (int q = 0; q < kWF; ++q) {
                    const int e = e0 + q * kThreadsF;
                    const int ec = min(e, nw - 1);
                    int rem;
                    const int row = frame_divmod(ec, rowlen, rinv, rem);
                    const int x = rem / Tt, rt = rem - x * Tt;   // channel within the row, raw tap
                    const int ol = a.wmode ? x : row, ci = a.wmode ? row : x;
                    const int wr = rt / Ts, wsc = rt - wr * Ts;   // stride 1: the filter is Tr x Ts
                    // kernel tap (tr, ts) of filter tap (wr, wsc): wr = wr0 + wrstep tr, wrstep = +-1
                    const int t = (wr - a.wr0) * a.wrstep * Ts + (wsc - a.ws0) * a.wsstep;
                    const int o = o0 + ol, cg = c0 + ci;
                    const int off = (o < a.Cout && cg < a.Cin) ? 4 * (o * w_os + cg * w_cs + rt) : kOOB;
                    wv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rw, off, 0, 0));
                    ws_[q] = e < nw ? (t * CC + ci) * kWS + ol : -1;
                }
            }
            if (b < nbp) {
                // window: item (channel, along, across), the input column fastest
                const int e0 = tid + b * kThreadsF * kPF;
#pragma unroll
                for (int q = 0; q < kPF; ++q) {
                    const int e = e0 + q * kThreadsF;
                    const int ec = min(e, np - 1);
                    int al, ac, ci;
                    if (!cm) { al = ec % PA; const int r = ec / PA; ac = r % TA; ci = r / TA; }
                    else { ac = ec % TA; const int r = ec / TA; al = r % PA; ci = r / PA; }
                    const int gr = row0 + (cm ? al : ac), gc = col0 + (cm ? ac : al);
                    const bool ok = gr >= 0 && gr < a.in_rows && gc >= 0 && gc < a.in_cols && c0 + ci < a.Cin;
                    const int off = ok ? 4 * ((c0 + ci) * iplane + gr * a.in_pitch + gc) : kOOB;
                    pv[q] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rin, off, 0, 0));
                    ps_[q] = e < np ? (ci * PA + al) * TA + ac : -1;
                }
            }
            if (b < nbw) {
#pragma unroll
                for (int q = 0; q < kWF; ++q)
                    if (ws_[q] >= 0) wl[ws_[q]] = wv[q];
            }
            if (b < nbp) {
#pragma unroll
                for (int q = 0; q < kPF; ++q)
                    if (ps_[q] >= 0) pl[ps_[q]] = pv[q];
            }
        }
        __syncthreads();

        // k-steps (tap t, channel pair c2), t-major; wave w takes the
        // contiguous eighth [w nk / 8, (w + 1) nk / 8)
        const int nk = Tt * CCH;
        const int kb = wave * nk / kWavesF, ke = (wave + 1) * nk / kWavesF;
        int t = kb / CCH, c2 = kb - t * CCH;
        auto kstep = [&]() __attribute__((always_inline)) {
            const int ci = 2 * c2 + hi;
            const int tr = t / Ts, ts = t - tr * Ts;
            const float A = wl[(t * CC + ci) * kWS + l32];
            const int al = l32 + (cm ? tr : ts), ac = cm ? ts : tr;
            const float B = pl[(ci * PA + al) * TA + ac];
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(A, B, acc, 0, 0, 0);
            const bool wrap = ++c2 == CCH;
            c2 = wrap ? 0 : c2;
            t += wrap ? 1 : 0;
        };
        // four steps per pass: their operand reads can be issued ahead of
        // the MFMAs
        int kk = kb;
        for (; kk + 4 <= ke; kk += 4) { kstep(); kstep(); kstep(); kstep(); }
        for (; kk < ke; ++kk) kstep();
    }
    frame_sum_store<kWavesF>(a, acc, smem, tile, n, o0, cm, u, v, n_out);
}

bool igemm_frame_plan(IgemmArgs& a, int dtype) {
    if (!a.frame || a.istr != 1 || a.Tr * a.Ts == 0 || a.bp) return false;
    // the tap flip is read back as (wr - wr0) * wrstep: unit tap steps only
    if ((a.wrstep != 1 && a.wrstep != -1) || (a.wsstep != 1 && a.wsstep != -1)) return false;
    // byte offsets of the buffer loads are 32-bit
    const int es = dtype == 1 ? 2 : 4;
    if (int64_t(a.Cin) * a.in_rows * a.in_pitch * es >= kOOB || int64_t(a.wK) * a.wC * a.R * a.S * es >= kOOB)
        return false;
    // channel chunks, widest first: bf16 multiples of 8 up to 64, fp32 even up to 32
    const int gran = dtype == 1 ? 8 : 2, maxcc = dtype == 1 ? 64 : 32;
    const int cin_r = (a.Cin + gran - 1) / gran * gran;
    int cands[8], nc = 0;
    cands[nc++] = std::min(cin_r, maxcc);
    for (int c = maxcc; c >= gran; c /= 2)
        if (c < cands[0]) cands[nc++] = c;
    const int limit = device_lds_limit();
    for (int budget : {std::min(80 * 1024, limit), limit}) {
        for (int i = 0; i < nc; ++i) {
            const int b = dtype == 1 ? frame_lds(a, cands[i]) : frame_lds_f32(a, cands[i]);
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

template <int TR, int TS>
static hipError_t launch_frame_f32(const IgemmArgs& a, dim3 grid, hipStream_t s) {
    const void* f = reinterpret_cast<const void*>(igemm_frame_f32_kernel<TR, TS>);
    if (a.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((igemm_frame_f32_kernel<TR, TS>), grid, dim3(kThreadsF), a.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_igemm_frame(const IgemmArgs& a, int dtype, hipStream_t s) {
    dim3 grid(a.fblk[a.fseg], (a.Cout + kOB - 1) / kOB, a.ntiles * a.Nn);
    if (grid.x == 0) return hipSuccess;   // an empty frame
    if (dtype != 1) {
        if (a.Tr == 3 && a.Ts == 3) return launch_frame_f32<3, 3>(a, grid, s);
        return launch_frame_f32<0, 0>(a, grid, s);
    }
    if (a.Tr == 3 && a.Ts == 3) return launch_frame_taps<3>(a, grid, s);
    if (a.Tr == 5 && a.Ts == 5) return launch_frame_taps<5>(a, grid, s);
    if (a.Tr == 7 && a.Ts == 7) return launch_frame_taps<7>(a, grid, s);
    return launch_frame_t<0, 0, 0>(a, grid, s);
}

}  // namespace dc
