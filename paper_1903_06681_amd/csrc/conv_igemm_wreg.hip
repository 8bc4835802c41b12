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

// One fp32 output value stored straight from the register that holds it
// (an accumulator AGPR), at device scope (sc1: written through to memory).
// Measured against the non-temporal hint: ResNet 1x1 input gradient
// (103 MB written) 48 -> 31 us, 3x3 56^2 layer 18.8 -> 18.2 us; the 5x5
// 32-channel tile and the 1x1 forward about 1 us slower.  (Choosing the
// scope per launch with a branch at every store cost more than either.)
__device__ __forceinline__ void wreg_store(float* p, float v) {
    asm volatile("global_store_dword %0, %1, off sc1" : : "v"(p), "a"(v) : "memory");
}

// The same through a buffer resource over the workgroup's output block, for
// the stores of interior blocks: the channel's offset oc * cstride (bytes)
// is formed by the scalar unit inside the statement (OC is a compile-time
// channel), added to the row's offset; the lane's part is voff.  Written as
// a 64-bit address expression, the per-channel offsets stayed live, ran the
// kernel out of scalar registers and were read back from lanes of a vector
// register (v_readlane) in front of every store.
template <int OC>
__device__ __forceinline__ void wreg_store_oc(__amdgpu_buffer_rsrc_t rs, int voff, int rowoff, int cstride, float v) {
    int so;
    asm volatile("s_mul_i32 %0, %1, %2\n\ts_add_i32 %0, %0, %3\n\tbuffer_store_dword %4, %5, %6, %0 offen sc1"
                 : "=&s"(so) : "s"(cstride), "n"(OC), "s"(rowoff), "a"(v), "v"(voff), "s"(rs));
}

static constexpr int kWThreads = 256;
static constexpr int kWWord3 = 0x00020000;   // buffer resource word 3 (gfx9 family: raw dword access)

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
            d[(2 * m) * 4 + j] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);      // low halves
            d[(2 * m + 1) * 4 + j] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);  // high halves
        }
}

// PH (forward at stride 2 with at most 4 channels): the strided correlation
// of Eq. (1) as a stride-1 one over the four phase images x[ci][2i + pr][2j +
// pc], phase channel c' = 4 ci + 2 pr + pc (padded to 16 with zero weights),
// phase taps (r', s') = filter tap (2r' + pr, 2s' + pc); TR x TS is then the
// phase filter.  Ring row m holds phase row u0 + m: each staging block loads
// the two 16-byte chunks of four (ci, pr) rows and keeps the columns of one
// parity per phase channel.
//
// BP (MODE 2; backward-data at stride 2 with at most 8 channels): the four
// output phases of Eq. (3) as one stride-1 correlation over dy.  Row o' =
// 4 c + 2 py + px of the weight image is output channel c at phase (py, px);
// window tap (a, b) holds filter tap (r0[py] - 2 (a - dr[py]), s0[px] - 2 (b -
// dc[px])), zero outside phase (py, px)'s own taps.  Output pixel (u, v) of
// the phase grid goes to dx[c][2u + py][2v + px].  The strips start bpvoff
// pixels early so that the staged dy columns are 16-byte aligned; pixels
// v < 0 are not stored.
// MF: the tile's pixel count is not a multiple of 64, so some strips are
// partial; their stores stay inside the MFMA stream, masked per lane (a
// separate instantiation, so that layers with whole strips keep exactly the
// code they had: that kernel is sensitive to small changes in its schedule).
template <int NOB, int TR, int TS, int CG, int MINWG, int MODE = 0, bool MF = false>
__global__ __launch_bounds__(kWThreads, MINWG) void igemm_wreg_kernel(IgemmArgs a) {
    constexpr bool PH = MODE == 1, BP = MODE == 2;
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
    // weight fragments held in AGPRs (fragment f = k * NOB + ob, f < NAG); the
    // two accumulator sets take 32 * NOB of the 256 AGPRs, the rest of Wf sits
    // in VGPRs
    constexpr int NAG = (NOB * KS < (256 - 32 * NOB) / 4) ? NOB * KS : (256 - 32 * NOB) / 4;
    constexpr int kPre = 3;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int vb = c % a.nvb; c /= a.nvb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int u0 = seg * a.rows_per_seg;
    const int u_end = min(u0 + a.rows_per_seg, a.Uo);
    const int v0 = vb * 64 - (BP ? a.bpvoff : 0);
    const int o0 = blockIdx.y * OBT;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;

    // ---- input ring addressing; the first ring rows are loaded before the
    // weights so that both latencies overlap
    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const uint16_t* in = static_cast<const uint16_t*>(a.in) + tile * a.in_tile +
                         int64_t(n) * a.Cin * plane;
    const int xr0 = PH ? u0 : u0 + a.base_r;       // input row (PH: phase row) of ring row 0
    const int xc0 = (PH ? 2 * v0 : v0) + a.base_c; // input column of staged pixel 0 (a multiple of 8)
    uint4 stg[BPT][8], stg1[BPT][8];

    auto load_rows = [&](uint4 (&sg)[BPT][8], int m0, int nrow) {   // ring rows m0 .. m0+nrow-1 -> registers
#pragma unroll
        for (int b = 0; b < BPT; ++b) {
            const int blk = tid + b * kWThreads;
            if (blk < nrow * BLK_ROW) {
                const int m = m0 + blk / BLK_ROW, rb = blk % BLK_ROW;
                const int cg8 = rb % NCG8, pg = rb / NCG8;
                // Unconditional 16-byte loads from clamped addresses: a row or
                // column outside the tile only ever feeds output pixels that
                // are not stored, so its values need no masking.
                if constexpr (PH) {
                    // phase channels 8 cg8 .. + 7 = four (ci, pr) rows x two parities
                    const int gc = min(xc0 + pg * 16, a.in_pitch - 8);
                    const int gc2 = min(xc0 + pg * 16 + 8, a.in_pitch - 8);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int cpq = cg8 * 8 + 2 * q, ci = min(cpq >> 2, a.Cin - 1), pr = (cpq >> 1) & 1;
                        const int gr = min(max(2 * (xr0 + m) + pr + a.base_r, 0), a.in_rows - 1);
                        const uint16_t* src = in + int64_t(ci) * plane + int64_t(gr) * a.in_pitch;
                        sg[b][2 * q] = *reinterpret_cast<const uint4*>(src + gc);
                        sg[b][2 * q + 1] = *reinterpret_cast<const uint4*>(src + gc2);
                    }
                } else {
                    const int gr = min(max(xr0 + m, 0), a.in_rows - 1);
                    const int gc = min(xc0 + pg * 8, a.in_pitch - 8);
                    const uint16_t* src = in + int64_t(gr) * a.in_pitch + gc + (cg8 * 8) * plane;
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        sg[b][j] = *reinterpret_cast<const uint4*>(src + j * plane);
                }
            }
        }
    };
    auto store_rows = [&](const uint4 (&sg)[BPT][8], int m0, int nrow) {
#pragma unroll
        for (int b = 0; b < BPT; ++b) {
            const int blk = tid + b * kWThreads;
            if (blk < nrow * BLK_ROW) {
                const int m = m0 + blk / BLK_ROW, rb = blk % BLK_ROW;
                const int cg8 = rb % NCG8, pg = rb / NCG8;
                uint4 t[8];
                if constexpr (PH) {
                    // channel 2q + pc: columns of parity pc of the q-th row's 16
                    uint4 ch[8];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t w8[8] = {sg[b][2 * q].x, sg[b][2 * q].y, sg[b][2 * q].z, sg[b][2 * q].w,
                                                sg[b][2 * q + 1].x, sg[b][2 * q + 1].y,
                                                sg[b][2 * q + 1].z, sg[b][2 * q + 1].w};
                        uint32_t e[4], o[4];
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            e[k] = (w8[2 * k] & 0xffffu) | (w8[2 * k + 1] << 16);
                            o[k] = (w8[2 * k] >> 16) | (w8[2 * k + 1] & 0xffff0000u);
                        }
                        ch[2 * q] = make_uint4(e[0], e[1], e[2], e[3]);
                        ch[2 * q + 1] = make_uint4(o[0], o[1], o[2], o[3]);
                    }
                    transpose8x8(ch, t);
                } else {
                    transpose8x8(sg[b], t);
                }
                uint16_t* dst = lds + (m % NRING) * ROWSZ + (pg * 8) * PS + cg8 * 8;
#pragma unroll
                for (int p = 0; p < 8; ++p) *reinterpret_cast<uint4*>(dst + p * PS) = t[p];
            }
        }
    };

    constexpr int NPRE = 1;   // row pairs loaded before the weights
    load_rows(stg, 0, min(2, TR + 1));
    if (NPRE > 1) load_rows(stg1, 2, min(2, TR - 1));

    // ---- weights -> A-fragments, in two passes:
    //  1. the workgroup's block of w goes to LDS, rows o of pitch PW:
    //       forward:       Wl[o][ci][t] = w[o0+o][ci][t]   (w's own order: a
    //                      straight 16-byte copy)
    //       backward-data: Wl[o][t][ci] = w[ci][o0+o][t]   (tap-major: the
    //                      transpose of w's first two axes is written by
    //                      lanes = consecutive ci, i.e. contiguous LDS bytes)
    //     rows o >= Cout - o0 hold whatever was read: they only feed output
    //     channels that are never stored;
    //  2. each lane builds, per (output block, 16-channel group), its T
    //     fragments of 8 channels: forward from its 8 channels x T taps
    //     (16*T contiguous bytes) regrouped with byte permutes; backward-data
    //     one aligned 16-byte read per fragment, the taps taken in reverse
    //     order (the flip of Eq. (3)).
    constexpr int T = TR * TS;
    constexpr int RL = CIN * T;                                    // row length
    constexpr int PW = ((RL * 2 + 239) / 256 * 256 + 16) / 2;      // 2*PW = 16 (mod 256)
    constexpr int PWB = ((RL * 2 + 111) / 128 * 128 + 16) / 2;     // 2*PWB = 16 (mod 128)
    const int nO = min(OBT, a.Cout - o0);                         // valid output channels here
    uint16_t* Wl = lds;
    {
        const uint16_t* w = static_cast<const uint16_t*>(a.w);
        if constexpr (BP) {
            // merged-phase image: Wl[o'][k][a * TS + b] (o' = 4 c + 2 py + px, k = dy channel)
            for (int e = tid; e < OBT * RL; e += kWThreads) {
                const int o = e / RL, r_ = e % RL, ci = r_ / T, t = r_ % T;
                const int c = o >> 2, py = (o >> 1) & 1, px = o & 1;
                const int tr = t / TS - a.bpdr[py], ts = t % TS - a.bpdc[px];
                const bool ok = c < a.bpC && tr >= 0 && tr < a.bptr[py] && ts >= 0 && ts < a.bpts[px];
                const int r = a.bpr0[py] - 2 * tr, sx = a.bps0[px] - 2 * ts;
                Wl[o * PW + r_] = ok ? w[((int64_t(ci) * a.wC + c) * a.R + r) * a.S + sx] : uint16_t(0);
            }
        } else if constexpr (PH) {
            // phase weights: Wl[o][c'][t'] = w[o0+o][ci][2r'+pr][2s'+pc], zero past
            // the filter and for the padding channels
            for (int e = tid; e < OBT * RL; e += kWThreads) {
                const int o = e / RL, r_ = e % RL, cp = r_ / T, t = r_ % T;
                const int ci = cp >> 2, r = 2 * (t / TS) + ((cp >> 1) & 1), sx = 2 * (t % TS) + (cp & 1);
                const int oc = min(o0 + o, a.Cout - 1);
                const bool ok = ci < a.wC && r < a.R && sx < a.S;
                Wl[o * PW + r_] = ok ? w[(int64_t(oc) * a.wC + ci) * a.R * a.S + r * a.S + sx] : uint16_t(0);
            }
        } else if (a.wvec && a.wmode == 0) {
            // rows o0 .. o0+OBT-1 of w are consecutive: 16-byte chunks straight to
            // LDS, all of a thread's loads in flight at once (chunks of rows
            // past Cout re-read the last valid chunk).  Every workgroup reads
            // the same block at the same moment; each starts at its own
            // offset so that the requests spread over the L2 channels
            // instead of queueing on the few that hold the first lines.
            constexpr int CPR = RL / 8, NCH = OBT * CPR, NB = (NCH + kWThreads - 1) / kWThreads;
            const int last = nO * CPR - 1;
            const int rot = ((blockIdx.x % 16) * (NB / 16 > 0 ? NB / 16 : 1) % NB) * kWThreads;   // < NB * kWThreads
            const uint4* src = reinterpret_cast<const uint4*>(w + int64_t(o0) * RL);
            uint4 buf[NB];
            int vv[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                int v = b * kWThreads + tid + rot;
                v = v >= NB * kWThreads ? v - NB * kWThreads : v;
                vv[b] = v;
                buf[b] = src[min(v, last)];
            }
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int v = vv[b];
                if (v < NCH) *reinterpret_cast<uint4*>(Wl + (v / CPR) * PW + (v % CPR) * 8) = buf[b];
            }
        } else if (a.wvec) {
            // row ci of w holds (o, t) of this block as OBT*T consecutive
            // elements (16-byte chunks c).  A thread takes 8x8 blocks (8 rows
            // ci x one chunk), loads the 8 chunks (consecutive threads:
            // consecutive chunks of the same rows), transposes them in
            // registers and writes 8 aligned 16-byte vectors Wl[o][t][ci..ci+7].
            // The workgroups start at different blocks (see the forward copy).
            constexpr int CPR = OBT * T / 8, NBLK = (CIN / 8) * CPR;
            constexpr int NB = (NBLK + kWThreads - 1) / kWThreads;
            const int64_t rs = int64_t(a.Cout) * T;                 // w row stride
            const int64_t last = int64_t(a.Cout) * T - 8;           // last chunk start in a row
            const int rot = (blockIdx.x % NB) * kWThreads;
            uint4 blk[NB][8];
            int bid[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                int v = b * kWThreads + tid + rot;
                v = v >= NB * kWThreads ? v - NB * kWThreads : v;
                bid[b] = v;
                const int vc = min(v, NBLK - 1), g = vc / CPR, c = vc - g * CPR;
                const uint16_t* src = w + min(int64_t(o0) * T + c * 8, last) + int64_t(g * 8) * rs;
#pragma unroll
                for (int r = 0; r < 8; ++r) blk[b][r] = *reinterpret_cast<const uint4*>(src + r * rs);
            }
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                if (bid[b] < NBLK) {
                    const int g = bid[b] / CPR, c = bid[b] - g * CPR;
                    uint4 t8[8];
                    transpose8x8(blk[b], t8);
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const int e = c * 8 + q, o = e / T, t = e - o * T;
                        *reinterpret_cast<uint4*>(Wl + o * PWB + t * CIN + g * 8) = t8[q];
                    }
                }
            }
        } else {
            // unaligned rows: element by element
            for (int e = tid; e < OBT * RL; e += kWThreads) {
                const int o = e / RL, r = e % RL, ci = r / T, t = r % T;
                const int oc = min(o0 + o, a.Cout - 1);
                if (a.wmode)
                    Wl[o * PWB + t * CIN + ci] = w[(int64_t(ci) * a.Cout + oc) * T + t];
                else
                    Wl[o * PW + r] = w[(int64_t(oc) * CIN + ci) * T + t];
            }
        }
    }
    __syncthreads();
    bf16x8 Wf[NOB][KS];
    if (a.wmode) {
        static_for<0, NOB * KS>([&](auto fc) {
            constexpr int f = decltype(fc)::value, ob = f % NOB, k = f / NOB, t = k / CG, cg = k % CG;
            Wf[ob][k] = *reinterpret_cast<const bf16x8*>(Wl + (ob * 32 + l32) * PWB + (T - 1 - t) * CIN +
                                                         cg * 16 + 8 * hi);
        });
    } else static_for<0, NOB * CG>([&](auto gc) {
        constexpr int g = decltype(gc)::value, ob = g / CG, cg = g % CG;
        const uint16_t* row = Wl + (ob * 32 + l32) * PW + (cg * 16 + 8 * hi) * T;
        uint32_t seg[4 * T];   // element c*T + t: channel c of the 8, tap t
#pragma unroll
        for (int m = 0; m < T; ++m) {
            const uint4 q = *reinterpret_cast<const uint4*>(row + 8 * m);
            seg[4 * m] = q.x; seg[4 * m + 1] = q.y; seg[4 * m + 2] = q.z; seg[4 * m + 3] = q.w;
        }
        static_for<0, T>([&](auto tc) {
            constexpr int t = decltype(tc)::value;
            Pack8 p;
            static_for<0, 4>([&](auto qc) {
                constexpr int q = decltype(qc)::value;
                constexpr int e0 = (2 * q) * T + t, e1 = (2 * q + 1) * T + t;
                // element e0 into the low half, e1 into the high half: one byte permute
                constexpr uint32_t sel = ((e0 & 1) ? 0x0302u : 0x0100u) | (((e1 & 1) ? 0x0706u : 0x0504u) << 16);
                p.d[q] = __builtin_amdgcn_perm(seg[e1 >> 1], seg[e0 >> 1], sel);
            });
            Wf[ob][t * CG + cg] = p.b;
        });
    });
    // settle each fragment in its register class before the loop
    static_for<0, NOB * KS>([&](auto fc) {
        constexpr int f = decltype(fc)::value;
        bf16x8& wf = Wf[f % NOB][f / NOB];
        if constexpr (f < NAG)
            asm volatile("" : "+a"(wf));
        else
            asm volatile("" : "+v"(wf));
    });
    __syncthreads();   // the image space becomes the input ring

    // ---- input ring
    // ring rows 0 .. TR (the inputs of the first two output rows)
    store_rows(stg, 0, min(2, TR + 1));
    if (NPRE > 1) store_rows(stg1, 2, min(2, TR - 1));
    for (int m = 2 * NPRE; m <= TR; m += 2) {
        const int nr = min(2, TR + 1 - m);
        load_rows(stg, m, nr);
        store_rows(stg, m, nr);
    }
    __syncthreads();

    const int wrow = wave >> 1;
    const int px = (wave & 1) * 32 + l32;
    const int v = v0 + px;
    const int nsteps = (u_end - u0 + 1) / 2;
    const int64_t oplane = int64_t(a.out_rows) * a.out_cols;
    // output of this lane's pixel at channel o0 + 4*hi; channel o0 + 4*hi + c is c*oplane further
    float* const out = a.out + tile * a.out_tile + (int64_t(n) * a.Cout + o0 + 4 * hi) * oplane +
                       int64_t(v) * a.ostr + a.oph_c;
    // the same as a buffer: base at channel o0, this lane's byte offset, and
    // the byte strides of a channel and a row (the plan keeps the block below
    // 2^31 bytes)
    float* const outb = a.out + tile * a.out_tile + (int64_t(n) * a.Cout + o0) * oplane;
    const __amdgpu_buffer_rsrc_t rout =
        __builtin_amdgcn_make_buffer_rsrc(outb, 0, int((int64_t(a.Cout) - o0) * oplane * 4), kWWord3);
    const int voff_out = int(((4 * hi) * oplane + int64_t(v) * a.ostr + a.oph_c) * 4);
    const int opl4 = int(oplane * 4);
    // every lane's pixel and every channel of the block in range: stores need no masks
    const bool block_full = !BP && (MF || v0 + 64 <= a.Vo) && (o0 + OBT <= a.Cout);
    auto out_row = [&](int u) { return out + int64_t(u * a.ostr + a.oph_r) * a.out_cols; };
    // D layout: value e of lane l is output channel 8*(e/4) + 4*(l/32) + e%4, pixel l%32
    auto store_masked = [&](const floatx16 (&acc)[NOB], int u) {
        if constexpr (BP) {
            // row o' = 8 (e/4) + 4 hi + e%4 = 4 c + 2 py + px: c = 2 (e/4) + hi
            if (u < u_end && v >= 0 && v < a.Vo) {
                const int64_t plane = int64_t(a.out_rows) * a.out_cols;
                float* const o = a.out + tile * a.out_tile + (int64_t(n) * a.bpC + hi) * plane +
                                 int64_t(2 * u) * a.out_cols + 2 * v;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int c = 2 * (e / 4) + hi, py = (e % 4) / 2, px = e % 2;
                    if (c < a.bpC) o[int64_t(2 * (e / 4)) * plane + py * a.out_cols + px] = acc[0][e];
                }
            }
            return;
        }
        if (u < u_end && v < a.Vo) {
            float* orow = out_row(u);
#pragma unroll
            for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int oc = ob * 32 + 8 * (e / 4) + (e % 4);
                    if (o0 + 4 * hi + oc < a.Cout) wreg_store(orow + int64_t(oc) * oplane, acc[ob][e]);
                }
        }
    };

    // One step: two output rows.  Within the MFMA stream of step i go
    //  - the stores of step i-1's accumulator (`prev`), two per MFMA from the
    //    start, so they drain while the matrix cores run (outputs are written
    //    once, at device scope: written through);
    //  - near the end, the transpose and LDS writes of the two input rows that
    //    step i+1 adds to the ring (loaded at the top of step i) -- their ring
    //    slots are not read in step i.
    // Loads and ring writes are unconditional (rows past the segment are
    // clamped reads, staged into slots no later step reads), so the waits
    // for them are exact.  The accumulators alternate between two register
    // sets from step to step.
    constexpr int NST = 16 * NOB;                       // stores per step
    constexpr int STAGE_AT = NOB * KS > 8 ? NOB * KS - 8 : 0;
    auto step = [&](int i, floatx16 (&acc)[NOB], const floatx16 (&prev)[NOB]) {
        load_rows(stg, 2 * i + TR + 1, 2);
        const int slot0 = (2 * i + wrow) % NRING;
        auto readB = [&](int k) {
            const int t = k / CG, cgi = k % CG;
            const int tr = t / TS, ts = t % TS;
            int slot = slot0 + tr;
            if (slot >= NRING) slot -= NRING;
            return *reinterpret_cast<const bf16x8*>(lds + slot * ROWSZ + (px + ts) * PS + cgi * 16 + 8 * hi);
        };
        const int u_prev = u0 + 2 * (i - 1) + wrow;
        const bool fast = i > 0 && block_full && u_prev < u_end;
        // (uniform in the wave: u_prev's row term depends on the wave only)
        const int prow4 = __builtin_amdgcn_readfirstlane(int(int64_t(u_prev * a.ostr + a.oph_r) * a.out_cols * 4));
        auto store_prev = [&](auto sc) {
            constexpr int s = decltype(sc)::value, sob = s / 16, e = s % 16;
            constexpr int oc = sob * 32 + 8 * (e / 4) + (e % 4);
            // (operands through locals: this compiler does not capture
            // variables that a lambda names only in asm operands)
            const __amdgpu_buffer_rsrc_t rs = rout;
            const int vo = voff_out, ro = prow4, cs = opl4;
            if constexpr (MF) {
                if (v < a.Vo) wreg_store_oc<oc>(rs, vo, ro, cs, prev[sob][e]);
            } else {
                wreg_store_oc<oc>(rs, vo, ro, cs, prev[sob][e]);
            }
        };
        auto mfmas = [&](auto with_stores) {
            // B operands run kPre k-steps ahead of the MFMAs that consume them
            bf16x8 Bq[kPre + 1];
#pragma unroll
            for (int k = 0; k < kPre && k < KS; ++k) Bq[k] = readB(k);
            static_for<0, NOB * KS>([&](auto fc) {
                constexpr int f = decltype(fc)::value, k = f / NOB, ob = f % NOB;
                if constexpr (ob == 0 && k + kPre < KS) Bq[(k + kPre) % (kPre + 1)] = readB(k + kPre);
                mfma32x32x16<(f < NAG), (k == 0)>(acc[ob], Wf[ob][k], Bq[k % (kPre + 1)]);
                if constexpr (decltype(with_stores)::value && 2 * f < NST) {
                    store_prev(std::integral_constant<int, 2 * f>{});
                    store_prev(std::integral_constant<int, 2 * f + 1>{});
                }
                if constexpr (f == STAGE_AT) store_rows(stg, 2 * i + TR + 1, 2);
            });
            if constexpr (decltype(with_stores)::value && 2 * NOB * KS < NST)   // fewer MFMAs than stores
                static_for<2 * NOB * KS, NST>([&](auto sc) { store_prev(sc); });
        };
        if (fast)
            mfmas(std::true_type{});
        else
            mfmas(std::false_type{});
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) mfma_drain(acc[ob]);
        if (i > 0 && !fast) store_masked(prev, u_prev);
        __syncthreads();
    };

    floatx16 accA[NOB], accB[NOB];
    int i = 0;
    for (; i + 1 < nsteps; i += 2) {
        step(i, accA, accB);
        step(i + 1, accB, accA);
    }
    if (i < nsteps) {
        step(i, accA, accB);
        store_masked(accA, u0 + 2 * i + wrow);
    } else if (nsteps > 0) {
        store_masked(accB, u0 + 2 * (i - 1) + wrow);
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

static int wreg_lds(int NOB, int TR, int TS, int CG) {
    const int CIN = CG * 16, PS = 8 * ((CIN / 8) | 1), RPX8 = (64 + TS - 1 + 7) / 8;
    const int ring = (TR + 3) * RPX8 * 8 * PS * 2;
    const int RL = CIN * TR * TS;
    const int PW = ((RL * 2 + 239) / 256 * 256 + 16) / 2;       // forward weight rows
    const int PWB = ((RL * 2 + 111) / 128 * 128 + 16) / 2;      // backward-data weight rows
    const int wl = NOB * 32 * (PW > PWB ? PW : PWB) * 2;
    return ring > wl ? ring : wl;
}

// the phase-image forward (stride 2, at most 4 channels): instantiated
// (NOB, phase filter) shapes
static bool wreg_phase_shape(int NOB, int TR, int TS) {
    return (NOB == 2 || NOB == 1) && ((TR == 4 && TS == 4) || (TR == 2 && TS == 2) || (TR == 3 && TS == 3));
}

static void wreg_segments(IgemmArgs& a) {
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
}

// merged-phase backward-data: instantiated (window, 16-channel groups) shapes
static bool wreg_bp_shape(int TR, int TS, int CG) {
    return (TR == 4 && TS == 4 && CG == 4) || (TR == 2 && TS == 2 && CG == 4);
}

bool igemm_wreg_plan(IgemmArgs& a) {
    if (a.bp) {
        // the caller's merged-phase request (see the kernel's BP mode)
        a.phase = 0;
        if (a.Cout > 32 || a.Cin % 16 != 0 || !wreg_bp_shape(a.Tr, a.Ts, a.Cin / 16)) return false;
        if (a.in_pitch % 8 != 0) return false;
        a.bpvoff = a.base_c % 8;                   // strips start this many pixels early
        const int lds = wreg_lds(1, a.Tr, a.Ts, a.Cin / 16);
        if (lds > device_lds_limit()) return false;
        a.OB = 32;
        a.wvec = 0;
        const int vo = a.Vo;
        a.Vo = vo + a.bpvoff;                      // the strips cover the early pixels too
        wreg_segments(a);
        a.Vo = vo;
        a.lds_bytes = lds;
        a.kind = 1;
        return true;
    }
    a.phase = 0;
    if (a.wmode == 0 && a.istr == 2 && a.ostr == 1 && 4 * a.Cin <= 16 && a.base_c % 8 == 0 &&
        a.in_pitch % 8 == 0 && a.Tr == a.R && a.Ts == a.S) {
        const int NOB = a.Cout <= 32 ? 1 : 2, TRp = (a.R + 1) / 2, TSp = (a.S + 1) / 2;
        if (wreg_phase_shape(NOB, TRp, TSp)) {
            const int lds = wreg_lds(NOB, TRp, TSp, 1);
            if (lds <= device_lds_limit()) {
                a.phase = 1;
                a.Tr = TRp; a.Ts = TSp;
                a.OB = NOB * 32;
                a.wvec = 0;
                wreg_segments(a);
                a.lds_bytes = lds;
                a.kind = 1;
                return true;
            }
        }
    }
    if (a.istr != 1 || a.Cin % 16 != 0 || a.Tr < 1 || a.Ts < 1) return false;
    if (a.base_c % 8 != 0 || a.in_pitch % 8 != 0) return false;   // 16-byte aligned row loads
    const int NOB = a.Cout <= 32 ? 1 : 2;
    const int CG = a.Cin / 16;
    if (!wreg_shape(NOB, a.Tr, a.Ts, CG)) return false;
    // taps in k-step order: the identity (forward) or the full flip (backward-data, stride 1)
    if (a.Tr != a.R || a.Ts != a.S) return false;
    if (a.wmode == 0 && !(a.wr0 == 0 && a.wrstep == 1 && a.ws0 == 0 && a.wsstep == 1)) return false;
    if (a.wmode == 1 && !(a.wr0 == a.R - 1 && a.wrstep == -1 && a.ws0 == a.S - 1 && a.wsstep == -1))
        return false;
    const int T = a.R * a.S;
    a.wvec = a.wmode ? int((int64_t(a.Cout) * T) % 8 == 0 && (int64_t(a.Cout) * T) >= 8)
                     : int((int64_t(a.Cin) * T) % 8 == 0);
    const int lds = wreg_lds(NOB, a.Tr, a.Ts, CG);
    if (lds > device_lds_limit()) return false;
    // interior stores address a sample's output channels with 32-bit byte offsets
    if (int64_t(a.Cout) * a.out_rows * a.out_cols * 4 >= (int64_t(1) << 31)) return false;
    a.OB = NOB * 32;
    wreg_segments(a);
    a.lds_bytes = lds;
    a.kind = 1;
    return true;
}

template <int NOB, int TR, int TS, int CG, int MINWG, int MODE = 0>
static hipError_t launch_one(const IgemmArgs& a, hipStream_t s) {
    if constexpr (MODE != 2) {   // partial strips: the masked-store instantiation
        if (a.Vo % 64 != 0) {
            auto k = igemm_wreg_kernel<NOB, TR, TS, CG, MINWG, MODE, true>;
            if (a.lds_bytes > 64 * 1024) {
                hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
                if (e != hipSuccess) return e;
            }
            dim3 grid(a.ntiles * a.Nn * a.nvb * a.nseg, (a.Cout + a.OB - 1) / a.OB);
            hipLaunchKernelGGL(k, grid, dim3(kWThreads), a.lds_bytes, s, a);
            return hipGetLastError();
        }
    }
    auto k = igemm_wreg_kernel<NOB, TR, TS, CG, MINWG, MODE>;
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
    if (a.bp) {
        if (a.Tr == 4 && a.Ts == 4 && CG == 4) return launch_one<1, 4, 4, 4, 1, 2>(a, s);
        if (a.Tr == 2 && a.Ts == 2 && CG == 4) return launch_one<1, 2, 2, 4, 1, 2>(a, s);
        return hipErrorInvalidValue;
    }
    if (a.phase) {
#define DC_WREG_PH(nob, t) \
        if (NOB == nob && a.Tr == t && a.Ts == t) return launch_one<nob, t, t, 1, 1, 1>(a, s);
        DC_WREG_PH(2, 4) DC_WREG_PH(1, 4) DC_WREG_PH(2, 2) DC_WREG_PH(1, 2) DC_WREG_PH(2, 3) DC_WREG_PH(1, 3)
#undef DC_WREG_PH
        return hipErrorInvalidValue;
    }
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
