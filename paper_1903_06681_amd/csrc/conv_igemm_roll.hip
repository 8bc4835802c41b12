// Forward / backward-data convolution, bf16, stride 1, weights in registers,
// rolling output rows (Eqs. (1) and (3) of Sec. II-A on a tile, Sec. III-A).
//
//   out[o][u][v] = sum_{r, s, ci} W[o][r, s, ci] * in[ci][u + r][v + s]
//
// Input row m of a segment feeds output rows m - r for every filter row r.
// A wave therefore keeps the accumulators of TR consecutive output rows live
// (one register set per row, set = row mod TR) and reads each input row from
// LDS once: one 16-byte operand read per (s, 16-channel group) feeds
// TR x NOB MFMAs, against NOB when every output row re-reads its TR input
// rows.  The cost is TR accumulator sets instead of two.
//
// A workgroup (4 waves) walks down a 128-column strip of one sample, one
// input row per step; wave w computes pixels 32 w .. 32 w + 31.  The input
// rows go through a two-slot LDS ring, channel-innermost ([pixel][channel],
// odd 16-byte pixel stride: conflict-free 16-byte operand reads).  Step j
// (input row j) runs, in one MFMA stream:
//  - phase A: the MFMAs of rows j - r for r >= 1, the operands of input row
//    j read once for all of them; the first of these MFMAs carry the
//    stores of row j - TR, which finished in step j - 1 and whose register
//    set row j takes over;
//  - phase B: the MFMAs of row j (r = 0), its operands read again (two
//    reads per (s, channel group) in all, against TR when every output row
//    reads its own input rows);
//  - the global loads of input row j + 1 (top of the step), their 8x8
//    register transposes and LDS writes into the other slot (at the end).
// Output stores are buffer stores (uniform row and channel offsets in
// scalar registers) at system scope: outputs are written once.
//
// The plan admits whole segments only (rows_per_seg divides Uo, 128-column
// strips tile Vo, 32- or 64-filter blocks tile Cout), so no store needs a mask.
// NM = rows_per_seg mod TR fixes, at compile time, which register set each
// step of the segment's tail uses.
#include <hip/hip_runtime.h>

#include "bf16util.h"
#include "kernels.h"

namespace dc {

static constexpr int kRThreads = 256;
static constexpr int kRStrip = 128;          // output columns per workgroup
static constexpr int kRWord3 = 0x00020000;   // buffer resource word 3 (gfx9 family: raw dword access)

// 8x8 transpose of 16-bit elements: in[c] holds 8 pixels of channel c,
// out[p] receives the 8 channels of pixel p.
__device__ __forceinline__ void roll_transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
    const uint32_t* s = reinterpret_cast<const uint32_t*>(in);
    uint32_t* d = reinterpret_cast<uint32_t*>(out);
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t lo = s[(2 * j) * 4 + m], hi = s[(2 * j + 1) * 4 + m];
            // one byte permute per word (v_perm_b32; the and/shift/or form
            // took two or three instructions): low halves, then high halves
            d[(2 * m) * 4 + j] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
            d[(2 * m + 1) * 4 + j] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);
        }
}

typedef unsigned roll_v4u __attribute__((ext_vector_type(4)));

// Wait states between the last MFMA writing a register set and its stores
// (32 >= passes + 4 for every 32x32 shape); ties every accumulator of the set.
template <int NOB>
__device__ __forceinline__ void roll_drain(floatx16 (&acc)[NOB]) {
    static_assert(NOB == 1 || NOB == 2, "one or two accumulators per set");
    if constexpr (NOB == 2)
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" : "+a"(acc[0]), "+a"(acc[1]));
    else
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" : "+a"(acc[0]));
}

// v_mfma_f32_32x32x16_bf16 with a weight fragment as the A operand (rows of
// D: output channels), read from AGPRs (WAG) or VGPRs, and the input pixels
// as the B operand (columns of D); ZERO starts a new accumulation.  A lane
// holds A[m = l%32][k = 8 (l/32) .. +7] = W[o = l%32][channels 8 (l/32) ..]
// and B[k = 8 (l/32) .. +7][n = l%32] = x[channels 8 (l/32) ..][pixel l%32].
// Pixels as the columns of D make each output store instruction write 128
// contiguous bytes of one channel plane per half-wave.
template <bool WAG, bool ZERO>
__device__ __forceinline__ void mfma_xw(floatx16& acc, const bf16x8& x, const bf16x8& w) {
    if constexpr (ZERO) {
        if constexpr (WAG)
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %2, %1, 0" : "=&a"(acc) : "v"(x), "a"(w));
        else
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %2, %1, 0" : "=&a"(acc) : "v"(x), "v"(w));
    } else {
        if constexpr (WAG)
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %2, %1, %0" : "+a"(acc) : "v"(x), "a"(w));
        else
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %2, %1, %0" : "+a"(acc) : "v"(x), "v"(w));
    }
}

template <int NOB, int TR, int TS, int CG, int NM>
__global__ __launch_bounds__(kRThreads, 1) void igemm_roll_kernel(IgemmArgs a) {
    static_assert(TR >= 2 && NM >= 0 && NM < TR, "rolling rows need TR >= 2");
    constexpr int NB = TS * CG;                 // operand reads per input row: (s, 16-channel group)
    constexpr int CIN = CG * 16;
    constexpr int PS = 8 * ((CIN / 8) | 1);     // ring pixel stride (elements)
    constexpr int RPX8 = (kRStrip + TS - 1 + 7) / 8;
    constexpr int ROWSZ = RPX8 * 8 * PS;
    constexpr int OBT = NOB * 32;
    constexpr int NCG8 = CIN / 8;
    constexpr int BLK_ROW = NCG8 * RPX8;        // 8x8 staging blocks per input row
    static_assert(BLK_ROW <= kRThreads, "one staging block per thread");
    constexpr int NSETS = TR;
    // weight fragments held in AGPRs (fragment f = k * NOB + ob, f < NAG);
    // the TR accumulator sets take 16 * NOB * TR of the 256 AGPRs
    constexpr int NWF = NOB * TR * TS * CG;
    constexpr int NAG = (NWF < (256 - 16 * NOB * NSETS) / 4) ? NWF : (256 - 16 * NOB * NSETS) / 4;
    constexpr int kPre = 2;                     // operand reads ahead of their MFMAs
    constexpr int NQ = kPre + 1;                // operand registers in flight
    constexpr int NST = 16 * NOB;               // 4-byte stores per output row and lane
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* lds = reinterpret_cast<uint16_t*>(smem);

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int vb = c % a.nvb; c /= a.nvb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int nrows = a.rows_per_seg;           // output rows of this segment (all segments full)
    const int u0 = seg * nrows;
    const int v0 = vb * kRStrip;
    const int o0 = blockIdx.y * OBT;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;

    // ---- input rows: buffer loads over this sample's channels
    const int64_t plane = int64_t(a.in_rows) * a.in_pitch;
    const uint16_t* in = static_cast<const uint16_t*>(a.in) + tile * a.in_tile + int64_t(n) * a.Cin * plane;
    const __amdgpu_buffer_rsrc_t rin =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(in), 0, int(a.Cin * plane * 2), kRWord3);
    const int xr0 = u0 + a.base_r;              // input row of ring row 0
    const int blk = tid;                        // this thread's staging block (if < BLK_ROW)
    const int cg8 = blk % NCG8, pg = blk / NCG8;
    const bool stager = blk < BLK_ROW;
    // unconditional 16-byte loads from clamped columns: columns past the
    // tile only feed pixels that are not stored
    const int gcol = min(a.base_c + v0 + pg * 8, a.in_pitch - 8);
    const int voff_in = int((int64_t(cg8 * 8) * plane + gcol) * 2);
    // The row loads and the output stores are written as instructions the
    // compiler does not see, so that its waits on the vector-memory counter
    // do not cover the stores: store_row waits for the loads itself, leaving
    // the NV stores issued since the loads in flight (the counter completes
    // in issue order).
    roll_v4u stg[8];
    auto load_row = [&](int m) __attribute__((always_inline)) {                // input row m of the segment -> registers
        if (stager) {
            const int gr = min(max(xr0 + m, 0), a.in_rows - 1);
            const int so = gr * a.in_pitch * 2;
            const int vo = voff_in;
            const __amdgpu_buffer_rsrc_t rs = rin;
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) {
                const int sj = so + int(jj * plane * 2);
                asm volatile("buffer_load_dwordx4 %0, %1, %2, %3 offen" : "=v"(stg[jj]) : "v"(vo), "s"(rs), "s"(sj));
            }
        }
    };
    auto store_row = [&](int m, auto nvc) __attribute__((always_inline)) {     // registers -> ring slot m & 1
        constexpr int NV = decltype(nvc)::value;
        static_assert(NV >= 0 && NV <= 63, "vector-memory counter range");
        if (stager) {
            asm volatile("s_waitcnt vmcnt(%8)"
                         : "+v"(stg[0]), "+v"(stg[1]), "+v"(stg[2]), "+v"(stg[3]), "+v"(stg[4]), "+v"(stg[5]),
                           "+v"(stg[6]), "+v"(stg[7])
                         : "n"(NV));
            uint4 in8[8];
#pragma unroll
            for (int p = 0; p < 8; ++p) in8[p] = make_uint4(stg[p].x, stg[p].y, stg[p].z, stg[p].w);
            uint4 t[8];
            roll_transpose8x8(in8, t);
            uint16_t* dst = lds + (m & 1) * ROWSZ + (pg * 8) * PS + cg8 * 8;
#pragma unroll
            for (int p = 0; p < 8; ++p) *reinterpret_cast<uint4*>(dst + p * PS) = t[p];
        }
    };

    load_row(0);   // in flight while the weights load

    // ---- weights -> A-fragments (the workgroup's block of w through LDS):
    //   forward:       Wl[o][ci][t] = w[o0+o][ci][t]   (16-byte chunk copies)
    //   backward-data: Wl[o][t][ci] = w[ci][o0+o][t]   (8x8 blocks transposed
    //                  in registers; the tap flip of Eq. (3) at read time)
    // Every workgroup reads the same block at the same moment; each starts at
    // its own offset so that the requests spread over the L2 channels.
    constexpr int T = TR * TS;
    constexpr int RL = CIN * T;
    constexpr int PW = ((RL * 2 + 239) / 256 * 256 + 16) / 2;      // 2*PW = 16 (mod 256)
    constexpr int PWB = ((RL * 2 + 111) / 128 * 128 + 16) / 2;     // 2*PWB = 16 (mod 128)
    uint16_t* Wl = lds;
    {
        const uint16_t* w = static_cast<const uint16_t*>(a.w);
        if (a.wmode == 0) {
            constexpr int CPR = RL / 8, NCH = OBT * CPR, NBW = (NCH + kRThreads - 1) / kRThreads;
            const int rot = ((blockIdx.x % 16) * (NBW / 16 > 0 ? NBW / 16 : 1) % NBW) * kRThreads;
            const uint4* src = reinterpret_cast<const uint4*>(w + int64_t(o0) * RL);
            uint4 buf[NBW];
            int vv[NBW];
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                int v = b * kRThreads + tid + rot;
                v = v >= NBW * kRThreads ? v - NBW * kRThreads : v;
                vv[b] = v;
                buf[b] = src[min(v, NCH - 1)];
            }
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const int v = vv[b];
                if (v < NCH) *reinterpret_cast<uint4*>(Wl + (v / CPR) * PW + (v % CPR) * 8) = buf[b];
            }
        } else {
            constexpr int CPR = OBT * T / 8, NBLK = (CIN / 8) * CPR;
            constexpr int NBW = (NBLK + kRThreads - 1) / kRThreads;
            const int64_t rs = int64_t(a.Cout) * T;                 // w row stride
            const int rot = (blockIdx.x % NBW) * kRThreads;
            uint4 bw[NBW][8];
            int bid[NBW];
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                int v = b * kRThreads + tid + rot;
                v = v >= NBW * kRThreads ? v - NBW * kRThreads : v;
                bid[b] = v;
                const int vc = min(v, NBLK - 1), g = vc / CPR, cc = vc - g * CPR;
                const uint16_t* src = w + int64_t(o0) * T + cc * 8 + int64_t(g * 8) * rs;
#pragma unroll
                for (int r = 0; r < 8; ++r) bw[b][r] = *reinterpret_cast<const uint4*>(src + r * rs);
            }
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                if (bid[b] < NBLK) {
                    const int g = bid[b] / CPR, cc = bid[b] - g * CPR;
                    uint4 t8[8];
                    roll_transpose8x8(bw[b], t8);
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const int e = cc * 8 + q, o = e / T, t = e - o * T;
                        *reinterpret_cast<uint4*>(Wl + o * PWB + t * CIN + g * 8) = t8[q];
                    }
                }
            }
        }
    }
    __syncthreads();
    // fragment k = t * CG + cg (t = r * TS + s) of output block ob: lane
    // (l32, hi) holds W[ob*32 + l32][tap t][cg*16 + 8 hi .. + 7]
    bf16x8 Wf[NOB][TR * TS * CG];
    if (a.wmode) {
        static_for<0, NWF>([&](auto fc) __attribute__((always_inline)) {
            constexpr int f = decltype(fc)::value, ob = f % NOB, k = f / NOB, t = k / CG, cg = k % CG;
            Wf[ob][k] = *reinterpret_cast<const bf16x8*>(Wl + (ob * 32 + l32) * PWB + (T - 1 - t) * CIN +
                                                         cg * 16 + 8 * hi);
        });
    } else static_for<0, NOB * CG>([&](auto gc) __attribute__((always_inline)) {
        constexpr int g = decltype(gc)::value, ob = g / CG, cg = g % CG;
        const uint16_t* row = Wl + (ob * 32 + l32) * PW + (cg * 16 + 8 * hi) * T;
        uint32_t sg[4 * T];   // element c*T + t: channel c of the 8, tap t
#pragma unroll
        for (int m = 0; m < T; ++m) {
            const uint4 q = *reinterpret_cast<const uint4*>(row + 8 * m);
            sg[4 * m] = q.x; sg[4 * m + 1] = q.y; sg[4 * m + 2] = q.z; sg[4 * m + 3] = q.w;
        }
        static_for<0, T>([&](auto tc) __attribute__((always_inline)) {
            constexpr int t = decltype(tc)::value;
            Pack8 p;
            static_for<0, 4>([&](auto qc) __attribute__((always_inline)) {
                constexpr int q = decltype(qc)::value;
                constexpr int e0 = (2 * q) * T + t, e1 = (2 * q + 1) * T + t;
                // element e0 into the low half, e1 into the high half: one byte permute
                constexpr uint32_t sel = ((e0 & 1) ? 0x0302u : 0x0100u) | (((e1 & 1) ? 0x0706u : 0x0504u) << 16);
                p.d[q] = __builtin_amdgcn_perm(sg[e1 >> 1], sg[e0 >> 1], sel);
            });
            Wf[ob][t * CG + cg] = p.b;
        });
    });
    static_for<0, NWF>([&](auto fc) __attribute__((always_inline)) {
        constexpr int f = decltype(fc)::value;
        bf16x8& wf = Wf[f % NOB][f / NOB];
        if constexpr (f < NAG)
            asm volatile("" : "+a"(wf));
        else
            asm volatile("" : "+v"(wf));
    });
    __syncthreads();   // the image space becomes the input ring

    store_row(0, std::integral_constant<int, 0>{});
    __syncthreads();

    // ---- outputs: buffer stores over the block's OBT channel planes of this sample
    const int64_t oplane = int64_t(a.out_rows) * a.out_cols;
    float* const outb = a.out + tile * a.out_tile + (int64_t(n) * a.Cout + o0) * oplane;
    const __amdgpu_buffer_rsrc_t rout =
        __builtin_amdgcn_make_buffer_rsrc(outb, 0, int(OBT * oplane * 4), kRWord3);
    const int px = wave * 32 + l32;
    // D layout: value e of lane l is output channel 8*(e/4) + 4*(l/32) + e%4
    // of the block ob, pixel l%32 of the wave's 32: sixteen 4-byte stores per
    // block; the lane's pixel and channel half are in its offset, the
    // channel's rest and the row are uniform
    const int voff_out = int((int64_t(4 * hi) * oplane + v0 + wave * 32 + l32) * 4);
    const int opl4 = int(oplane * 4);
    const int ocol4 = a.out_cols * 4;

    floatx16 acc[NSETS][NOB];
    auto store_set = [&](auto setc, auto sc, int q) __attribute__((always_inline)) {   // store s of output row q
        constexpr int SET = decltype(setc)::value, s = decltype(sc)::value, sob = s / 16, e = s % 16;
        constexpr int oc = sob * 32 + 8 * (e / 4) + e % 4;
        // Stored straight from the accumulator register: the builtin store
        // copies every value to a VGPR first, and with the VGPRs full those
        // copies share registers with the staged input rows.  The set's last
        // MFMA ended a step earlier (drained), and phase B overwrites the set
        // only 2 NOB MFMAs after the last store.  Nothing in the kernel reads
        // the output, so no memory clobber and no wait on the store.  System
        // scope (sc0 sc1): written through to memory; on c5a 1 us faster than
        // the non-temporal hint, 0.3 us faster than device scope (sc1).
        // The channel's offset is formed by the scalar unit inside the
        // statement (oc is a compile-time channel): as a plain expression the
        // compiler keeps all 32 channel offsets live, runs out of scalar
        // registers, parks them in lanes of a vector register and reads each
        // back (v_readlane, then a scalar add) in front of its store, a
        // dependent chain ahead of the next MFMA; about 0.8 us per pass on a
        // 64-channel 3x3 layer.
        // (operands through locals: this compiler does not capture variables
        // that a lambda names only in asm operands)
        const float f = acc[SET][sob][e];
        const int vo = voff_out, ro = (u0 + q) * ocol4, pl = opl4;
        const __amdgpu_buffer_rsrc_t rs = rout;
        int so;
        asm volatile("s_mul_i32 %0, %1, %3\n\ts_add_i32 %0, %0, %2\n\tbuffer_store_dword %4, %5, %6, %0 offen sc0 sc1"
                     : "=&s"(so) : "s"(pl), "s"(ro), "n"(oc), "a"(f), "v"(vo), "s"(rs));
    };

    // One step: input row j, register set J = j mod TR, filter rows
    // RLO..RHI active (rows j - r inside the segment), ST: store row j - TR.
    auto step = [&](auto Jc, auto RLOc, auto RHIc, auto STc, auto LDc, int j) __attribute__((always_inline)) {
        constexpr int J = decltype(Jc)::value, RLO = decltype(RLOc)::value, RHI = decltype(RHIc)::value;
        constexpr bool ST = decltype(STc)::value, LD = decltype(LDc)::value;
        constexpr int RIM = RLO > 1 ? RLO : 1;                    // lowest filter row of phase A
        constexpr int NIMM = RHI >= RIM ? RHI - RIM + 1 : 0;      // filter rows of phase A
        constexpr int NA = NIMM > 0 ? NB : 0;                     // phase A reads (rows j - r, r >= 1)
        constexpr int NR = NA + (RLO == 0 ? NB : 0);              // + phase B reads (row j, r = 0)
        // stores ride on the first AVAIL of phase A's MFMAs, spread evenly
        // (store i after MFMA i AVAIL / NST), the last at least 2 NOB MFMAs
        // before phase B reuses the set
        constexpr int SLOTS = NA * NIMM * NOB;
        constexpr int AVAIL = SLOTS - 2 * NOB;
        static_assert(!ST || AVAIL > 0, "stores need phase A MFMAs to ride on");
        constexpr int STAGE_X = NR > 2 ? NR - 2 : 0;
        if constexpr (LD) load_row(j + 1);
        const uint16_t* slot = lds + (j & 1) * ROWSZ + px * PS + 8 * hi;
        auto readB = [&](int x) __attribute__((always_inline)) {   // x: read index of the step
            const int b = x < NA ? x : x - NA, s = b / CG, cg = b % CG;
            return *reinterpret_cast<const bf16x8*>(slot + s * PS + cg * 16);
        };
        const int qst = j - TR;
        bf16x8 Bq[NQ];
#pragma unroll
        for (int x = 0; x < kPre && x < NR; ++x) Bq[x] = readB(x);
        static_for<0, NR>([&](auto xc) __attribute__((always_inline)) {
            constexpr int x = decltype(xc)::value;
            if constexpr (x + kPre < NR) Bq[(x + kPre) % NQ] = readB(x + kPre);
            if constexpr (x < NA) {
                constexpr int s = x / CG, cg = x % CG;
                static_for<0, NIMM>([&](auto ric) __attribute__((always_inline)) {
                    constexpr int r = RHI - decltype(ric)::value;          // RHI down to RIM
                    constexpr int SET = (J - r + NSETS) % NSETS;
                    static_for<0, NOB>([&](auto obc) __attribute__((always_inline)) {
                        constexpr int ob = decltype(obc)::value, k = (r * TS + s) * CG + cg, f = k * NOB + ob;
                        mfma_xw<(f < NAG), false>(acc[SET][ob], Bq[x % NQ], Wf[ob][k]);
                        if constexpr (ST) {
                            constexpr int m = (x * NIMM + decltype(ric)::value) * NOB + ob;
                            static_for<0, NST>([&](auto ic) __attribute__((always_inline)) {
                                constexpr int i = decltype(ic)::value;
                                if constexpr (i * AVAIL / NST == m) store_set(Jc, ic, qst);
                            });
                        }
                    });
                });
            } else {
                constexpr int b = x - NA, s = b / CG, cg = b % CG;
                static_for<0, NOB>([&](auto obc) __attribute__((always_inline)) {
                    constexpr int ob = decltype(obc)::value, f = (s * CG + cg) * NOB + ob;
                    mfma_xw<(f < NAG), (b == 0)>(acc[J][ob], Bq[x % NQ], Wf[ob][s * CG + cg]);
                });
            }
            if constexpr (LD && x == STAGE_X) {
                // stores issued since the loads: those riding MFMAs 0 .. MX-1
                constexpr int MX = (x < NA ? x + 1 : NA) * NIMM * NOB;
                constexpr int NV = [] {
                    int c = 0;
                    for (int i = 0; i < NST; ++i) c += (ST && i * AVAIL / NST < MX) ? 1 : 0;
                    return c;
                }();
                store_row(j + 1, std::integral_constant<int, NV>{});
            }
        });
        // the set finishing in this step (row j - TR + 1) is stored in the next one
        roll_drain(acc[(J + 1) % NSETS]);
        __syncthreads();
    };
    using I0 = std::integral_constant<int, 0>;
    using T_ = std::true_type;
    using F_ = std::false_type;
    // warm-up: input rows 0 .. TR-2 feed only rows 0 .. j
    static_for<0, TR - 1>([&](auto jc) __attribute__((always_inline)) {
        constexpr int jw = decltype(jc)::value;
        step(std::integral_constant<int, jw % NSETS>{}, I0{}, std::integral_constant<int, jw>{}, F_{}, T_{}, jw);
    });
    // first full step (j = TR-1): nothing finished yet
    step(std::integral_constant<int, (TR - 1) % NSETS>{}, I0{}, std::integral_constant<int, TR - 1>{}, F_{},
         T_{}, TR - 1);
    // steady steps j = TR .. nrows-1, TR at a time (set j mod TR = 0, 1, ...)
    int j = TR;
    for (; j + TR <= nrows; j += TR) {
        static_for<0, TR>([&](auto ic) __attribute__((always_inline)) {
            constexpr int i = decltype(ic)::value;
            step(std::integral_constant<int, i>{}, I0{}, std::integral_constant<int, TR - 1>{}, T_{}, T_{}, j + i);
        });
    }
    // (nrows - TR) mod TR = NM leftover steps: sets 0 .. NM-1
    static_for<0, NM>([&](auto ic) __attribute__((always_inline)) {
        constexpr int i = decltype(ic)::value;
        step(std::integral_constant<int, i>{}, I0{}, std::integral_constant<int, TR - 1>{}, T_{}, T_{}, j + i);
    });
    j += NM;   // = nrows
    // tail: input rows nrows .. nrows+TR-2 finish rows nrows-TR+1 .. nrows-1
    static_for<0, TR - 1>([&](auto tc) __attribute__((always_inline)) {
        constexpr int t = decltype(tc)::value;
        step(std::integral_constant<int, (NM + t) % NSETS>{}, std::integral_constant<int, t + 1>{},
             std::integral_constant<int, TR - 1>{}, T_{}, std::bool_constant<(t + 2 < TR)>{}, j + t);
    });
    // the last row (nrows - 1, set (NM + TR - 1) mod TR), drained by the last step
    static_for<0, NST>([&](auto sc) __attribute__((always_inline)) {
        store_set(std::integral_constant<int, (NM + TR - 1) % NSETS>{}, sc, nrows - 1);
    });
}

// ---------------------------------------------------------------- planning

// instantiated shapes: 3x3 with 64 channels and 64-filter blocks; 5x5 with
// 32 channels and 32-filter blocks
static bool roll_shape(int NOB, int TR, int TS, int CG) {
    return (NOB == 2 && TR == 3 && TS == 3 && CG == 4) || (NOB == 1 && TR == 5 && TS == 5 && CG == 2);
}

static int roll_lds(int NOB, int TR, int TS, int CG) {
    const int CIN = CG * 16, PS = 8 * ((CIN / 8) | 1), RPX8 = (kRStrip + TS - 1 + 7) / 8;
    const int ring = 2 * RPX8 * 8 * PS * 2;
    const int RL = CIN * TR * TS;
    const int PW = ((RL * 2 + 239) / 256 * 256 + 16) / 2;
    const int PWB = ((RL * 2 + 111) / 128 * 128 + 16) / 2;
    const int wl = NOB * 32 * (PW > PWB ? PW : PWB) * 2;
    return ring > wl ? ring : wl;
}

// Takes a stride-1 bf16 layer the register-weight strip kernel would run
// when its shape is one the rolling kernel is instantiated for and the tile
// splits into whole strips and equal row segments.
bool igemm_roll_plan(IgemmArgs& a) {
    if (a.bp || a.istr != 1 || a.ostr != 1 || a.oph_r != 0 || a.oph_c != 0) return false;
    if (a.Cin % 16 != 0 || a.Cout % 32 != 0 || a.Vo % kRStrip != 0) return false;
    if (a.base_c % 8 != 0 || a.in_pitch % 8 != 0 || a.Tr != a.R || a.Ts != a.S) return false;
    const int NOB = a.Cout % 64 == 0 ? 2 : 1, CG = a.Cin / 16;
    if (!roll_shape(NOB, a.Tr, a.Ts, CG)) return false;
    if (a.wmode == 0 && !(a.wr0 == 0 && a.wrstep == 1 && a.ws0 == 0 && a.wsstep == 1)) return false;
    if (a.wmode == 1 && !(a.wr0 == a.R - 1 && a.wrstep == -1 && a.ws0 == a.S - 1 && a.wsstep == -1))
        return false;
    const int T = a.R * a.S;
    if (a.wmode == 0 && (int64_t(a.Cin) * T) % 8 != 0) return false;
    if (a.wmode == 1 && (int64_t(a.Cout) * T) % 8 != 0) return false;
    // 32-bit buffer offsets
    const int64_t in_plane = int64_t(a.in_rows) * a.in_pitch, oplane = int64_t(a.out_rows) * a.out_cols;
    if (int64_t(a.Cin) * in_plane * 2 >= (int64_t(1) << 31) || 64 * oplane * 4 >= (int64_t(1) << 31)) return false;
    if (a.out_rows < a.Uo || a.out_cols < a.Vo) return false;
    const int lds = roll_lds(NOB, a.Tr, a.Ts, CG);
    if (lds > device_lds_limit()) return false;
    // equal segments of at least TR rows, about 256 workgroups
    a.nvb = a.Vo / kRStrip;
    const int strips = a.ntiles * a.Nn * a.nvb * (a.Cout / (32 * NOB));
    int best = 0;
    for (int rps = a.Tr; rps <= a.Uo; ++rps) {
        if (a.Uo % rps != 0) continue;
        best = rps;
        if (int64_t(strips) * (a.Uo / rps) <= 256) break;
    }
    if (best == 0) return false;
    a.rows_per_seg = best;
    a.nseg = a.Uo / best;
    a.OB = 32 * NOB;
    a.wvec = 1;
    a.phase = 0;
    a.lds_bytes = lds;
    a.kind = 3;
    return true;
}

template <int NOB, int TR, int TS, int CG, int NM>
static hipError_t launch_roll(const IgemmArgs& a, hipStream_t s) {
    auto k = igemm_roll_kernel<NOB, TR, TS, CG, NM>;
    if (a.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, a.lds_bytes);
        if (e != hipSuccess) return e;
    }
    dim3 grid(a.ntiles * a.Nn * a.nvb * a.nseg, a.Cout / (32 * NOB));
    hipLaunchKernelGGL(k, grid, dim3(kRThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_igemm_roll(const IgemmArgs& a, hipStream_t s) {
    const int CG = a.Cin / 16;
    if (a.OB == 64 && a.Tr == 3 && a.Ts == 3 && CG == 4 && a.rows_per_seg >= 3) {
        switch (a.rows_per_seg % 3) {
            case 0: return launch_roll<2, 3, 3, 4, 0>(a, s);
            case 1: return launch_roll<2, 3, 3, 4, 1>(a, s);
            default: return launch_roll<2, 3, 3, 4, 2>(a, s);
        }
    }
    if (a.OB == 32 && a.Tr == 5 && a.Ts == 5 && CG == 2 && a.rows_per_seg >= 5) {
        switch (a.rows_per_seg % 5) {
            case 0: return launch_roll<1, 5, 5, 2, 0>(a, s);
            case 1: return launch_roll<1, 5, 5, 2, 1>(a, s);
            case 2: return launch_roll<1, 5, 5, 2, 2>(a, s);
            case 3: return launch_roll<1, 5, 5, 2, 3>(a, s);
            default: return launch_roll<1, 5, 5, 2, 4>(a, s);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace dc
