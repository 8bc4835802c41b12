// Weight gradient on a padded tile (Eq. (2) of Sec. II-A restricted to the
// tile, Sec. III-A) as a GEMM whose reduction runs over output pixels:
//
//   dw[o][ci, r, s] = sum_{pixels} dy[o][pixel] * x[ci][pixel shifted by (r, s)]
//
// NCHW keeps both operands contiguous along the reduction (pixels), so no
// transpose is needed.  The pixels of a tile are split into chunks; each
// workgroup reduces one chunk into a partial in the workspace, and a second
// kernel adds the partials in chunk order (fixed order, no atomics:
// deterministic).  Only the interior of the dy tile is read -- the weight
// gradient needs no dy halo (Sec. III-A).
//
// Strip kernel (bf16, stride 1): a workgroup walks down a 64-column strip of
// one sample.  x rows live in an LDS ring (a new row per output row, the
// filter rows reuse the previous ones) next to a double-buffered dy row; the
// next row's 16-byte global loads are in flight while the current row runs
// on v_mfma_f32_32x32x16_bf16.  Four waves = 2 blocks of 32 filters x 2
// blocks of 32 channels; each wave keeps its 32 x 32 block at every tap of
// its filter rows in accumulators.  A k-step is 16 pixels (8 per half-wave);
// the 8 pixels a lane feeds for tap s start s elements into the staged x row,
// cut from two aligned 16-byte LDS reads with byte-align operations.
// Partials are stored in MFMA fragment order (coalesced) and mapped back to
// the dw layout by the reduction.
//
// Row kernels (general fallback: bf16 stride > 1, fp32): stage one output row
// segment per step; partials in dw order.  fp32 uses v_mfma_f32_32x32x2_f32
// with flattened (ci, r, s) columns in blocks of 32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>

#include "bf16util.h"
#include "kernels.h"

namespace dc {

typedef float f32x4v __attribute__((ext_vector_type(4)));

static constexpr int kThreads = 256;
static constexpr int kBQ = 64;          // output columns staged per step
static constexpr int kTargetWGs = 256;  // workgroups aimed for per launch (one per CU)
static constexpr int kDepth = 2;        // strip kernel: steps between a row's loads and its use


// ---------------------------------------------------------------- planning

static int bf16_trb(int S) { return std::max(1, 9 / S); }

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
static constexpr int kXP = 72;    // strip kernel: staged x row pitch (bf16): 9 x 16 bytes

struct Plan {
    int kind, gy, gz, TRB, nchunks;
    int chunks_per_tile, rows_per_chunk;
    int nqb, nseg, rows_per_seg;
    int64_t F;
    int frag;
};

// tap-split kernel: square filters whose R*S taps spread over four waves fit
// the accumulators (at most 14 tiles of 32x32 per wave)
static bool taps_filter(int R, int S) { return R == S && R >= 2 && R <= 7; }
// stride-2 tap-split kernel: instantiated phase filters (ceil(R/2) of 2 to 4,
// square), i.e. filters of 3 x 3 to 8 x 8
static bool taps2_filter(int R, int S) {
    const int rp = (R + 1) / 2, sp = (S + 1) / 2;
    return rp == sp && rp >= 2 && rp <= 4;
}

// k-slice kernel geometry (kernel below)
template <int NW>
struct KsliceGeom {
    static constexpr int QW = 16 * NW;            // output columns per strip
    static constexpr int XU8 = 2 * NW + 1;        // 16-byte chunks per staged row (QW + 8 columns)
    static constexpr int P = 8 * XU8;             // staged row pitch (elements): rows 4 banks apart
    static constexpr int NI = (32 * XU8 + 63) / 64;   // 64-chunk loads per staged block (x or dy)
    static constexpr int REG = NI * 64 * 8;       // elements of a block's region (spare chunks at the end)
    static constexpr int BUF = 2 * REG + 64 * 8;  // x region, dy region, 64 chunks nobody reads (prologue)
    static constexpr int LPW = (2 * NI + NW - 1) / NW;   // loads per wave per step
    static constexpr int kDepth = 5;              // steps between a row's request and its use
    static constexpr int nbuf = kDepth + 1;       // step buffers (a barrier every second step)
    static constexpr int loop_lds = (nbuf + 2) * BUF * 2;   // + the first two window rows (3-row filters)
};

// k-slice kernel: instantiated filters, and whether a sample's x and dy
// planes are addressed with 32-bit byte offsets (a bound that holds for any
// halo up to the tile size)
static bool kslice_filter(int R, int S) { return R == 3 && S == 3; }
static constexpr int kKsliceNW = 8;   // waves of the k-slice kernel (strip of 16 * NW columns)
// layers whose staged elements all lie inside the tile: whole 32-blocks of
// channels and filters, whole strips, halo at least the padding (x window
// rows and columns inside the tile), dy columns at most one element past a
// 16-byte boundary
static bool kslice_layer(int C, int K, int R, int S, int Wot, int base_c, int dy_off) {
    return kslice_filter(R, S) && C % 32 == 0 && K % 32 == 0 && Wot % (16 * kKsliceNW) == 0 &&
           base_c >= 0 && base_c % 8 == 0 && (dy_off & 7) <= 1;
}
static bool kslice_offsets_fit(int C, int K, int R, int S, int Hot, int Wot) {
    const int64_t rows = 3 * (int64_t(Hot) + R + 8), cols = 3 * (int64_t(Wot) + S + 16);
    return 2 * int64_t(std::max(C, K)) * rows * cols < (int64_t(1) << 32);
}
// fp32 flattened-column kernel: compiled for a channel capacity class (the
// smallest of 4, 8, .., 32 that holds C, and 18 for the mesh layer's 17-18;
// 0: none) and 3x3 or 1x1 filters; it runs any C up to its class
static int f32w_class(int C) {
    if (C < 1 || C > 32) return 0;
    if (C == 17 || C == 18) return 18;
    return (C + 3) / 4 * 4;
}
static bool f32w_shape(int C, int R, int S) {
    return f32w_class(C) > 0 && ((R == 3 && S == 3) || (R == 1 && S == 1));
}
static int f32w_lds(int C, int R, int S) {
    const int XW = 64 + S - 1 + 3, XWP = (XW + 3) / 4 * 4 + 4, DYP = 17 * 4 + 4;
    const int ring = ((R + 1) * C * XWP + 2 * 32 * DYP) * 4;
    const int red = 4 * ((C * R * S + 31) / 32) * 1024 * 4;
    return ring > red ? ring : red;
}

static bool make_plan(int dtype, int ntiles, int N, int C, int K, int R, int S, int stride,
                      int Hot, int Wot, int base_c, int dy_off, Plan* pl) {
    std::memset(pl, 0, sizeof(*pl));
    const bool xcol_aligned = base_c % 8 == 0;   // strip staging reads whole 16-byte x chunks
    const bool phase2 = dtype == 1 && stride == 2 && 4 * C <= 32 && xcol_aligned && taps2_filter(R, S);
    if ((dtype == 1 && stride == 1 && S <= 7 && xcol_aligned) || phase2) {
        int qw = kBQ;   // strip width
        if (phase2) {
            // the phase images: a stride-1 ceil(R/2) x ceil(S/2) filter on 4C channels
            pl->kind = WGRAD_TAPS2_BF16;
            pl->TRB = (R + 1) / 2;
            pl->gy = 1;
            pl->gz = (K + 31) / 32;
            pl->frag = 3;
        } else if (kslice_layer(C, K, R, S, Wot, base_c, dy_off) &&
                   kslice_offsets_fit(C, K, R, S, Hot, Wot)) {
            // 32x32 blocks over strips of 16 * NW columns, every tap in one workgroup
            pl->kind = WGRAD_KSLICE_BF16;
            pl->TRB = R;
            pl->gy = 1;
            pl->gz = ((K + 31) / 32) * ((C + 31) / 32);
            pl->frag = 5;
            qw = 16 * kKsliceNW;
        } else if (C <= 32 && K <= 32 && taps_filter(R, S)) {
            // one 32x32 block, every tap in one row group: x and dy are read once
            pl->kind = WGRAD_TAPS_BF16;
            pl->TRB = R;
            pl->gy = 1;
            pl->gz = 1;
            pl->frag = 2;
        } else {
            pl->kind = WGRAD_STRIP_BF16;
            // filter rows per workgroup: the largest divisor of R that fits the
            // accumulators (rows x S <= 9 tiles of 32x32), so every group is full
            int trb = 1;
            for (int d = 1; d <= std::min(bf16_trb(S), R); ++d)
                if (R % d == 0) trb = d;
            pl->TRB = trb;
            pl->gy = (R + pl->TRB - 1) / pl->TRB;
            pl->gz = ((K + 63) / 64) * ((C + 63) / 64);
            pl->frag = 1;
        }
        pl->nqb = (Wot + qw - 1) / qw;
        const int strips = ntiles * N * pl->nqb;
        const int want = std::max(1, kTargetWGs / (pl->gy * pl->gz));
        int nseg = std::max(1, std::min(Hot, (want + strips - 1) / strips));
        pl->rows_per_seg = (Hot + nseg - 1) / nseg;
        pl->nseg = (Hot + pl->rows_per_seg - 1) / pl->rows_per_seg;
        pl->nchunks = strips * pl->nseg;
        const int SP = phase2 ? (S + 1) / 2 : S;   // filter width the kernel walks
        pl->F = int64_t(pl->gy) * pl->gz * (pl->frag == 1 ? 4 : 1) * pl->TRB * SP * 1024;
        return true;
    }
    if (dtype == 0 && stride == 1 && f32w_shape(C, R, S)) {
        pl->kind = WGRAD_F32W;
        pl->TRB = R;
        pl->gy = 1;
        pl->gz = (K + 31) / 32;
        pl->nqb = (Wot + kBQ - 1) / kBQ;
        const int strips = ntiles * N * pl->nqb;
        const int want = std::max(1, kTargetWGs / pl->gz);
        int nseg = std::max(1, std::min(Hot, (want + strips - 1) / strips));
        pl->rows_per_seg = (Hot + nseg - 1) / nseg;
        pl->nseg = (Hot + pl->rows_per_seg - 1) / pl->rows_per_seg;
        pl->nchunks = strips * pl->nseg;
        pl->F = int64_t(pl->gz) * ((C * R * S + 31) / 32) * 1024;
        pl->frag = 4;
        return true;
    }
    if (dtype == 1) {
        if (S > 7) return false;
        pl->kind = WGRAD_ROWS_BF16;
        pl->TRB = std::min(bf16_trb(S), R);
        pl->gy = (R + pl->TRB - 1) / pl->TRB;
        pl->gz = ((K + 63) / 64) * ((C + 63) / 64);
    } else {
        const int NCB = (C * R * S + 31) / 32;
        pl->kind = WGRAD_ROWS_F32;
        pl->TRB = R;
        pl->gy = (NCB + 7) / 8;   // 4 waves x 2 column blocks per workgroup
        pl->gz = (K + 63) / 64;
    }
    const int rows = N * Hot;
    const int want = std::max(1, kTargetWGs / (pl->gy * pl->gz));
    const int cpt = std::max(1, std::min(rows, (want + ntiles - 1) / ntiles));
    pl->rows_per_chunk = (rows + cpt - 1) / cpt;
    pl->chunks_per_tile = (rows + pl->rows_per_chunk - 1) / pl->rows_per_chunk;
    pl->nchunks = ntiles * pl->chunks_per_tile;
    pl->F = int64_t(K) * C * R * S;
    pl->frag = 0;
    return true;
}

size_t wgrad_workspace_bytes(int dtype, int ntiles, int N, int C, int K, int R, int S,
                             int stride, int Hot, int Wot, int base_c, int dy_off) {
    Plan pl;
    if (!make_plan(dtype, ntiles, N, C, K, R, S, stride, Hot, Wot, base_c, dy_off, &pl)) return 0;
    return size_t(pl.nchunks) * size_t(pl.F) * sizeof(float);
}

bool wgrad_plan(WgradArgs& a, int dtype) {
    Plan pl;
    if (!make_plan(dtype, a.ntiles, a.Nn, a.C, a.K, a.R, a.S, a.istr, a.Hot, a.Wot, a.base_c, a.dy_off,
                   &pl))
        return false;
    a.kind = pl.kind; a.gy = pl.gy; a.gz = pl.gz; a.TRB = pl.TRB; a.nchunks = pl.nchunks;
    a.chunks_per_tile = pl.chunks_per_tile; a.rows_per_chunk = pl.rows_per_chunk;
    a.nqb = pl.nqb; a.nseg = pl.nseg; a.rows_per_seg = pl.rows_per_seg;
    a.F = pl.F; a.frag = pl.frag;
    if (a.kind == WGRAD_F32W) {
        a.lds_bytes = f32w_lds(f32w_class(a.C), a.R, a.S);
    } else if (a.kind == WGRAD_KSLICE_BF16) {
        // the staging buffers; after the loop the waves' sums (NW/2 of them at once)
        const int bufs = KsliceGeom<kKsliceNW>::loop_lds;
        const int red = kKsliceNW * ((4 * a.R * a.S + 1) / 2) * 1024;
        a.lds_bytes = std::max(bufs, red);
    } else if (a.kind == WGRAD_STRIP_BF16 || a.kind == WGRAD_TAPS_BF16 || a.kind == WGRAD_TAPS2_BF16) {
        const int cb = a.kind == WGRAD_STRIP_BF16 ? 64 : 32;
        a.lds_bytes = ((a.TRB + 1) * cb * kXP + 2 * cb * kXP) * 2;
    } else if (a.kind == WGRAD_ROWS_BF16) {
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

// ---------------------------------------------------------------- strip kernel (bf16)

// Three ways to share a workgroup's block among its waves:
//  * kBlock64 (4 waves): 64 filters x 64 channels; wave = (filter half,
//    channel half), each wave accumulates its 32 x 32 block at every tap of
//    the row group;
//  * kPair64 (8 waves): the same block, two waves per 32 x 32 sub-block that
//    split its taps: by filter rows (first ceil(TRB/2) rows / the rest), so
//    that the two read disjoint x rows, or, for one row, its taps.  Two waves per
//    SIMD: one wave's LDS reads, byte-aligns and staging issue while the
//    other's matrix instructions run, which a single wave cannot overlap;
//  * kTapSplit (4 waves): one 32 x 32 block (small channel counts); the row
//    group's taps are dealt to the waves in four contiguous runs.
// In every mode a wave reads only the x rows its taps touch.
enum StripMode { kBlock64 = 0, kTapSplit = 1, kPair64 = 2 };

template <int MODE, int TRB, int SS>
struct TapRange {   // taps [first(W), first(W) + count(W)) of wave group W
    static constexpr int NT = TRB * SS;
    static constexpr int PAIR0 = TRB >= 2 ? (TRB + 1) / 2 * SS : (SS + 1) / 2;   // taps of group 0
    static constexpr int first(int W) {
        return MODE == kBlock64 ? 0
             : MODE == kPair64  ? (W == 0 ? 0 : PAIR0)
                                : W * (NT / 4) + (W < NT % 4 ? W : NT % 4);
    }
    static constexpr int count(int W) {
        return MODE == kBlock64 ? NT
             : MODE == kPair64  ? (W == 0 ? PAIR0 : NT - PAIR0)
                                : NT / 4 + (W < NT % 4 ? 1 : 0);
    }
};
template <int MODE> struct StripThreads { static constexpr int value = MODE == kPair64 ? 512 : 256; };

// PH (stride 2): the strided correlation is run as a stride-1 one over the
// four phase images x[ci][2i + pr][2j + pc]: phase channel c' = 4 ci + 2 pr
// + pc, phase taps (r', s') with r = 2 r' + pr, s = 2 s' + pc (Eq. (2) with
// the sum over the filter split by the parity of r and s).  Staging loads
// the two x rows of a phase row and keeps every other column; SS and TRB are
// then the phase filter's width and height.
template <int SS, int TRB, int MODE, int W, bool PH = false>
__device__ __forceinline__ void strip_body(const WgradArgs& a, unsigned char* smem) {
    constexpr int CB = MODE == kTapSplit ? 32 : 64;         // channels / filters staged
    constexpr int NTH = StripThreads<MODE>::value;
    constexpr int NR = TRB + 1;                             // x ring slots
    uint16_t* xring = reinterpret_cast<uint16_t*>(smem);    // [NR][CB ci][kXP]
    uint16_t* dyb = xring + NR * CB * kXP;                  // [2][CB o][kXP]
    constexpr int NT = TRB * SS;                            // taps of the row group
    constexpr int FST = TapRange<MODE, TRB, SS>::first(W), FCNT = TapRange<MODE, TRB, SS>::count(W);
    constexpr int RLO = FST / SS, NRW = (FST + FCNT - 1) / SS - RLO + 1;   // x rows this wave reads

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int qb = c % a.nqb; c /= a.nqb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int p0 = seg * a.rows_per_seg;
    const int nrows = min(a.rows_per_seg, a.Hot - p0);
    const int q0 = qb * kBQ;
    const int r0 = blockIdx.y * TRB;
    constexpr int nTR = TRB;                      // the plan makes every row group full
    const int Cst = PH ? 4 * a.C : a.C;           // channels of the staged image
    const int ncsb = (Cst + CB - 1) / CB;
    const int o0 = (blockIdx.z / ncsb) * CB, c0 = (blockIdx.z % ncsb) * CB;

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;
    const int ow = MODE == kTapSplit ? 0 : wave & 1, cw = MODE == kTapSplit ? 0 : (wave >> 1) & 1;

    const uint16_t* xt = static_cast<const uint16_t*>(a.x) + tile * a.x_tile +
                         int64_t(n) * a.C * a.x_rows * a.x_pitch;
    const int dy_rows = a.Hot + 2 * a.dy_off;
    const uint16_t* dyt = static_cast<const uint16_t*>(a.dy) + tile * a.dy_tile +
                          int64_t(n) * a.K * dy_rows * a.dy_pitch;
    const int64_t xplane = int64_t(a.x_rows) * a.x_pitch;
    const int64_t dyplane = int64_t(dy_rows) * a.dy_pitch;
    const int xg0 = (PH ? 2 * q0 : q0) + a.base_c; // global column of staged x column 0
    const int dyg0 = q0 + a.dy_off;                // global column of staged dy column 0
    const int dy_end = a.dy_off + a.Wot;           // dy interior ends here
    const int xrow0 = PH ? p0 + r0 : p0 + a.base_r + r0;   // x row (PH: phase row) of ring row 0
    const int dysh = dyg0 & 7, dya0 = dyg0 - dysh;

    // staging units: x row = CB channels x 9 groups of 8; dy row = CB filters x 8 groups
    constexpr int XU = CB * 9, DU = CB * 8;
    constexpr int XPT = (XU + NTH - 1) / NTH, DPT = DU / NTH;
    static_assert(DPT * NTH == DU, "dy units must spread evenly over the threads");
    // Staging in two phases so that global loads overlap the MFMAs:
    // load_*() only issues unconditional 16-byte loads from clamped addresses
    // into registers; store_*() (after the next row's MFMAs) shifts the
    // misaligned dy chunks, zeroes everything outside the tile and writes LDS.
    // kDepth register buffers: the data of step j (x row j+nTR-1, dy row j)
    // is loaded at the start of step j-kDepth and stored to LDS at the end of
    // step j-1; buffer j % kDepth holds it.
    struct Regs {
        uint4 x[XPT];
        uint4 x2[PH ? XPT : 1];   // PH: the next 8 columns (a phase row needs 16 x columns per 8)
        uint4 d0[DPT], d1[DPT];
    };
    Regs buf[kDepth];

    auto load_x = [&](int m, Regs& r) {   // ring row m -> registers
#pragma unroll
        for (int k = 0; k < XPT; ++k) {
            const int u = min(tid + k * NTH, XU - 1);
            const int ci = u / 9, g8 = u - ci * 9;
            if constexpr (PH) {
                const int cp = min(c0 + ci, Cst - 1), pr = (cp >> 1) & 1;
                const int gr = min(max(2 * (xrow0 + m) + pr + a.base_r, 0), a.x_rows - 1);
                const uint16_t* row = xt + (cp >> 2) * xplane + int64_t(gr) * a.x_pitch;
                r.x[k] = *reinterpret_cast<const uint4*>(row + min(xg0 + 16 * g8, a.x_pitch - 8));
                r.x2[k] = *reinterpret_cast<const uint4*>(row + min(xg0 + 16 * g8 + 8, a.x_pitch - 8));
            } else {
                const int gr = min(max(xrow0 + m, 0), a.x_rows - 1);
                const int gc = min(xg0 + 8 * g8, a.x_pitch - 8);
                r.x[k] = *reinterpret_cast<const uint4*>(xt + min(c0 + ci, a.C - 1) * xplane +
                                                         int64_t(gr) * a.x_pitch + gc);
            }
        }
    };
    auto store_x = [&](int m, Regs& r) {
        uint16_t* slot = xring + (m % NR) * CB * kXP;
        if constexpr (PH) {
            // columns 2j + pc of the two loaded chunks; zero outside the tile
#pragma unroll
            for (int k = 0; k < XPT; ++k) {
                const int u = min(tid + k * NTH, XU - 1);
                const int ci = u / 9, g8 = u - ci * 9;
                const int cp = c0 + ci, pr = (cp >> 1) & 1, pc = cp & 1;
                const int gr = 2 * (xrow0 + m) + pr + a.base_r;
                const int col = xg0 + 16 * g8 + pc;   // x column of element 0
                const int nv = (gr >= 0 && gr < a.x_rows && cp < Cst && col < a.x_cols)
                                   ? (a.x_cols - col + 1) / 2 : 0;
                const uint32_t sw[8] = {r.x[k].x, r.x[k].y, r.x[k].z, r.x[k].w,
                                        r.x2[k].x, r.x2[k].y, r.x2[k].z, r.x2[k].w};
                uint32_t o[4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    o[j] = pc ? ((sw[2 * j] >> 16) | (sw[2 * j + 1] & 0xffff0000u))
                              : ((sw[2 * j] & 0xffffu) | (sw[2 * j + 1] << 16));
                if (NT > 1 || tid + k * NTH < XU)
                    *reinterpret_cast<uint4*>(slot + ci * kXP + 8 * g8) =
                        mask8(make_uint4(o[0], o[1], o[2], o[3]), nv);
            }
            return;
        }
        const int gr = xrow0 + m;
        const bool rok = gr >= 0 && gr < a.x_rows;
        // With several taps the staging stays branch-free, so that it can sit
        // in the MFMA stream: units past XU repeat unit XU-1 (same clamped
        // load, same mask) and their duplicate stores write identical bytes.
        // A single tap leaves nothing to overlap: skip the duplicates.
#pragma unroll
        for (int k = 0; k < XPT; ++k) {
            const int u = min(tid + k * NTH, XU - 1);
            const int ci = u / 9, g8 = u - ci * 9;
            const int nv = (rok && c0 + ci < a.C) ? a.x_cols - (xg0 + 8 * g8) : 0;
            if (NT > 1 || tid + k * NTH < XU)
                *reinterpret_cast<uint4*>(slot + ci * kXP + 8 * g8) = mask8(r.x[k], nv);
        }
    };
    auto load_dy = [&](int i, Regs& r) {   // output row p0 + i -> registers (clamped)
        const int gr = min(p0 + i + a.dy_off, dy_rows - 1);
#pragma unroll
        for (int k = 0; k < DPT; ++k) {
            const int u = tid + k * NTH;
            const int o = u >> 3, g8 = u & 7;
            const uint16_t* row = dyt + min(o0 + o, a.K - 1) * dyplane + int64_t(gr) * a.dy_pitch;
            const int ga = dya0 + 8 * g8;
            r.d0[k] = *reinterpret_cast<const uint4*>(row + min(ga, a.dy_pitch - 8));
            r.d1[k] = *reinterpret_cast<const uint4*>(row + min(ga + 8, a.dy_pitch - 8));
        }
    };
    auto store_dy = [&](int i, Regs& r) {
        uint16_t* slot = dyb + (i & 1) * CB * kXP;
#pragma unroll
        for (int k = 0; k < DPT; ++k) {
            const int u = tid + k * NTH;
            const int o = u >> 3, g8 = u & 7;
            const uint4 v0 = r.d0[k];
            const uint32_t d[8] = {v0.x, v0.y, v0.z, v0.w, r.d1[k].x, r.d1[k].y, r.d1[k].z, r.d1[k].w};
            uint4 v = v0;
            if constexpr (NT > 1)
                v = window8_sel(d, dysh);
            else if (dysh != 0)
                v = window8_rt(d, dysh);
            const int nv = (o0 + o < a.K) ? dy_end - (dyg0 + 8 * g8) : 0;
            *reinterpret_cast<uint4*>(slot + o * kXP + 8 * g8) = mask8(v, nv);
        }
    };

    // accumulators (one per tap of this wave) live in AGPRs (the MFMAs are
    // written out, see mfma32x32x16); the empty statement after zeroing
    // settles them there
    floatx16 acc[FCNT];
#pragma unroll
    for (int j = 0; j < FCNT; ++j) {
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
        asm volatile("s_nop 2" : "+a"(acc[j]));
    }

    // prologue: the filter rows of the first output row and its dy row (two
    // rows in flight at a time), then the loads of steps 1 .. kDepth-1
    load_dy(0, buf[0]);
    for (int m = 0; m < nTR; m += 2) {
        load_x(m, buf[0]);
        if (m + 1 < nTR) load_x(m + 1, buf[1]);
        store_x(m, buf[0]);
        if (m + 1 < nTR) store_x(m + 1, buf[1]);
    }
    store_dy(0, buf[0]);
    static_for<1, kDepth>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        load_x(j + nTR - 1, buf[j]);
        load_dy(j, buf[j]);
    });
    __syncthreads();

    // One k-step = 16 pixels: the dy chunk (A) of this lane's filter row and,
    // per filter row the wave's taps touch, the 8 + (SS - 1) staged x
    // elements from which the SS shifted windows (B) are cut.  The LDS reads
    // of k-step kq+1 are issued before the MFMAs of k-step kq.
    constexpr int XH = SS <= 3 ? 1 : SS <= 5 ? 2 : 4;   // dwords read past the first 8 elements
    struct KData {
        uint4 A;
        uint32_t x[NRW][4 + XH];
    };
    // Loads and LDS stores are unconditional (rows past the chunk are clamped
    // reads, staged into slots no later step reads): with no branches around
    // them the wait for the loads of two steps back leaves the newer ones in
    // flight.
    auto step = [&](int i, Regs& cur, Regs& nxt) __attribute__((always_inline)) {
        const uint16_t* dyrow = dyb + (i & 1) * CB * kXP + (ow * 32 + l32) * kXP;
        const uint16_t* xrows[NRW];
#pragma unroll
        for (int tr = 0; tr < NRW; ++tr)
            xrows[tr] = xring + ((i + RLO + tr) % NR) * CB * kXP + (cw * 32 + l32) * kXP;
        auto read_k = [&](int kq, KData& d) {
            const int qc = kq * 16 + 8 * hi;
            d.A = *reinterpret_cast<const uint4*>(dyrow + qc);
#pragma unroll
            for (int tr = 0; tr < NRW; ++tr) {
                const uint4 lo = *reinterpret_cast<const uint4*>(xrows[tr] + qc);
                d.x[tr][0] = lo.x; d.x[tr][1] = lo.y; d.x[tr][2] = lo.z; d.x[tr][3] = lo.w;
                if constexpr (XH == 1) {
                    d.x[tr][4] = *reinterpret_cast<const uint32_t*>(xrows[tr] + qc + 8);
                } else if constexpr (XH == 2) {
                    const uint2 h = *reinterpret_cast<const uint2*>(xrows[tr] + qc + 8);
                    d.x[tr][4] = h.x; d.x[tr][5] = h.y;
                } else {
                    const uint4 h = *reinterpret_cast<const uint4*>(xrows[tr] + qc + 8);
                    d.x[tr][4] = h.x; d.x[tr][5] = h.y; d.x[tr][6] = h.z; d.x[tr][7] = h.w;
                }
            }
        };
        // MFMAs of one k-step; `mid` runs after the first `at` of them, so that
        // its VALU and memory work issues while the matrix cores are busy
        auto mfmas_k = [&](const KData& d, auto at, auto&& mid) {
            Pack8 A;
            A.v = d.A;
            constexpr int AT0 = decltype(at)::value;
            constexpr int AT = AT0 < 0 ? -1 : (AT0 < FCNT ? AT0 : FCNT - 1);
            static_for<0, FCNT>([&](auto jc) {
                constexpr int j = decltype(jc)::value, f = FST + j;
                constexpr int tr = f / SS - RLO, s = f % SS;
                if constexpr (j == AT) mid();
                Pack8 B;
                uint32_t* o = B.d;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if constexpr ((s & 1) == 0)
                        o[j] = d.x[tr][s / 2 + j];
                    else
                        o[j] = __builtin_amdgcn_alignbyte(d.x[tr][s / 2 + j + 1], d.x[tr][s / 2 + j], 2);
                }
                floatx16& ac = acc[j];
                const bf16x8 av = A.b, bv = B.b;
                // B is written by VALU (byte-align or register copies) just before
                if constexpr (s == 0)
                    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(ac) : "v"(av), "v"(bv));
                else
                    asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                                 : "+a"(ac) : "v"(av), "v"(bv));
            });
        };
        constexpr int NK = kBQ / 16;
        KData kd[2];
        read_k(0, kd[0]);
        static_for<0, NK>([&](auto kc) {
            constexpr int kq = decltype(kc)::value;
            if constexpr (kq + 1 < NK) read_k(kq + 1, kd[(kq + 1) & 1]);
            if constexpr (kq == 0) {
                // step i+kDepth's data: kDepth steps of MFMAs to arrive
                mfmas_k(kd[0], std::integral_constant<int, 1>{}, [&] {
                    load_x(i + kDepth + nTR - 1, cur);
                    load_dy(i + kDepth, cur);
                });
            } else if constexpr (kq == NK - 1) {
                // step i+1's data (loaded during step i-1) into slots this step does not read
                mfmas_k(kd[kq & 1], std::integral_constant<int, 1>{}, [&] {
                    store_x(i + nTR, nxt);
                    store_dy(i + 1, nxt);
                });
            } else {
                mfmas_k(kd[kq & 1], std::integral_constant<int, -1>{}, [] {});
            }
        });
        __syncthreads();
    };
    // unrolled by kDepth so that every buffer index is a constant: step i+j
    // loads into buffer j (step i+j+kDepth) and stores buffer j+1 (step i+j+1)
    int i = 0;
    for (; i + kDepth <= nrows; i += kDepth)
        static_for<0, kDepth>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            step(i + j, buf[j], buf[(j + 1) % kDepth]);
        });
    static_for<0, kDepth - 1>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        if (i + j < nrows) step(i + j, buf[j], buf[(j + 1) % kDepth]);
    });
#pragma unroll
    for (int j = 0; j < FCNT; ++j) mfma_drain(acc[j]);

    // partial in fragment order: kBlock64 / kPair64 [chunk][gy][gz][sub-block][tap][16][64],
    // kTapSplit [chunk][gy][gz][tap][16][64] (tap = tr * SS + s)
    const int64_t blk = int64_t(blockIdx.y) * a.gz + blockIdx.z;
    float* part = a.part + int64_t(blockIdx.x) * a.F +
                  (MODE == kTapSplit ? blk * NT + FST : (blk * 4 + (wave & 3)) * NT + FST) * 1024;
#pragma unroll
    for (int j = 0; j < FCNT; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) part[j * 1024 + e * 64 + lane] = acc[j][e];
}

template <int SS, int TRB>
__global__ __launch_bounds__(kThreads) void wgrad_strip_bf16_kernel(WgradArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    strip_body<SS, TRB, kBlock64, 0>(a, smem);
}

// the wave index selects the (compile-time) tap run; the branch is uniform
template <int SS, int TRB>
__global__ __launch_bounds__(512) void wgrad_pair_bf16_kernel(WgradArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    if (threadIdx.x < 256)
        strip_body<SS, TRB, kPair64, 0>(a, smem);
    else
        strip_body<SS, TRB, kPair64, 1>(a, smem);
}

// stride 2, at most 8 channels (32 phase channels): the tap-split kernel on
// the phase images
template <int SS, int TRB>
__global__ __launch_bounds__(kThreads) void wgrad_taps2_bf16_kernel(WgradArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    switch (threadIdx.x >> 6) {
        case 0: strip_body<SS, TRB, kTapSplit, 0, true>(a, smem); break;
        case 1: strip_body<SS, TRB, kTapSplit, 1, true>(a, smem); break;
        case 2: strip_body<SS, TRB, kTapSplit, 2, true>(a, smem); break;
        default: strip_body<SS, TRB, kTapSplit, 3, true>(a, smem); break;
    }
}

template <int SS, int TRB>
__global__ __launch_bounds__(kThreads) void wgrad_taps_bf16_kernel(WgradArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    switch (threadIdx.x >> 6) {
        case 0: strip_body<SS, TRB, kTapSplit, 0>(a, smem); break;
        case 1: strip_body<SS, TRB, kTapSplit, 1>(a, smem); break;
        case 2: strip_body<SS, TRB, kTapSplit, 2>(a, smem); break;
        default: strip_body<SS, TRB, kTapSplit, 3>(a, smem); break;
    }
}

// ---------------------------------------------------------------- k-slice kernel (bf16)
//
// One 32 x 32 block (filters o0 .. o0+31, channels c0 .. c0+31) per workgroup
// over a strip of 16 * NW output columns of one sample.  Wave w owns pixels
// [16 w, 16 w + 16) of every output row (one MFMA k-step) and keeps all TR x SS
// taps of the block in accumulators.  Per output row a wave reads from LDS
// one dy fragment (A) and the fragment of the single x row that enters the
// filter window (into the registers of the row that leaves it, once that
// row's MFMAs have issued); the other TR - 1 x fragments stay in registers.
// With four times fewer workgroups per output block than the 64 x 64 strip
// kernel the partials are four times smaller.  At the end the waves' sums are
// added in LDS in a fixed tree order (deterministic) and wave 0 stores the
// partial in fragment order [chunk][block][tap][16][64].
//
// Staging copies rows global -> LDS with the 16-byte direct loads of gfx950
// (lane l's 16 bytes land at the wave's LDS base + 16 l): no registers and no
// VALU, so the rows of a step are requested kDepth steps ahead.  The plan
// admits only layers where every staged element an MFMA reads lies inside
// the tile (channels and filters in whole blocks of 32, whole strips, halo >=
// padding), so nothing is masked.  The data of step j (x row j + TR - 1 of the
// window, dy row j) goes to buffer j % nbuf: requested in step j - kDepth,
// read into registers in step j - 1, multiplied in step j.  A barrier ends
// every odd step, after each wave has waited for its loads of the next two
// steps' data; with nbuf = kDepth + 1 a buffer is requested again only after
// a barrier has passed its last read.

// unit range [lo, hi) of range index k (r bits, first halving first) after r
// halvings of [0, n): bit 0 keeps the lower half, bit 1 the upper
__host__ __device__ constexpr int ks_lo(int n, int r, int k) {
    int lo = 0, hi = n;
    for (int b = r - 1; b >= 0; --b) {
        const int mid = (lo + hi) / 2;
        if ((k >> b) & 1) lo = mid; else hi = mid;
    }
    return lo;
}
__host__ __device__ constexpr int ks_hi(int n, int r, int k) {
    int lo = 0, hi = n;
    for (int b = r - 1; b >= 0; --b) {
        const int mid = (lo + hi) / 2;
        if ((k >> b) & 1) lo = mid; else hi = mid;
    }
    return hi;
}

template <int TR, int SS, int NW, int DYSH>
__global__ __launch_bounds__(64 * NW) void wgrad_kslice_bf16_kernel(WgradArgs a) {
    using G = KsliceGeom<NW>;
    constexpr int NT = TR * SS, P = G::P, XU8 = G::XU8, KD = G::kDepth, NB = G::nbuf;
    constexpr int NSLOT = TR;                         // x fragments held in registers
    constexpr int U = NSLOT % 2 == 0 ? NSLOT : 2 * NSLOT;
    constexpr int UL = (U % NB == 0) ? U : (NB % U == 0 ? NB : U * NB);   // every index repeats
    static_assert(UL % 2 == 0 && KD >= 3, "barrier parity, two steps of data ahead");
    static_assert(SS <= 3 && TR <= 3, "a lane's x window is one 16-byte and one 4-byte read");
    static_assert(DYSH == 0 || DYSH == 1, "dy window: at most one element past a 16-byte boundary");
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* const lds = reinterpret_cast<uint16_t*>(smem);

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int qb = c % a.nqb; c /= a.nqb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int p0 = seg * a.rows_per_seg;
    const int nrows = min(a.rows_per_seg, a.Hot - p0);
    const int q0 = qb * G::QW;
    const int ncsb = a.C / 32;
    const int o0 = (blockIdx.z / ncsb) * 32, c0 = (blockIdx.z % ncsb) * 32;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, hi = lane >> 5;

    const uint16_t* xt = static_cast<const uint16_t*>(a.x) + tile * a.x_tile +
                         int64_t(n) * a.C * a.x_rows * a.x_pitch;
    const int dy_rows = a.Hot + 2 * a.dy_off;
    const uint16_t* dyt = static_cast<const uint16_t*>(a.dy) + tile * a.dy_tile +
                          int64_t(n) * a.K * dy_rows * a.dy_pitch;
    const int xg0 = q0 + a.base_c;                 // x column of staged column 0 (a multiple of 8)
    const int dya0 = q0 + a.dy_off - DYSH;         // dy column of staged column 0 (a multiple of 8)
    const int xrow0 = p0 + a.base_r;               // x row of window row 0 in step 0

    // This wave's loads of a step: load k is number wave + k * NW of the
    // step's 2 NI (x region, then dy region); only waves below NX have a load
    // in the last slot.  Lane offsets (bytes inside a sample, below 2^32 by
    // the plan) are fixed; a step adds the row.
    uint32_t loff[G::LPW];
    int ldst[G::LPW];            // LDS element offset of the load's 64 chunks in a buffer
    bool lx[G::LPW];             // the load reads x (else dy)
    const uint32_t jx = uint32_t((int64_t(c0) * a.x_rows * a.x_pitch + xg0) * 2);   // a junk load's x chunk
    constexpr int NX = 2 * G::NI - (G::LPW - 1) * NW;   // waves with LPW loads a step (the rest LPW - 1)
    const bool full = wave < NX;
#pragma unroll
    for (int k = 0; k < G::LPW; ++k) {
        const int id = wave + k * NW;
        const bool isx = id < G::NI || id >= 2 * G::NI;
        const int ii = id < G::NI ? id : id - G::NI;
        const int cc = min(64 * ii + lane, 32 * XU8 - 1);   // chunk (spare chunks repeat the last)
        const int rr = cc / XU8, g8 = cc - rr * XU8;
        if (id >= 2 * G::NI) {
            loff[k] = jx;
            ldst[k] = 2 * G::REG;
        } else if (isx) {
            loff[k] = uint32_t((int64_t(c0 + rr) * a.x_rows * a.x_pitch + min(xg0 + 8 * g8, a.x_pitch - 8)) * 2);
            ldst[k] = 64 * ii * 8;
        } else {
            loff[k] = uint32_t((int64_t(o0 + rr) * dy_rows * a.dy_pitch + min(dya0 + 8 * g8, a.dy_pitch - 8)) * 2);
            ldst[k] = G::REG + 64 * ii * 8;
        }
        lx[k] = isx;
    }
    // The loads are written out: the compiler would otherwise wait for every
    // direct load before any LDS read.  The waits are wait_loads() below.
    const uint32_t lds0 = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char*)smem));
    auto dma = [](const char* base, uint32_t off, uint32_t ldsaddr) {
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                     :: "s"(ldsaddr), "v"(off), "s"(base) : "memory", "m0");
    };
    auto request = [&](int j, int b) {   // step j's rows -> LDS buffer b
        const char* xr = reinterpret_cast<const char*>(
            xt + int64_t(min(max(xrow0 + j + TR - 1, 0), a.x_rows - 1)) * a.x_pitch);
        const char* dr = reinterpret_cast<const char*>(
            dyt + int64_t(min(p0 + j + a.dy_off, dy_rows - 1)) * a.dy_pitch);
#pragma unroll
        for (int k = 0; k < G::LPW; ++k)
            if (k < G::LPW - 1 || full) dma(lx[k] ? xr : dr, loff[k], lds0 + 2 * (b * G::BUF + ldst[k]));
    };
    auto request_x = [&](int m, int b) {   // window row m alone (its x loads; the rest repeat them)
        const char* xr = reinterpret_cast<const char*>(
            xt + int64_t(min(max(xrow0 + m, 0), a.x_rows - 1)) * a.x_pitch);
#pragma unroll
        for (int k = 0; k < G::LPW; ++k)
            if (k < G::LPW - 1 || full)
                dma(xr, lx[k] ? loff[k] : jx, lds0 + 2 * (b * G::BUF + (lx[k] ? ldst[k] : 2 * G::REG)));
    };
    // wait for this wave's loads, all but the newest n steps' (the count of
    // a step depends on the wave; the branch is uniform)
    auto wait_loads = [&](auto nc) {
        constexpr int n = decltype(nc)::value;
        static_assert(n * G::LPW < 64, "vmcnt range");
        if (full)
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n * G::LPW) : "memory");
        else
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(n * (G::LPW - 1)) : "memory");
    };

    // a lane's fragments: x channel c0 + l32 / dy filter o0 + l32, pixels 16 w + 8 hi .. + 7
    const int fo = l32 * P + 16 * wave + 8 * hi;
    uint32_t xf[NSLOT][5];     // 10 x elements: the window of shift s starts s elements in
    uint4 A[2];
    auto read_x = [&](const uint16_t* buf, auto slotc) {
        constexpr int sl = decltype(slotc)::value;
        const uint4 v = *reinterpret_cast<const uint4*>(buf + fo);
        xf[sl][0] = v.x; xf[sl][1] = v.y; xf[sl][2] = v.z; xf[sl][3] = v.w;
        xf[sl][4] = *reinterpret_cast<const uint32_t*>(buf + fo + 8);
    };
    auto read_dy = [&](const uint16_t* buf) {
        const uint4 v = *reinterpret_cast<const uint4*>(buf + G::REG + fo);
        if constexpr (DYSH == 0) return v;
        const uint32_t e = *reinterpret_cast<const uint32_t*>(buf + G::REG + fo + 8);
        return make_uint4(__builtin_amdgcn_alignbyte(v.y, v.x, 2), __builtin_amdgcn_alignbyte(v.z, v.y, 2),
                          __builtin_amdgcn_alignbyte(v.w, v.z, 2), __builtin_amdgcn_alignbyte(e, v.w, 2));
    };

    floatx16 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[t][e] = 0.f;

    // prologue, one round trip: window rows 0 .. TR-2 (buffers nbuf ..,
    // into register slots 0 .. TR-2) and steps 0 .. kDepth-1 requested
    // together; step 0 read into registers (slot TR-1, A[0]); steps 1 and 2
    // in LDS before the loop (as after an odd step)
    static_for<0, TR - 1>([&](auto rc) { request_x(decltype(rc)::value, NB + decltype(rc)::value); });
    static_for<0, KD>([&](auto jc) { request(decltype(jc)::value, decltype(jc)::value); });
    wait_loads(std::integral_constant<int, KD - 1>{});
    __syncthreads();
    static_for<0, TR - 1>([&](auto rc) { read_x(lds + (NB + decltype(rc)::value) * G::BUF, rc); });
    read_x(lds, std::integral_constant<int, TR - 1>{});
    A[0] = read_dy(lds);
    wait_loads(std::integral_constant<int, KD - 3>{});
    __syncthreads();

    // The MFMAs are written out (volatile): the LDS reads and the loads keep
    // their place between them.  A B operand built by VALU (shifts, register
    // copies) gets the two wait states an MFMA source needs after a VALU write.
    auto step = [&](int i, auto Jc) __attribute__((always_inline)) {
        constexpr int J = decltype(Jc)::value;
        constexpr int SN = J % NSLOT;
        const uint16_t* bn = lds + ((J + 1) % NB) * G::BUF;
        request(i + KD, (J + KD) % NB);       // last read in step i-2, a barrier ago
        A[(J + 1) % 2] = read_dy(bn);          // step i+1's dy fragment
        Pack8 Av;
        Av.v = A[J % 2];
        static_for<0, NT>([&](auto tc) {
            constexpr int t = decltype(tc)::value, r = t / SS, s = t % SS, sl = (J + r) % NSLOT;
            Pack8 B;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                B.d[q] = s & 1 ? __builtin_amdgcn_alignbyte(xf[sl][q + s / 2 + 1], xf[sl][q + s / 2], 2)
                               : xf[sl][q + s / 2];
            if constexpr (s == 0)
                asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc[t]) : "v"(Av.b), "v"(B.b));
            else
                asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                             : "+v"(acc[t]) : "v"(Av.b), "v"(B.b));
            // step i+1's x row into the registers of window row 0, now issued
            if constexpr (t == SS - 1) read_x(bn, std::integral_constant<int, SN>{});
        });
        if constexpr (J % 2 == 1) {
            wait_loads(std::integral_constant<int, KD - 3>{});   // steps i+2 and i+3 are in LDS
            __syncthreads();
        }
    };
    int i = 0;
    for (; i + UL <= nrows; i += UL)
        static_for<0, UL>([&](auto Jc) { step(i + decltype(Jc)::value, Jc); });
    static_for<0, UL - 1>([&](auto Jc) {
        if (i + decltype(Jc)::value < nrows) step(i + decltype(Jc)::value, Jc);
    });
    wait_loads(std::integral_constant<int, 0>{});   // no load may land in the LDS reused below
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NT; ++t) asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc[t]));

    // The waves' sums, by recursive halving: unit u = 4 t + q is the float4
    // acc[t][4q .. 4q+3] of a lane.  In the round of distance D a wave and
    // its partner wave ^ D hold the same unit range; the one without bit D
    // keeps the lower half and hands over the upper, the other the reverse.
    // After log2(NW) rounds wave w owns the sums of its own share of the
    // units (in a fixed order of additions) and stores them.
    constexpr int NU = 4 * NT, LOGW = NW == 8 ? 3 : NW == 4 ? 2 : 1;
    static_assert(NW == (1 << LOGW), "power-of-two waves");
    float4* red = reinterpret_cast<float4*>(smem);   // [wave][unit slot][64] float4
    constexpr int SLOT = (NU + 1) / 2;               // units handed over in the first round
    static_for<0, LOGW>([&](auto rc) {
        constexpr int r = decltype(rc)::value, D = NW >> (r + 1);
        const int path = wave >> (LOGW - r);          // the wave's range before this round
        const bool upper = (wave & D) != 0;
        float4* mine = red + wave * SLOT * 64 + lane;
        const float4* theirs = red + (wave ^ D) * SLOT * 64 + lane;
        static_for<0, (1 << r)>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            constexpr int LO = ks_lo(NU, r, k), HI = ks_hi(NU, r, k), MID = (LO + HI) / 2;
            if (path == k) {
                if (upper)
                    static_for<LO, MID>([&](auto uc) {
                        constexpr int u = decltype(uc)::value, q = u % 4;
                        const floatx16& v = acc[u / 4];
                        mine[(u - LO) * 64] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
                    });
                else
                    static_for<MID, HI>([&](auto uc) {
                        constexpr int u = decltype(uc)::value, q = u % 4;
                        const floatx16& v = acc[u / 4];
                        mine[(u - MID) * 64] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
                    });
            }
        });
        __syncthreads();
        static_for<0, (1 << r)>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            constexpr int LO = ks_lo(NU, r, k), HI = ks_hi(NU, r, k), MID = (LO + HI) / 2;
            auto add = [&](auto uc, int pos) {
                constexpr int u = decltype(uc)::value, q = u % 4;
                floatx16& v = acc[u / 4];
                const float4 w = theirs[pos * 64];
                v[4 * q] += w.x; v[4 * q + 1] += w.y; v[4 * q + 2] += w.z; v[4 * q + 3] += w.w;
            };
            if (path == k) {
                if (upper)   // partner handed over [MID, HI) at slots 0 ..
                    static_for<MID, HI>([&](auto uc) { add(uc, decltype(uc)::value - MID); });
                else         // partner handed over [LO, MID)
                    static_for<LO, MID>([&](auto uc) { add(uc, decltype(uc)::value - LO); });
            }
        });
        __syncthreads();
    });
    // partial, [chunk][block][unit][64 lanes][4]: this wave's units.  The
    // partials are stored at device scope (sc1, written through): the reduce
    // launch reads them from another XCD anyway, and the kernel then ends with
    // no dirty lines for the end-of-kernel L2 write-back (about 1 us less per
    // pass on a 64-channel 3x3 layer than plain write-back stores).
    float4* part = reinterpret_cast<float4*>(a.part + int64_t(blockIdx.x) * a.F +
                                             int64_t(blockIdx.z) * NT * 1024) + lane;
    static_for<0, NW>([&](auto kc) {
        constexpr int k = decltype(kc)::value;
        constexpr int LO = ks_lo(NU, LOGW, k), HI = ks_hi(NU, LOGW, k);
        if (wave == k)
            static_for<LO, HI>([&](auto uc) {
                constexpr int u = decltype(uc)::value, q = u % 4;
                const floatx16& v = acc[u / 4];
                const f32x4v val = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
                float4* dst = part + u * 64;
                asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(dst), "v"(val) : "memory");
            });
    });
}

// ---------------------------------------------------------------- bf16

template <int SS, int TRB>
__global__ __launch_bounds__(kThreads) void wgrad_rows_bf16_kernel(WgradArgs a) {
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
    float* part = a.part + int64_t(chunk) * a.F;
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

// RB: the tile's x and dy are under 2^31 bytes: the staging gathers are
// buffer loads (an element past the tile or the filters is an offset past
// the buffer's end, which reads zero) issued kRF per thread before the first
// wait; otherwise one load round trip per element.
static constexpr int kRF = 8;
static constexpr int kRFWord3 = 0x00020000;   // buffer resource word 3 (gfx9 family: raw access)
static constexpr int kRFOOB = 0x7fffffff;     // byte offset past every buffer here: the load returns 0

// n / d and n % d (0 <= n < 2^22, d >= 1) from a float reciprocal of d: the
// product is within one of the quotient, which one correction each way
// makes exact.
__device__ __forceinline__ int rf_divmod(int n, int d, float inv, int& r) {
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

template <int NBW, bool RB>
__global__ __launch_bounds__(kThreads) void wgrad_rows_f32_kernel(WgradArgs a) {
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
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(xt), 0, RB ? int(int64_t(a.Nn) * a.C * xplane * 4) : 0, kRFWord3);
    const __amdgpu_buffer_rsrc_t rdy = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dyt), 0, RB ? int(int64_t(a.Nn) * a.K * dyplane * 4) : 0, kRFWord3);
    const float inv_xw = 1.0f / float(XW), inv_r = 1.0f / float(a.R);

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
            if constexpr (RB) {
                for (int e0 = tid; e0 < 64 * kBQ; e0 += kThreads * kRF) {
                    float v[kRF];
#pragma unroll
                    for (int u = 0; u < kRF; ++u) {
                        const int e = e0 + u * kThreads;
                        const int q = e % kBQ, ol = e / kBQ;
                        const int o = o0 + ol;
                        const bool ok = e < 64 * kBQ && o < a.K && q0 + q < a.Wot;
                        const int off = ok ? 4 * int((int64_t(n) * a.K + o) * dyplane +
                                                     int64_t(p + a.dy_off) * a.dy_pitch + a.dy_off + q0 + q)
                                           : kRFOOB;
                        v[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rdy, off, 0, 0));
                    }
#pragma unroll
                    for (int u = 0; u < kRF; ++u) {
                        const int e = e0 + u * kThreads;
                        if (e < 64 * kBQ) dyl[(e / kBQ) * DYP + e % kBQ] = v[u];
                    }
                }
                const int nx = span * a.R * XW;
                for (int e0 = tid; e0 < nx; e0 += kThreads * kRF) {
                    float v[kRF];
#pragma unroll
                    for (int u = 0; u < kRF; ++u) {
                        const int e = e0 + u * kThreads;
                        int xc, r;
                        const int rest = rf_divmod(e, XW, inv_xw, xc);
                        const int cl = rf_divmod(rest, a.R, inv_r, r);
                        const int gr = p * a.istr + a.base_r + r;
                        const int gc = q0 * a.istr + a.base_c + xc;
                        const bool ok = e < nx && gr < a.x_rows && gc < a.x_cols;
                        const int off = ok ? 4 * int((int64_t(n) * a.C + ci_lo + cl) * xplane +
                                                     int64_t(gr) * a.x_pitch + gc)
                                           : kRFOOB;
                        v[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rx, off, 0, 0));
                    }
#pragma unroll
                    for (int u = 0; u < kRF; ++u)
                        if (e0 + u * kThreads < nx) xl[e0 + u * kThreads] = v[u];
                }
            } else {
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
    float* part = a.part + int64_t(chunk) * a.F;
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


// ---------------------------------------------------------------- fp32, columns in registers

// fp32 stride 1 with few flattened columns (C*R*S <= 256): v_mfma_f32_32x32x2_f32
// with rows = 32 filters, columns = 32 flattened (ci, r, s), a k-step = two
// output pixels.  A workgroup walks down a 64-column strip; each wave owns 16
// pixels of every row (8 k-steps) and keeps all NB column blocks in
// accumulators; A (dy) and B (x) are single 4-byte LDS reads at per-lane
// offsets (rows are staged from aligned 16-byte chunks; the misalignment is
// absorbed in the read offset).  The four waves' sums are added in LDS at
// the end (fixed order) and written as one partial in fragment order.
namespace {
typedef float f32x4w __attribute__((ext_vector_type(4)));
template <int S_> struct F32WgGeom {
    static constexpr int XW = 64 + S_ - 1 + 3;             // staged x columns (+3: alignment shift)
    static constexpr int XV = (XW + 3) / 4;                // 16-byte units per staged x row
    static constexpr int XWP = XV * 4 + 4;                 // x row pitch (floats)
    static constexpr int DV = 17;                          // 16-byte units per staged dy row (64 + 3)
    static constexpr int DYP = DV * 4 + 4;                 // dy row pitch (floats)
};
}  // namespace

// CIN is the channel capacity: channels a.C .. CIN-1 are staged as zeros,
// and only the nb = ceil(a.C R S / 32) column blocks that hold real columns
// are written (blocks past them repeat the last real column; a branch per
// block in the MFMA loop cost the mesh layer 4 us)
template <int CIN, int RR, int SS>
__global__ __launch_bounds__(kThreads, 1) void wgrad_f32w_kernel(WgradArgs a) {
    using G = F32WgGeom<SS>;
    constexpr int CRS = CIN * RR * SS, NB = (CRS + 31) / 32;
    const int crs = a.C * RR * SS, nb = (crs + 31) / 32;
    constexpr int NRX = RR + 1;                             // x ring slots
    constexpr int XSL = CIN * G::XWP;                       // floats per x slot
    constexpr int XUN = CIN * G::XV, DUN = 32 * G::DV;      // 16-byte units per x / dy row
    constexpr int XPT = (XUN + kThreads - 1) / kThreads, DPT = (DUN + kThreads - 1) / kThreads;
    extern __shared__ __align__(16) unsigned char smem[];
    float* xring = reinterpret_cast<float*>(smem);          // [NRX][CIN][XWP]
    float* dyb = xring + NRX * XSL;                         // [2][32][DYP]

    int c = blockIdx.x;
    const int seg = c % a.nseg; c /= a.nseg;
    const int qb = c % a.nqb; c /= a.nqb;
    const int n = c % a.Nn;
    const int tile = c / a.Nn;
    const int p0 = seg * a.rows_per_seg;
    const int nrows = min(a.rows_per_seg, a.Hot - p0);
    const int q0 = qb * kBQ;
    const int o0 = blockIdx.z * 32;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hi = lane >> 5;

    const float* xt = static_cast<const float*>(a.x) + tile * a.x_tile +
                      int64_t(n) * a.C * a.x_rows * a.x_pitch;
    const int dy_rows = a.Hot + 2 * a.dy_off;
    const float* dyt = static_cast<const float*>(a.dy) + tile * a.dy_tile +
                       int64_t(n) * a.K * dy_rows * a.dy_pitch;
    const int64_t xplane = int64_t(a.x_rows) * a.x_pitch;
    const int64_t dyplane = int64_t(dy_rows) * a.dy_pitch;
    const int xg = q0 + a.base_c, xa = xg & ~3, xsh = xg - xa;           // x column of pixel 0
    const int dg = q0 + a.dy_off, da = dg & ~3, dsh = dg - da;           // dy column of pixel 0
    const int dy_end = a.dy_off + a.Wot;
    const int xrow0 = p0 + a.base_r;

    f32x4w xs[XPT], ds[DPT];
    auto load_x = [&](int m) {   // ring row m (x row xrow0 + m) -> registers
        const int gr = min(max(xrow0 + m, 0), a.x_rows - 1);
        static_for<0, XPT>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int u = min(tid + k * kThreads, XUN - 1);
            const int ci = u / G::XV, g = u % G::XV;
            xs[k] = ci < a.C ? *reinterpret_cast<const f32x4w*>(xt + ci * xplane + int64_t(gr) * a.x_pitch +
                                                                min(xa + 4 * g, a.x_pitch - 4))
                             : f32x4w{0.f, 0.f, 0.f, 0.f};
        });
    };
    auto store_x = [&](int m) {   // zero outside the tile: padding columns feed masked pixels
        float* slot = xring + (m % NRX) * XSL;
        static_for<0, XPT>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int u = min(tid + k * kThreads, XUN - 1);
            const int ci = u / G::XV, g = u % G::XV;
            const int col = xa + 4 * g;
            f32x4w v = xs[k];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = col + e < a.x_cols ? v[e] : 0.f;
            *reinterpret_cast<f32x4w*>(slot + ci * G::XWP + 4 * g) = v;
        });
    };
    auto load_dy = [&](int i) {   // output row p0 + i -> registers (clamped)
        const int gr = min(p0 + i + a.dy_off, dy_rows - 1);
        static_for<0, DPT>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int u = min(tid + k * kThreads, DUN - 1);
            const int o = u / G::DV, g = u % G::DV;
            ds[k] = *reinterpret_cast<const f32x4w*>(dyt + min(o0 + o, a.K - 1) * dyplane +
                                                     int64_t(gr) * a.dy_pitch + min(da + 4 * g, a.dy_pitch - 4));
        });
    };
    auto store_dy = [&](int i) {  // only the interior of filters < K: other pixels add zero
        float* slot = dyb + (i & 1) * 32 * G::DYP;
        static_for<0, DPT>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int u = min(tid + k * kThreads, DUN - 1);
            const int o = u / G::DV, g = u % G::DV;
            const int col = da + 4 * g;
            f32x4w v = ds[k];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] = (o0 + o < a.K && col + e >= dg && col + e < dy_end) ? v[e] : 0.f;
            *reinterpret_cast<f32x4w*>(slot + o * G::DYP + 4 * g) = v;
        });
    };

    // per-lane column (ci, r, s) of each block: x offset inside a slot and filter row
    int boff[NB], brow[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int col = min(32 * b + l32, crs - 1);   // columns past crs are never stored
        const int ci = col / (RR * SS), r = (col / SS) % RR, sx = col % SS;
        boff[b] = ci * G::XWP + xsh + sx;
        brow[b] = r;
    }
    floatx16 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[b][e] = 0.f;

    for (int m = 0; m < RR; ++m) {
        load_x(m);
        store_x(m);
    }
    load_dy(0);
    store_dy(0);
    __syncthreads();

    const int pw = 16 * wave + hi;   // this lane's first pixel; k-step k adds 2k
    for (int i = 0; i < nrows; ++i) {
        load_x(i + RR);
        load_dy(i + 1);
        const float* arow = dyb + (i & 1) * 32 * G::DYP + l32 * G::DYP + dsh + pw;
        const float* bsl[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) bsl[b] = xring + ((i + brow[b]) % NRX) * XSL + boff[b] + pw;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float av = arow[2 * k];
            float bv[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) bv[b] = bsl[b][2 * k];
#pragma unroll
            for (int b = 0; b < NB; ++b) acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv[b], acc[b], 0, 0, 0);
        }
        // x slot (i + RR) % NRX and dy buffer (i + 1) & 1 were last read in step i - 1
        store_x(i + RR);
        store_dy(i + 1);
        __syncthreads();
    }

    // the four waves' sums, added in wave order in LDS, one partial per chunk:
    // [chunk][gz][block][16][64] in fragment order
    float* red = xring;   // the ring is free now: 4 x NB x 1024 floats
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) red[((wave * NB + b) * 16 + e) * 64 + lane] = acc[b][e];
    __syncthreads();
    float* part = a.part + int64_t(blockIdx.x) * a.F + int64_t(blockIdx.z) * nb * 1024;
    for (int f = tid; f < nb * 1024; f += kThreads)
        part[f] = ((red[f] + red[NB * 1024 + f]) + red[2 * NB * 1024 + f]) + red[3 * NB * 1024 + f];
}

// ---------------------------------------------------------------- reduction

// dw = (accumulate ? dw : 0) + sum over chunks of the partials, in a fixed
// order: chunk group g (of 4) sums chunks g, g+4, g+8, ... in increasing
// order, then the four group sums are added in order 0..3.  A workgroup
// covers 64 partial positions x 4 chunk groups; loads are coalesced along
// the positions.
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(WgradArgs a) {
    __shared__ float red[4][64];
    const int64_t f = int64_t(blockIdx.x) * 64 + (threadIdx.x & 63);
    const int g = threadIdx.x >> 6;
    float sum = 0.f;
    if (f < a.F) {
        const float* src = a.part + f;
        int c = g;
        for (; c + 28 < a.nchunks; c += 32) {   // eight loads in flight, summed in chunk order
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = src[int64_t(c + 4 * j) * a.F];
#pragma unroll
            for (int j = 0; j < 8; ++j) sum += v[j];
        }
        for (; c < a.nchunks; c += 4) sum += src[int64_t(c) * a.F];
    }
    red[g][threadIdx.x & 63] = sum;
    __syncthreads();
    if (g != 0 || f >= a.F) return;
    const int l = threadIdx.x;
    const float total = ((red[0][l] + red[1][l]) + red[2][l]) + red[3][l];
    int64_t idx;
    if (a.frag == 4) {
        // fp32 flattened columns: [gz][block][16][64], rows = filters, columns = (ci, r, s)
        const int NB = (a.C * a.R * a.S + 31) / 32;
        int64_t t = f;
        const int lane = int(t % 64); t /= 64;
        const int e = int(t % 16); t /= 16;
        const int b = int(t % NB); t /= NB;
        const int bz = int(t);
        const int o = bz * 32 + 8 * (e / 4) + 4 * (lane / 32) + (e % 4);
        const int col = 32 * b + (lane & 31);
        if (o >= a.K || col >= a.C * a.R * a.S) return;
        idx = int64_t(o) * a.C * a.R * a.S + col;
    } else if (a.frag == 3) {
        // phase images: [gy][gz][phase tap][16][64], 32x32 blocks of (filter,
        // phase channel 4 ci + 2 pr + pc); tap (r', s') is filter tap (2r' + pr, 2s' + pc)
        const int SP = (a.S + 1) / 2, NT = a.TRB * SP;
        int64_t t = f;
        const int lane = int(t % 64); t /= 64;
        const int e = int(t % 16); t /= 16;
        const int tap = int(t % NT); t /= NT;
        const int bz = int(t % a.gz);
        const int o = bz * 32 + 8 * (e / 4) + 4 * (lane / 32) + (e % 4);
        const int cp = lane & 31, ci = cp >> 2;
        const int r = 2 * (tap / SP) + ((cp >> 1) & 1), s = 2 * (tap % SP) + (cp & 1);
        if (r >= a.R || s >= a.S || o >= a.K || ci >= a.C) return;
        idx = ((int64_t(o) * a.C + ci) * a.R + r) * a.S + s;
    } else if (a.frag == 5) {
        // [gz][tap][q][64 lanes][4]: value j of float4 q is fragment element e = 4 q + j
        const int NT = a.R * a.S;
        int64_t t = f;
        const int j = int(t % 4); t /= 4;
        const int lane = int(t % 64); t /= 64;
        const int q = int(t % 4); t /= 4;
        const int tap = int(t % NT); t /= NT;
        const int bz = int(t);
        const int ncsb = (a.C + 31) / 32;
        const int o = (bz / ncsb) * 32 + 8 * q + 4 * (lane / 32) + j;
        const int ci = (bz % ncsb) * 32 + (lane & 31);
        const int r = tap / a.S, s = tap % a.S;
        if (o >= a.K || ci >= a.C) return;
        idx = ((int64_t(o) * a.C + ci) * a.R + r) * a.S + s;
    } else if (a.frag == 2) {
        // [gy][gz][tap][16][64] -> (o, ci, r, s), 32x32 blocks
        const int NT = a.TRB * a.S;
        int64_t t = f;
        const int lane = int(t % 64); t /= 64;
        const int e = int(t % 16); t /= 16;
        const int tap = int(t % NT); t /= NT;
        const int bz = int(t % a.gz);
        const int by = int(t / a.gz);
        const int ncsb = (a.C + 31) / 32;
        const int o = (bz / ncsb) * 32 + 8 * (e / 4) + 4 * (lane / 32) + (e % 4);
        const int ci = (bz % ncsb) * 32 + (lane & 31);
        const int r = by * a.TRB + tap / a.S, s = tap % a.S;
        if (r >= a.R || o >= a.K || ci >= a.C) return;
        idx = ((int64_t(o) * a.C + ci) * a.R + r) * a.S + s;
    } else if (a.frag) {
        // [gy][gz][wave][tr][s][16][64] -> (o, ci, r, s)
        const int SS = a.S;
        int64_t t = f;
        const int lane = int(t % 64); t /= 64;
        const int e = int(t % 16); t /= 16;
        const int s = int(t % SS); t /= SS;
        const int tr = int(t % a.TRB); t /= a.TRB;
        const int wave = int(t % 4); t /= 4;
        const int bz = int(t % a.gz);
        const int by = int(t / a.gz);
        const int ncsb = (a.C + 63) / 64;
        const int o = (bz / ncsb) * 64 + (wave & 1) * 32 + 8 * (e / 4) + 4 * (lane / 32) + (e % 4);
        const int ci = (bz % ncsb) * 64 + (wave >> 1) * 32 + (lane & 31);
        const int r = by * a.TRB + tr;
        if (tr >= a.TRB || r >= a.R || o >= a.K || ci >= a.C) return;
        idx = ((int64_t(o) * a.C + ci) * a.R + r) * a.S + s;
    } else {
        idx = f;
    }
    a.dw[idx] = a.accumulate ? a.dw[idx] + total : total;
}

template <typename K>
static hipError_t set_lds(K kernel, int bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

// one filter tap per workgroup: four waves, each with its whole 32x32 block;
// more taps: eight waves, two per sub-block
template <int SS, int TRB>
static hipError_t launch_strip(const WgradArgs& a, dim3 grid, hipStream_t s) {
    if constexpr (SS * TRB == 1) {
        hipError_t e = set_lds(wgrad_strip_bf16_kernel<SS, TRB>, a.lds_bytes);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((wgrad_strip_bf16_kernel<SS, TRB>), grid, dim3(kThreads), a.lds_bytes, s, a);
    } else {
        hipError_t e = set_lds(wgrad_pair_bf16_kernel<SS, TRB>, a.lds_bytes);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((wgrad_pair_bf16_kernel<SS, TRB>), grid, dim3(512), a.lds_bytes, s, a);
    }
    return hipGetLastError();
}

template <int C_, int R_, int S_>
static hipError_t launch_f32wg(const WgradArgs& a, dim3 grid, hipStream_t s) {
    hipError_t e = set_lds(wgrad_f32w_kernel<C_, R_, S_>, a.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wgrad_f32w_kernel<C_, R_, S_>), grid, dim3(kThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

template <int TR, int SS, int DYSH>
static hipError_t launch_kslice(const WgradArgs& a, dim3 grid, hipStream_t s) {
    auto k = wgrad_kslice_bf16_kernel<TR, SS, kKsliceNW, DYSH>;
    hipError_t e = set_lds(k, a.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k, grid, dim3(64 * kKsliceNW), a.lds_bytes, s, a);
    return hipGetLastError();
}

template <int SS>
static hipError_t launch_taps2(const WgradArgs& a, dim3 grid, hipStream_t s) {
    hipError_t e = set_lds(wgrad_taps2_bf16_kernel<SS, SS>, a.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wgrad_taps2_bf16_kernel<SS, SS>), grid, dim3(kThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

template <int SS>
static hipError_t launch_taps(const WgradArgs& a, dim3 grid, hipStream_t s) {
    hipError_t e = set_lds(wgrad_taps_bf16_kernel<SS, SS>, a.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wgrad_taps_bf16_kernel<SS, SS>), grid, dim3(kThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

template <int SS>
static hipError_t launch_rows_bf16(const WgradArgs& a, dim3 grid, hipStream_t s) {
    constexpr int TRB = SS == 1 ? 9 : (9 / SS > 0 ? 9 / SS : 1);
    hipError_t e = set_lds(wgrad_rows_bf16_kernel<SS, TRB>, a.lds_bytes);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((wgrad_rows_bf16_kernel<SS, TRB>), grid, dim3(kThreads), a.lds_bytes, s, a);
    return hipGetLastError();
}

hipError_t launch_wgrad(const WgradArgs& a, int dtype, hipStream_t s) {
    dim3 grid(a.nchunks, a.gy, a.gz);
    hipError_t e = hipErrorInvalidValue;
    if (a.kind == WGRAD_STRIP_BF16) {
        // one instantiation per (filter width, filter rows per workgroup)
#define DC_STRIP(ss, trb) \
        if (a.S == ss && a.TRB == trb) e = launch_strip<ss, trb>(a, grid, s); else
        DC_STRIP(1, 1) DC_STRIP(1, 2) DC_STRIP(1, 3) DC_STRIP(1, 4) DC_STRIP(1, 5) DC_STRIP(1, 6)
        DC_STRIP(1, 7) DC_STRIP(1, 8) DC_STRIP(1, 9) DC_STRIP(2, 1) DC_STRIP(2, 2) DC_STRIP(2, 3)
        DC_STRIP(2, 4) DC_STRIP(3, 1) DC_STRIP(3, 2) DC_STRIP(3, 3) DC_STRIP(4, 1) DC_STRIP(4, 2)
        DC_STRIP(5, 1) DC_STRIP(6, 1) DC_STRIP(7, 1)
        return hipErrorInvalidValue;
#undef DC_STRIP
    } else if (a.kind == WGRAD_F32W) {
        const int cc = f32w_class(a.C);
#define DC_F32WG(c, r, s_) \
        if (cc == c && a.R == r && a.S == s_) e = launch_f32wg<c, r, s_>(a, grid, s); else
        DC_F32WG(4, 3, 3) DC_F32WG(8, 3, 3) DC_F32WG(12, 3, 3) DC_F32WG(16, 3, 3) DC_F32WG(18, 3, 3)
        DC_F32WG(20, 3, 3) DC_F32WG(24, 3, 3) DC_F32WG(28, 3, 3) DC_F32WG(32, 3, 3)
        DC_F32WG(4, 1, 1) DC_F32WG(8, 1, 1) DC_F32WG(12, 1, 1) DC_F32WG(16, 1, 1) DC_F32WG(18, 1, 1)
        DC_F32WG(20, 1, 1) DC_F32WG(24, 1, 1) DC_F32WG(28, 1, 1) DC_F32WG(32, 1, 1)
        return hipErrorInvalidValue;
#undef DC_F32WG
    } else if (a.kind == WGRAD_KSLICE_BF16) {
        // the dy columns of a strip start dy_off & 7 elements past a 16-byte boundary
        if (a.R == 3 && a.S == 3 && (a.dy_off & 7) == 0) e = launch_kslice<3, 3, 0>(a, grid, s);
        else if (a.R == 3 && a.S == 3 && (a.dy_off & 7) == 1) e = launch_kslice<3, 3, 1>(a, grid, s);
        else return hipErrorInvalidValue;
    } else if (a.kind == WGRAD_TAPS2_BF16) {
        switch ((a.S + 1) / 2) {
            case 2: e = launch_taps2<2>(a, grid, s); break;
            case 3: e = launch_taps2<3>(a, grid, s); break;
            case 4: e = launch_taps2<4>(a, grid, s); break;
            default: return hipErrorInvalidValue;
        }
    } else if (a.kind == WGRAD_TAPS_BF16) {
        switch (a.S) {
            case 2: e = launch_taps<2>(a, grid, s); break;
            case 3: e = launch_taps<3>(a, grid, s); break;
            case 4: e = launch_taps<4>(a, grid, s); break;
            case 5: e = launch_taps<5>(a, grid, s); break;
            case 6: e = launch_taps<6>(a, grid, s); break;
            case 7: e = launch_taps<7>(a, grid, s); break;
            default: return hipErrorInvalidValue;
        }
    } else if (a.kind == WGRAD_ROWS_BF16) {
        switch (a.S) {
            case 1: e = launch_rows_bf16<1>(a, grid, s); break;
            case 2: e = launch_rows_bf16<2>(a, grid, s); break;
            case 3: e = launch_rows_bf16<3>(a, grid, s); break;
            case 4: e = launch_rows_bf16<4>(a, grid, s); break;
            case 5: e = launch_rows_bf16<5>(a, grid, s); break;
            case 6: e = launch_rows_bf16<6>(a, grid, s); break;
            case 7: e = launch_rows_bf16<7>(a, grid, s); break;
            default: return hipErrorInvalidValue;
        }
    } else {
        // buffer loads when the tile's x and dy are under 2^31 bytes
        const int64_t xb = int64_t(a.Nn) * a.C * a.x_rows * a.x_pitch * 4;
        const int64_t dyb = int64_t(a.Nn) * a.K * (a.Hot + 2 * a.dy_off) * a.dy_pitch * 4;
        if (xb < kRFOOB && dyb < kRFOOB) {
            e = set_lds(wgrad_rows_f32_kernel<2, true>, a.lds_bytes);
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL((wgrad_rows_f32_kernel<2, true>), grid, dim3(kThreads), a.lds_bytes, s, a);
        } else {
            e = set_lds(wgrad_rows_f32_kernel<2, false>, a.lds_bytes);
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL((wgrad_rows_f32_kernel<2, false>), grid, dim3(kThreads), a.lds_bytes, s, a);
        }
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(unsigned((a.F + 63) / 64)), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------- fixed workspace

// Chunk partials of dc_conv_bwd_filter_noalloc: a file-scope device array
// instead of a caller's buffer, for callers that cannot allocate.  Each GPU
// holds its own copy until the process ends.  Host code must never pass the
// array's name to a kernel (on the host it is only a stand-in for the symbol):
// the device address comes from hipGetSymbolAddress, once per device, with
// that device current.  The kernels write every partial they later read, so
// nothing in it has to start at zero.
static constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

size_t wgrad_scratch_capacity() { return kScratchBytes; }

hipError_t wgrad_scratch_ptr(void** ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

}  // namespace dc
