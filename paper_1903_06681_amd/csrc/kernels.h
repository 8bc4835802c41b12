// Launch interfaces of the HIP kernels behind the dc_* entry points.
// Host code builds these argument blocks from a validated Geo; every kernel
// trusts them (bounds were checked on the host).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "dc.h"

namespace dc {

// ---------------------------------------------------------------- halo

// Packed halo format: eight regions, order N, S, W, E, NW, NE, SW, SE, each
// [planes][rows][cols].  Region d of a receive buffer has the shape of margin
// d's band (rows bw[0] above / bw[1] below or ht; cols bw[2] left / bw[3]
// right or wt); region d of a send buffer the shape of the band the neighbour
// in direction d receives (its margin opposite(d)).  Offsets roff / soff are
// prefix sums of those sizes.
struct HaloArgs {
    const void* src;     // pack: padded tiles; unpack: packed buffers
    void* dst;           // pack: packed buffers; unpack: padded tiles
    int64_t tile_elems;  // elements per padded tile
    int64_t halo_elems;  // elements per packed buffer
    int64_t src_elems;   // elements readable from src (unpack: bounds of the vector reads)
    int64_t roff[8];     // receive buffer region offsets
    int64_t soff[8];     // send buffer region offsets
    int planes;          // N * channels
    int rows, pitch;     // padded tile rows and row pitch
    int ht, wt, h;       // tile extent and margin width
    int bw[4];           // band widths: rows above, rows below, cols left, cols right
    int P, Q;
    int tile0;           // first tile handled by this launch
    int ntiles;          // tiles handled by this launch
    int all_tiles;       // unpack: read neighbours' send buffers directly
    int bands;           // DC_BAND_* classes moved by this launch
    int vec;             // N/S rows may move as aligned 16-byte vectors
    int ppw;             // planes per workgroup
};

hipError_t launch_halo_pack(const HaloArgs& a, int esize, hipStream_t s);
hipError_t launch_halo_unpack(const HaloArgs& a, int esize, hipStream_t s);

// ------------------------------------------- implicit-GEMM conv (fwd / bwd-data)
//
// out[n, o, u*ostr + oph_r, v*ostr + oph_c] =
//     sum_{ci, tr, ts} in[n, ci, u*istr + tr + base_r, v*istr + ts + base_c]
//                      * w[o*w_os + ci*w_cs + (wr0 + wrstep*tr)*S + (ws0 + wsstep*ts)]
// for u < Uo, v < Vo.  Forward: in = x tile, o = filter.  Backward-data at
// stride 1 (or one stride phase): in = dy tile, o = input channel, taps
// reversed.  Input coordinates are padded-tile coordinates.

struct IgemmArgs {
    const void* in;
    const void* w;
    float* out;
    int64_t in_tile, out_tile;   // elements between consecutive tiles (all-tiles mode)
    int ntiles, Nn;
    int Cin, Cout;
    int in_rows, in_cols, in_pitch;
    int Uo, Vo;
    int out_rows, out_cols;
    int ostr, oph_r, oph_c;
    int istr;
    int Tr, Ts;
    int base_r, base_c;
    int wr0, wrstep, ws0, wsstep;
    int R, S;                    // filter height, width of w
    int64_t w_os, w_cs;          // weight strides of o and ci
    int wK, wC;                  // w is [wK][wC][R][S]
    int wmode;                   // 0: o indexes wK, ci indexes wC (forward); 1: swapped (backward-data)
    int wvec;                    // weight rows allow 16-byte chunk copies (set by the plan)
    int CC;                      // channels per LDS chunk (multiple of 8 for bf16, 2 for fp32)
    int OB;                      // output channels per workgroup (32 or 64)
    int lds_bytes;
    int kind;                    // 0: chunked kernel; 1, 2: register-weight strip kernel (bf16, fp32);
                                 // 3: register-weight rolling-row kernel (bf16); 4: frame kernel (bf16, fp32)
    int phase;                   // register-weight bf16 forward over the stride-2 phase images
    // merged-phase backward-data (stride 2, C <= 8): all four output phases
    // as one stride-1 correlation over dy; rows o' = 4 c + 2 py + px of the
    // weight image, window origin (base_r, base_c).  bp: requested by the
    // caller; bpC: C; bpvoff: pixels the strips start early (16-byte aligned
    // staging); per row phase py: window-row offset bpdr, taps bptr, first
    // filter row bpr0 (then -2 per window row); per column phase likewise
    int bp, bpC, bpvoff;
    int bpdr[2], bptr[2], bpr0[2], bpdc[2], bpts[2], bps0[2];
    int nvb, nseg, rows_per_seg; // strip kernels: 64- (128-, rolling) column strips, row segments
    // frame mode (chunked and frame kernels): the launch covers only the
    // output rectangles [fu0, fu0 + fnu) x [fv0, fv0 + fnv) of fseg segments,
    // whose workgroups are numbered from fblk[seg] (prefix sums, fblk[fseg]
    // total; the plan sets them for the kernel it picks)
    int frame, fseg;
    int fu0[4], fv0[4], fnu[4], fnv[4], fcm[4], fblk[5];
};

// Largest dynamic LDS allocation per workgroup on the current device (bytes).
int device_lds_limit();
// Compute units of the current device.
int device_cu_count();

// Frame mode: the output rows above / below and columns left / right of the
// interior, of widths bands[0..3] (clamped to the Uo x Vo output), as the
// segments of one launch of the chunked kernel.
void igemm_set_frame(IgemmArgs& a, const int bands[4]);

// Chooses the channel chunk and LDS size; returns false if no variant fits.
bool igemm_plan(IgemmArgs& a, int dtype);
hipError_t launch_igemm(const IgemmArgs& a, int dtype, hipStream_t s);
bool igemm_wreg_plan(IgemmArgs& a);
hipError_t launch_igemm_wreg(const IgemmArgs& a, hipStream_t s);
bool igemm_roll_plan(IgemmArgs& a);
hipError_t launch_igemm_roll(const IgemmArgs& a, hipStream_t s);
bool igemm_f32w_plan(IgemmArgs& a);
hipError_t launch_igemm_f32w(const IgemmArgs& a, hipStream_t s);
bool igemm_frame_plan(IgemmArgs& a, int dtype);
hipError_t launch_igemm_frame(const IgemmArgs& a, int dtype, hipStream_t s);

// ----------------------------------------------------- weight gradient
//
// Each workgroup reduces one chunk of a tile's output pixels into a partial
// weight gradient in the workspace; a second kernel adds the partials in
// chunk order:  dw = (accumulate ? dw : 0) + sum_chunk part[chunk].
//   part = dy[n, o, p, q] * x[n, ci, p*istr + r + base_r, q*istr + s + base_c]
// summed over the chunk's (n, p, q).

enum WgradKind { WGRAD_STRIP_BF16 = 0, WGRAD_ROWS_BF16 = 1, WGRAD_ROWS_F32 = 2, WGRAD_TAPS_BF16 = 3,
                 WGRAD_TAPS2_BF16 = 4, WGRAD_F32W = 5, WGRAD_KSLICE_BF16 = 6 };

struct WgradArgs {
    const void* x;               // padded x tiles
    const void* dy;              // padded dy tiles (interior read only)
    float* part;                 // workspace partials [nchunks][F]
    float* dw;
    int64_t x_tile, dy_tile;
    int ntiles, Nn;
    int C, K, R, S;
    int x_rows, x_cols, x_pitch;
    int dy_pitch, dy_off;        // dy interior origin (= h) in the padded tile
    int Hot, Wot;
    int istr;
    int base_r, base_c;
    int accumulate;
    // plan
    int kind;                    // WgradKind
    int gy, gz;                  // grid: filter-row groups (or column groups), channel superblocks
    int TRB;                     // filter rows per workgroup
    int nchunks;
    int chunks_per_tile, rows_per_chunk;   // row kinds: flattened (n, p) rows per chunk
    int nqb, nseg, rows_per_seg;           // strip kinds: column strips, row segments
    int64_t F;                   // floats per chunk partial
    int frag;                    // 0: partials in dw order; 1 .. 5: in MFMA fragment order (64x64
                                 // blocks, 32x32 blocks, 32x32 blocks of stride-2 phase images,
                                 // fp32 32 filters x 32 flattened (ci, r, s), 32x32 blocks as
                                 // float4 per lane)
    int lds_bytes;
};

size_t wgrad_workspace_bytes(int dtype, int ntiles, int N, int C, int K, int R, int S,
                             int stride, int Hot, int Wot, int base_c, int dy_off);
bool wgrad_plan(WgradArgs& a, int dtype);
hipError_t launch_wgrad(const WgradArgs& a, int dtype, hipStream_t s);

// Fixed device workspace of the allocation-free weight-gradient entry point:
// its capacity in bytes, and its address on the current device (looked up
// once per device, on the first call there).
size_t wgrad_scratch_capacity();
hipError_t wgrad_scratch_ptr(void** ptr);

}  // namespace dc
