/*
 * dc.h -- one GPU's share of a spatially decomposed 2-D convolution layer on
 * AMD MI355X (gfx950): forward, backward-data and backward-filter on an NCHW
 * sub-domain tile, and the halo pack/unpack that borders the tile.
 *
 * Method: Dryden et al., "Improving Strong-Scaling of CNN Training by
 * Exploiting Finer-Grained Parallelism" (IPDPS 2019, arXiv 1903.06681).
 *   - the layer and its six tensors: Sec. II-A; Eqs. (1) forward, (2) weight
 *     gradient, (3) input gradient;
 *   - blocked spatial (+ sample) distribution, the halo set and the local
 *     passes on a tile: Sec. III-A;
 *   - halo message terms (north/south, east/west, four corners): Sec. V-A.
 *
 * Notation map (paper -> this interface): N -> N (this GPU's samples),
 * C -> C, F (filters) -> K, filter K x K -> R x S, stride S -> stride,
 * padding P -> pad, O = floor(K/2) (halo width) -> halo.  The paper's blocked
 * distributions of H and W are the P x Q grid below; C and F are replicated.
 *
 * Everything is C ABI, never throws, allocates and frees nothing, keeps no
 * state and is reentrant.  All device pointers are caller-owned.  Work is
 * enqueued on `stream` (a hipStream_t; NULL = the null stream) and the calls
 * return without synchronising.
 */
#ifndef DC_H
#define DC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DC_OK              =  0,
    DC_ERR_NULL        = -1,  /* a required pointer is NULL */
    DC_ERR_SHAPE       = -2,  /* a size is non-positive, or sizes are inconsistent */
    DC_ERR_DTYPE       = -3,  /* dtype is not DC_F32 / DC_BF16 */
    DC_ERR_HALO        = -4,  /* halo narrower than the pass needs, or wider than a tile */
    DC_ERR_UNSUPPORTED = -5,  /* uneven tiles, or a decomposed output grid not aligned with the input grid */
    DC_ERR_WORKSPACE   = -6,  /* workspace NULL or smaller than dc_bwd_filter_workspace_bytes() */
    DC_ERR_ALIGN       = -7,  /* a device pointer is not 16-byte aligned */
    DC_ERR_HIP         = -8,  /* the HIP runtime reported an error at launch */
    DC_ERR_TILE        = -9,  /* tile index out of range */
    DC_ERR_ARG         = -10, /* other invalid argument (which, accumulate) */
    DC_ERR_TOO_LARGE   = -11  /* a tensor exceeds the 32-bit element indexing of the kernels */
} dc_status;

typedef enum { DC_F32 = 0, DC_BF16 = 1 } dc_dtype;   /* dtype of x, w and dy; y, dx, dw are fp32 */
typedef enum { DC_X = 0, DC_DY = 1 } dc_which;       /* which tensor a tile/halo call refers to */

#define DC_ALL_TILES (-1)   /* every tile of the grid in one launch (single-device emulation) */

/*
 * The layer and its decomposition (Sec. II-A, Sec. III-A).
 *
 * H, W are the GLOBAL input extents.  The grid splits them into P x Q
 * blocked tiles of Ht = H/P by Wt = W/Q input pixels (the paper's blocked
 * distributions of H and W).  The global output is Ho x Wo with
 * Ho = (H + 2*pad - R)/stride + 1; a tile owns Hot = Ho/P by Wot = Wo/Q of it.
 * With P = Q = 1 any geometry with Ho, Wo >= 1 is accepted; with more than one
 * tile the output grid must line up with the input grid, Ho * stride = H and
 * Wo * stride = W (stride 1: "same" output), and Ho % P = Wo % Q = 0, so that
 * a tile owns exactly the outputs whose taps start in its input block.  At
 * stride > 1 a tile may need no halo on one side (e.g. 3x3 stride 2 pad 1: x
 * 1 below, 0 above): the layout keeps the margin h on every side, and the
 * halo calls move only the band each side needs (dc_halo_bands).
 *
 * halo is the margin width h kept on every side of every tile (for both the x
 * and the dy tile).  It must be at least what each pass reads beyond the tile
 * (see dc_required_halo) and, with more than one tile along an axis, at most
 * the input and the output tile extent along it (halos come from the
 * adjacent tile only).
 */
typedef struct {
    int32_t N, C, K;       /* samples on this GPU, input channels, filters */
    int32_t H, W;          /* global input height, width */
    int32_t R, S;          /* filter height, width */
    int32_t stride, pad;   /* same in both spatial dimensions */
    int32_t P, Q;          /* spatial grid: P tiles along H, Q along W */
    int32_t halo;          /* margin width h on every side of a tile */
    int32_t dtype;         /* dc_dtype */
} dc_problem;

/*
 * Tile layouts (all dense, row-major, element type = dtype unless stated):
 *   x_pad  [N][C][Ht+2h][pitch_x]     interior (owned block) at row h, col h
 *   dy_pad [N][K][Hot+2h][pitch_dy]   interior at row h, col h
 *   w      [K][C][R][S]               replicated on every tile (Sec. III-A)
 *   y      [N][K][Hot][Wot]   fp32
 *   dx     [N][C][Ht][Wt]     fp32
 *   dw     [K][C][R][S]       fp32
 * pitch = dc_tile_pitch(): at least width+2h, rounded up to 16 bytes.  Pitch
 * columns beyond width+2h are never written; kernels may read them (as part
 * of an aligned 16-byte access), and their values never reach a result.
 *
 * Tiles are numbered tile = ti*Q + tj, ti = 0..P-1 top to bottom, tj = 0..Q-1
 * left to right.  With tile = DC_ALL_TILES every per-tile buffer argument
 * (tile, send/recv, y, dx) is an array of P*Q consecutive per-tile buffers in
 * tile order, and one launch serves the whole grid.
 *
 * Halo bands (Sec. III-A).  A tile's margin ring is supplied by its eight
 * neighbours; the band from each side is as wide as the passes read on that
 * side (dc_halo_bands: rows above bN, below bS, columns left bW, right bE;
 * all equal to h for the usual stride-1 "same" layers).  Margin cells outside
 * the bands, and bands whose neighbour does not exist, hold zeros after
 * unpack: the convolution's zero padding.
 *
 * Packed halo buffers (send/recv) hold eight regions, in the order
 * N, S, W, E, NW, NE, SW, SE, each laid out [N][channels][rows][cols].
 * Region d of a RECV buffer holds the band of margin d: N bN x Wt, S bS x Wt,
 * W Ht x bW, E Ht x bE, NW bN x bW, NE bN x bE, SW bS x bW, SE bS x bE
 * (output-tile extents Hot, Wot for dy).  Region d of a SEND buffer holds the
 * band of the owned block that the neighbour in direction d receives, i.e.
 * the shape of that neighbour's margin opposite to d (S for d = N, ...).
 * Regions follow each other without gaps; the two layouts have the same
 * total.  dc_halo_elems() is that total rounded up to a multiple of 16 bytes
 * (the padding at the end is never written), so the consecutive buffers of an
 * all-tiles call each start 16-byte aligned.
 */

/* band classes of the margin ring, for dc_halo_pack_bands / dc_halo_unpack_bands */
#define DC_BAND_NS      1   /* rows above and below the owned block (regions N, S) */
#define DC_BAND_WE      2   /* columns left and right of it (regions W, E) */
#define DC_BAND_CORNERS 4   /* the four corner blocks (regions NW, NE, SW, SE) */
#define DC_BAND_ALL     7

/* ---- the five operations ---- */

/*
 * Forward propagation on one tile, Eq. (1) (Sec. II-A) restricted to the
 * tile's samples and output pixels (Sec. III-A):
 *   y[n,k,p,q] = sum_{c,r,s} x[n,c, p*stride-pad+r, q*stride-pad+s] * w[k,c,r,s]
 * reading x from x_pad, halo included.  Cross-correlation, no bias, fp32
 * accumulation.  Writes all of y; reads only what the sum touches.
 */
dc_status dc_conv_fwd(const dc_problem* prob, int32_t tile, const void* x_pad,
                      const void* w, float* y, void* stream);

/*
 * Input gradient on one tile, Eq. (3) (Sec. II-A; Sec. III-A):
 *   dx[n,c,i,j] = sum_{k,r,s} dy[n,k,(i+pad-r)/stride,(j+pad-s)/stride] * w[k,c,r,s]
 * (terms exist where both divisions are exact), reading dy from dy_pad, halo
 * included.  Writes all of dx.
 */
dc_status dc_conv_bwd_data(const dc_problem* prob, int32_t tile, const void* dy_pad,
                           const void* w, float* dx, void* stream);

/*
 * Local weight gradient of one tile, Eq. (2) restricted to the tile's samples
 * and output pixels (Sec. III-A):
 *   dw[k,c,r,s] (=|+=) sum_{n,p,q in tile} dy[n,k,p,q] * x[n,c,p*stride-pad+r,q*stride-pad+s]
 * reading x from x_pad (halo included) and only the interior of dy_pad: the
 * dy halo is not needed (Sec. III-A), so this pass may overlap the dy halo
 * exchange.  accumulate = 0 overwrites dw, 1 adds the partial to dw.
 * With tile = DC_ALL_TILES, dw receives the sum over all tiles in row-major
 * tile order: the single-device stand-in for the allreduce that completes dw.
 * workspace: device scratch of at least dc_bwd_filter_workspace_bytes(prob,
 * tile) bytes, contents undefined on entry and exit.  Results are
 * deterministic: a fixed summation order, no atomics.
 */
dc_status dc_conv_bwd_filter(const dc_problem* prob, int32_t tile, const void* x_pad,
                             const void* dy_pad, float* dw, int32_t accumulate,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * Allocation-free weight gradient, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Same operation, arguments, kernels and results as
 * dc_conv_bwd_filter, without a workspace argument: the chunk partials live
 * in a fixed device array of DC_BWD_FILTER_NOALLOC_MAX_BYTES that the library
 * holds on every GPU it runs on until the process ends (its address is looked
 * up on the first call on a device).  Returns DC_ERR_WORKSPACE, launching
 * nothing, when dc_bwd_filter_workspace_bytes(prob, tile) exceeds that size.
 * Calls no hipMalloc, hipFree or allocating routine.  Every call on one GPU
 * shares that GPU's array: calls that overlap on one GPU (two streams, two
 * host threads) race and must be serialised by the caller.
 */
#define DC_BWD_FILTER_NOALLOC_MAX_BYTES ((size_t)64 << 20)
dc_status dc_conv_bwd_filter_noalloc(const dc_problem* prob, int32_t tile, const void* x_pad,
                                     const void* dy_pad, float* dw, int32_t accumulate,
                                     void* stream);

/*
 * Halo pack (Sec. III-A; message terms of Sec. V-A): copy the bands of the
 * owned block of t_pad (which = DC_X: an x tile; DC_DY: a dy tile) that each
 * existing neighbour needs into the send buffer.  Reads only the owned block
 * (and pitch columns, see above); writes only regions whose neighbour
 * exists.  Bitwise copy.  When dc_halo_elems is 0 (every band empty: a
 * margin no pass reads, e.g. a 1x1 filter) send may be NULL and nothing is
 * launched; for dc_halo_unpack recv may then be NULL, and the call only
 * zero-fills the margin ring.
 */
dc_status dc_halo_pack(const dc_problem* prob, int32_t tile, int32_t which,
                       const void* t_pad, void* send, void* stream);

/*
 * Halo unpack (Sec. III-A): write the whole h-wide margin ring of t_pad.  The
 * band of margin d receives region d of recv when the neighbour in direction
 * d exists; every other margin cell becomes zero (the convolution's zero
 * padding, Sec. II-A, and margin beyond the band widths).  Writes only
 * margins, never the owned block.  With tile = DC_ALL_TILES, recv is the
 * array of all tiles' SEND buffers and each margin is read directly from the
 * neighbour's opposite region: that read is the emulated exchange.
 */
dc_status dc_halo_unpack(const dc_problem* prob, int32_t tile, int32_t which,
                         const void* recv, void* t_pad, void* stream);

/*
 * dc_halo_pack / dc_halo_unpack restricted to some band classes (bands: an OR
 * of DC_BAND_*; DC_BAND_ALL is the full call): pack writes only the regions of
 * those classes, unpack writes only the margin cells of those classes.  Lets
 * a caller move the contiguous N/S rows and the strided W/E columns at
 * different times (or time them apart).  DC_ERR_ARG for an empty or unknown
 * mask.
 */
dc_status dc_halo_pack_bands(const dc_problem* prob, int32_t tile, int32_t which, int32_t bands,
                             const void* t_pad, void* send, void* stream);
dc_status dc_halo_unpack_bands(const dc_problem* prob, int32_t tile, int32_t which, int32_t bands,
                               const void* recv, void* t_pad, void* stream);

/*
 * Interior / boundary split of the forward and input-gradient passes, so that
 * the halo exchange can overlap computation (Sec. IV-A; stride 1 only, else
 * DC_ERR_UNSUPPORTED).  The boundary of the output tile is the frame of
 * outputs whose sum reads a margin: for dc_conv_fwd_region the rows above /
 * below and columns left / right of widths dc_halo_bands(DC_X); for
 * dc_conv_bwd_data_region those of dc_halo_bands(DC_DY).
 *   DC_REGION_ALL:      the plain call.
 *   DC_REGION_INTERIOR: every output outside the frame is final; the frame is
 *                       left unspecified.  It may run while the margins are
 *                       being written (e.g. by dc_halo_unpack on another
 *                       stream): margin values reach frame outputs only.
 *   DC_REGION_BOUNDARY: computes the frame only (the margins must be in
 *                       place); every other output is left untouched.
 * INTERIOR followed by BOUNDARY gives the plain call's result.
 */
typedef enum { DC_REGION_ALL = 0, DC_REGION_INTERIOR = 1, DC_REGION_BOUNDARY = 2 } dc_region;
dc_status dc_conv_fwd_region(const dc_problem* prob, int32_t tile, int32_t region, const void* x_pad,
                             const void* w, float* y, void* stream);
dc_status dc_conv_bwd_data_region(const dc_problem* prob, int32_t tile, int32_t region,
                                  const void* dy_pad, const void* w, float* dx, void* stream);

/* ---- host-only helpers (no GPU needed) ---- */

/* Check a problem and tile index (DC_ALL_TILES allowed); no launch. */
dc_status dc_validate(const dc_problem* prob, int32_t tile);

/* Row pitch (elements) of the padded x or dy tile; -1 on an invalid problem. */
int64_t dc_tile_pitch(const dc_problem* prob, int32_t which);

/* Elements of one padded x or dy tile ([N][ch][rows+2h][pitch]); -1 if invalid. */
int64_t dc_tile_elems(const dc_problem* prob, int32_t which);

/* Elements of one tile's packed halo buffer for x or dy (16-byte multiple); -1 if invalid. */
int64_t dc_halo_elems(const dc_problem* prob, int32_t which);

/* Workspace bytes dc_conv_bwd_filter needs for this tile argument (0 if none). */
size_t dc_bwd_filter_workspace_bytes(const dc_problem* prob, int32_t tile);

/*
 * Margins each pass reads beyond a tile, independent of the halo field:
 * which = DC_X: rows/cols of x the forward pass (and weight gradient) reads
 * before (lohi[0]) and after (lohi[1]) the tile; which = DC_DY: the same for
 * the dy rows the input gradient reads.  Same in both spatial dimensions.
 */
dc_status dc_required_halo(const dc_problem* prob, int32_t which, int32_t lohi[2]);

/*
 * Band widths the halo calls move for x (which = DC_X) or dy (DC_DY):
 * bw = {rows above, rows below, columns left, columns right} of a tile, the
 * margins the passes read (x: forward and weight gradient, Eq. (1)/(2);
 * dy: input gradient, Eq. (3)).  Each is at most the problem's halo.
 */
dc_status dc_halo_bands(const dc_problem* prob, int32_t which, int32_t bw[4]);

/* Tile extents: dims = {Ht, Wt, Hot, Wot}. */
dc_status dc_tile_dims(const dc_problem* prob, int32_t dims[4]);

/* Static string for a status code. */
const char* dc_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* DC_H */
