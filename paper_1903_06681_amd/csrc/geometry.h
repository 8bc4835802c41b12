// Host-side tile geometry and validation for the dc_* interface.
//
// Blocked spatial distribution of Sec. III-A: a P x Q grid of Ht x Wt input
// tiles (Hot x Wot output tiles), each padded by a margin of h on every side
// that holds the halo set (neighbours' bands, zeros outside the domain).
#pragma once

#include <cstdint>

#include "dc.h"

namespace dc {

struct Geo {
    int N, C, K, H, W, R, S, stride, pad, P, Q, h, dtype, esize;
    int Ht, Wt;          // input tile extent
    int Ho, Wo;          // global output extent
    int Hot, Wot;        // output tile extent
    int x_rows, x_cols, x_pitch;      // padded x tile: Ht+2h rows, Wt+2h valid cols, pitch
    int dy_rows, dy_cols, dy_pitch;   // padded dy tile: Hot+2h rows, Wot+2h valid cols, pitch
    int64_t x_tile, dy_tile;          // elements per padded tile
    int64_t x_halo, dy_halo;          // elements per packed halo buffer
    int ntiles;
    // margins the passes read beyond a tile, per spatial dimension
    int need_x_lo_r, need_x_hi_r, need_x_lo_s, need_x_hi_s;
    int need_dy_lo_r, need_dy_hi_r, need_dy_lo_s, need_dy_hi_s;
    // halo bands moved by pack/unpack: rows above, below, cols left, right
    int bw_x[4], bw_dy[4];
    // convolution launches take the samples in groups of spg, so that each
    // launch's per-tile tensors stay within 32-bit element indexing
    int spg;
    int64_t x_sample, dy_sample, y_sample, dx_sample;   // elements per sample of each tile tensor
};

// Fill g from prob and check everything that does not depend on a tile index.
dc_status make_geo(const dc_problem* prob, Geo* g);

// make_geo + tile index check (DC_ALL_TILES allowed).
dc_status make_geo_tile(const dc_problem* prob, int32_t tile, Geo* g);

inline int64_t floor_div(int64_t a, int64_t b) {  // b > 0
    int64_t q = a / b;
    return (a % b != 0 && a < 0) ? q - 1 : q;
}
inline int64_t ceil_div(int64_t a, int64_t b) { return -floor_div(-a, b); }

}  // namespace dc
