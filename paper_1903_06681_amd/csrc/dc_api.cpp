// C entry points of libdc: argument validation, tile geometry and kernel
// dispatch.  No allocation, no state, no synchronisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

#include "dc.h"
#include "geometry.h"
#include "kernels.h"

namespace dc {

static const int64_t kMaxElems = (int64_t(1) << 31) - 1;

static int round_up(int v, int m) { return (v + m - 1) / m * m; }

// Margins Eq. (1) reads around a tile of `t_in` input / `t_out` output
// positions along one axis: output positions p read inputs p*stride-pad+r.
static void x_margins(int t_in, int t_out, int R, int stride, int pad, int* lo, int* hi) {
    *lo = pad;
    int last = (t_out - 1) * stride - pad + R - 1;   // furthest input read
    *hi = std::max(0, last - (t_in - 1));
}

// Margins Eq. (3) reads around a tile: input position i reads output
// positions (i+pad-r)/stride where the division is exact.
static void dy_margins(int t_in, int t_out, int R, int stride, int pad, int* lo, int* hi) {
    int64_t mmin = ceil_div(int64_t(pad) - (R - 1), stride);
    int64_t mmax = floor_div(int64_t(t_in) - 1 + pad, stride);
    *lo = int(std::max<int64_t>(0, -mmin));
    *hi = int(std::max<int64_t>(0, mmax - (t_out - 1)));
}

// Elements per plane of the eight bands of a ht x wt tile with band widths
// bw = {above, below, left, right}.
static int64_t halo_band_elems(const int bw[4], int ht, int wt) {
    const int64_t rows = bw[0] + bw[1], cols = bw[2] + bw[3];
    return rows * wt + int64_t(ht) * cols + rows * cols;
}

dc_status make_geo(const dc_problem* p, Geo* g) {
    if (!p || !g) return DC_ERR_NULL;
    std::memset(g, 0, sizeof(*g));
    if (p->N < 1 || p->C < 1 || p->K < 1 || p->H < 1 || p->W < 1 || p->R < 1 || p->S < 1 ||
        p->stride < 1 || p->pad < 0 || p->P < 1 || p->Q < 1 || p->halo < 0)
        return DC_ERR_SHAPE;
    if (p->dtype != DC_F32 && p->dtype != DC_BF16) return DC_ERR_DTYPE;
    g->N = p->N; g->C = p->C; g->K = p->K; g->H = p->H; g->W = p->W;
    g->R = p->R; g->S = p->S; g->stride = p->stride; g->pad = p->pad;
    g->P = p->P; g->Q = p->Q; g->h = p->halo; g->dtype = p->dtype;
    g->esize = p->dtype == DC_BF16 ? 2 : 4;

    int64_t ho = floor_div(int64_t(p->H) + 2 * int64_t(p->pad) - p->R, p->stride) + 1;
    int64_t wo = floor_div(int64_t(p->W) + 2 * int64_t(p->pad) - p->S, p->stride) + 1;
    if (ho < 1 || wo < 1) return DC_ERR_SHAPE;
    g->Ho = int(ho); g->Wo = int(wo);
    if (p->H % p->P != 0 || p->W % p->Q != 0) return DC_ERR_UNSUPPORTED;
    g->ntiles = p->P * p->Q;
    if (g->ntiles > 1) {
        // Decomposed layers (Sec. III-A): the output grid must line up with
        // the input grid, Ho * stride == H, so that the Ht/stride x Wt/stride
        // output block of a tile is exactly the outputs whose taps start in
        // it; and the output tiles must divide evenly too.
        if (int64_t(g->Ho) * p->stride != p->H || int64_t(g->Wo) * p->stride != p->W)
            return DC_ERR_UNSUPPORTED;
        if (g->Ho % p->P != 0 || g->Wo % p->Q != 0) return DC_ERR_UNSUPPORTED;
    }
    g->Ht = p->H / p->P; g->Wt = p->W / p->Q;
    g->Hot = g->Ho / p->P; g->Wot = g->Wo / p->Q;

    x_margins(g->Ht, g->Hot, p->R, p->stride, p->pad, &g->need_x_lo_r, &g->need_x_hi_r);
    x_margins(g->Wt, g->Wot, p->S, p->stride, p->pad, &g->need_x_lo_s, &g->need_x_hi_s);
    dy_margins(g->Ht, g->Hot, p->R, p->stride, p->pad, &g->need_dy_lo_r, &g->need_dy_hi_r);
    dy_margins(g->Wt, g->Wot, p->S, p->stride, p->pad, &g->need_dy_lo_s, &g->need_dy_hi_s);
    int need = std::max({g->need_x_lo_r, g->need_x_hi_r, g->need_x_lo_s, g->need_x_hi_s,
                         g->need_dy_lo_r, g->need_dy_hi_r, g->need_dy_lo_s, g->need_dy_hi_s});
    if (g->h < need) return DC_ERR_HALO;
    // halos come from the adjacent tile only (for x and for dy tiles)
    if ((p->P > 1 && (g->h > g->Ht || g->h > g->Hot)) || (p->Q > 1 && (g->h > g->Wt || g->h > g->Wot)))
        return DC_ERR_HALO;

    const int align = 16 / g->esize;
    g->x_rows = g->Ht + 2 * g->h;  g->x_cols = g->Wt + 2 * g->h;
    g->dy_rows = g->Hot + 2 * g->h; g->dy_cols = g->Wot + 2 * g->h;
    g->x_pitch = round_up(g->x_cols, align);
    g->dy_pitch = round_up(g->dy_cols, align);
    g->x_tile = int64_t(g->N) * g->C * g->x_rows * g->x_pitch;
    g->dy_tile = int64_t(g->N) * g->K * g->dy_rows * g->dy_pitch;
    // bands: the margins each pass reads (Sec. III-A), per side
    const int bx[4] = {g->need_x_lo_r, g->need_x_hi_r, g->need_x_lo_s, g->need_x_hi_s};
    const int by[4] = {g->need_dy_lo_r, g->need_dy_hi_r, g->need_dy_lo_s, g->need_dy_hi_s};
    for (int i = 0; i < 4; ++i) { g->bw_x[i] = bx[i]; g->bw_dy[i] = by[i]; }
    // packed buffers end on a 16-byte boundary, so that the consecutive
    // per-tile buffers of an all-tiles call each start 16-byte aligned
    auto round16 = [&](int64_t e) { const int64_t a = 16 / g->esize; return (e + a - 1) / a * a; };
    g->x_halo = round16(int64_t(g->N) * g->C * halo_band_elems(g->bw_x, g->Ht, g->Wt));
    g->dy_halo = round16(int64_t(g->N) * g->K * halo_band_elems(g->bw_dy, g->Hot, g->Wot));
    g->x_sample = int64_t(g->C) * g->x_rows * g->x_pitch;
    g->dy_sample = int64_t(g->K) * g->dy_rows * g->dy_pitch;
    g->y_sample = int64_t(g->K) * g->Hot * g->Wot;
    g->dx_sample = int64_t(g->C) * g->Ht * g->Wt;
    const int64_t w_elems = int64_t(g->K) * g->C * g->R * g->S;
    const int64_t per_sample = std::max({g->x_sample, g->dy_sample, g->y_sample, g->dx_sample});
    // the kernels index one launch's tile tensors with 32-bit element offsets:
    // larger tiles are run in groups of samples (one sample must fit)
    if (per_sample > kMaxElems || w_elems > kMaxElems) return DC_ERR_TOO_LARGE;
    g->spg = int(std::min<int64_t>(g->N, kMaxElems / per_sample));
    return DC_OK;
}

dc_status make_geo_tile(const dc_problem* p, int32_t tile, Geo* g) {
    dc_status st = make_geo(p, g);
    if (st != DC_OK) return st;
    if (tile != DC_ALL_TILES && (tile < 0 || tile >= g->ntiles)) return DC_ERR_TILE;
    return DC_OK;
}

int device_lds_limit() {
    // per-device cache; a benign race at worst re-queries the same value
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 64 * 1024;
    if (cache[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
            v <= 0)
            v = 64 * 1024;
        cache[dev] = v;
    }
    return cache[dev];
}

int device_cu_count() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
            v = 256;
        cache[dev] = v;
    }
    return cache[dev];
}

static bool misaligned(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) != 0; }

static dc_status launched(hipError_t e) {
    if (e != hipSuccess) return DC_ERR_HIP;
    return hipGetLastError() == hipSuccess ? DC_OK : DC_ERR_HIP;
}

// hipGetLastError reports the last error of any earlier HIP call on this
// thread, including the caller's own; clear it before launching so that only
// this call's launches can turn into DC_ERR_HIP.
static void clear_stale_error() { (void)hipGetLastError(); }

// ---------------------------------------------------------------- halo

static dc_status halo_common(const dc_problem* prob, int32_t tile, int32_t which, int32_t bands,
                             const void* src, void* dst, bool unpack, void* stream) {
    Geo g;
    dc_status st = make_geo_tile(prob, tile, &g);
    if (st != DC_OK) return st;
    if (which != DC_X && which != DC_DY) return DC_ERR_ARG;
    if (bands <= 0 || (bands & ~DC_BAND_ALL) != 0) return DC_ERR_ARG;
    const bool x = which == DC_X;
    const int ch = x ? g.C : g.K;
    const int Ht = x ? g.Ht : g.Hot, Wt = x ? g.Wt : g.Wot;
    if (g.h == 0) return DC_OK;  // K = 1: no margin at all (Sec. III-A)
    // the packed buffer (send of a pack, recv of an unpack) may be null when
    // every band is empty (a margin that no pass reads): there is nothing to
    // send, and the unpack only zero-fills the margin ring
    const bool empty = (x ? g.x_halo : g.dy_halo) == 0;
    const void* packed = unpack ? src : dst;
    const void* tile_pad = unpack ? dst : src;
    if (!tile_pad || (!packed && !empty)) return DC_ERR_NULL;
    if (misaligned(tile_pad) || (packed && misaligned(packed))) return DC_ERR_ALIGN;
    if (empty && !unpack) return DC_OK;
    HaloArgs a;
    std::memset(&a, 0, sizeof(a));
    a.src = src; a.dst = dst;
    a.tile_elems = x ? g.x_tile : g.dy_tile;
    a.halo_elems = x ? g.x_halo : g.dy_halo;
    a.planes = g.N * ch;
    a.rows = x ? g.x_rows : g.dy_rows;
    a.pitch = x ? g.x_pitch : g.dy_pitch;
    a.ht = Ht; a.wt = Wt; a.h = g.h;
    const int* bw = x ? g.bw_x : g.bw_dy;
    for (int i = 0; i < 4; ++i) a.bw[i] = bw[i];
    // region offsets: receive region d has margin d's band shape, send region
    // d the shape of margin opposite(d) (order N, S, W, E, NW, NE, SW, SE)
    static const int di[8] = {-1, 1, 0, 0, -1, -1, 1, 1}, dj[8] = {0, 0, -1, 1, -1, 1, -1, 1};
    auto band = [&](int d) {
        const int64_t r = di[d] < 0 ? bw[0] : di[d] > 0 ? bw[1] : Ht;
        const int64_t c = dj[d] < 0 ? bw[2] : dj[d] > 0 ? bw[3] : Wt;
        return int64_t(a.planes) * r * c;
    };
    static const int opp[8] = {1, 0, 3, 2, 7, 6, 5, 4};
    int64_t ro = 0, so = 0;
    for (int d = 0; d < 8; ++d) {
        a.roff[d] = ro; ro += band(d);
        a.soff[d] = so; so += band(opp[d]);
    }
    a.P = g.P; a.Q = g.Q;
    a.all_tiles = tile == DC_ALL_TILES;
    a.tile0 = a.all_tiles ? 0 : tile;
    a.ntiles = a.all_tiles ? g.ntiles : 1;
    a.src_elems = unpack ? (a.all_tiles ? int64_t(g.ntiles) * a.halo_elems : a.halo_elems) : a.tile_elems;
    a.bands = bands;
    // N/S rows as aligned 16-byte vectors: rows of whole vectors that start on
    // a 16-byte boundary in every buffer (tile rows are 16-byte aligned)
    const int ve = 16 / g.esize;
    a.vec = Wt % ve == 0 && a.halo_elems % ve == 0 && a.roff[1] % ve == 0 && a.soff[1] % ve == 0;
    // Row bands and corners: a few hundred workgroups per launch, several
    // planes each beyond that (thousands of tiny workgroups cost more to
    // dispatch than they move).  With W/E columns one plane per workgroup:
    // their gathers touch a cache line per element and go faster with more
    // workgroups in flight (measured on a 4x4 grid of 256x256 tiles).
    const int64_t planes_total = int64_t(a.planes) * a.ntiles;
    a.ppw = (bands & DC_BAND_WE) ? 1 : int(std::max<int64_t>(1, std::min<int64_t>(16, planes_total / 512)));
    hipStream_t s = static_cast<hipStream_t>(stream);
    clear_stale_error();
    return launched(unpack ? launch_halo_unpack(a, g.esize, s) : launch_halo_pack(a, g.esize, s));
}

// ---------------------------------------------------------------- convs

static void igemm_common(const Geo& g, int32_t tile, IgemmArgs& a) {
    std::memset(&a, 0, sizeof(a));
    a.ntiles = tile == DC_ALL_TILES ? g.ntiles : 1;
    a.Nn = g.N;
    a.R = g.R; a.S = g.S;
    a.wK = g.K; a.wC = g.C;
}

// One launch per group of g.spg samples (a single one unless the tile's
// tensors exceed 32-bit indexing): the input and output pointers advance by
// in_sample / out_sample elements per sample; tile strides stay those of the
// whole tile.  Each launch is planned here; false if one cannot be.
static bool plan_groups(const Geo& g, const IgemmArgs& a, int64_t in_sample, int64_t out_sample,
                        std::vector<IgemmArgs>& out) {
    const int64_t ebytes = g.esize;
    for (int n0 = 0; n0 < g.N; n0 += g.spg) {
        IgemmArgs ak = a;
        ak.Nn = std::min(g.spg, g.N - n0);
        ak.in = static_cast<const char*>(a.in) + n0 * in_sample * ebytes;
        ak.out = a.out + n0 * out_sample;
        if (!igemm_plan(ak, g.dtype)) return false;
        out.push_back(ak);
    }
    return true;
}

// Workspace of the weight gradient: the largest of its sample groups' (they
// run one after another on the stream and share it).
static size_t bwd_filter_need(const Geo& g, int32_t tile) {
    const int nt = tile == DC_ALL_TILES ? g.ntiles : 1;
    size_t need = 0;
    for (int n0 = 0; n0 < g.N; n0 += g.spg)
        need = std::max(need, wgrad_workspace_bytes(g.dtype, nt, std::min(g.spg, g.N - n0), g.C, g.K, g.R,
                                                     g.S, g.stride, g.Hot, g.Wot, g.h - g.pad, g.h));
    return need;
}

static dc_status launch_all(const std::vector<IgemmArgs>& v, int dtype, hipStream_t s) {
    clear_stale_error();
    for (const IgemmArgs& a : v) {
        dc_status r = launched(launch_igemm(a, dtype, s));
        if (r != DC_OK) return r;
    }
    return DC_OK;
}

}  // namespace dc

using namespace dc;

extern "C" {

dc_status dc_validate(const dc_problem* prob, int32_t tile) {
    Geo g;
    return make_geo_tile(prob, tile, &g);
}

int64_t dc_tile_pitch(const dc_problem* prob, int32_t which) {
    Geo g;
    if (make_geo(prob, &g) != DC_OK || (which != DC_X && which != DC_DY)) return -1;
    return which == DC_X ? g.x_pitch : g.dy_pitch;
}

int64_t dc_tile_elems(const dc_problem* prob, int32_t which) {
    Geo g;
    if (make_geo(prob, &g) != DC_OK || (which != DC_X && which != DC_DY)) return -1;
    return which == DC_X ? g.x_tile : g.dy_tile;
}

int64_t dc_halo_elems(const dc_problem* prob, int32_t which) {
    Geo g;
    if (make_geo(prob, &g) != DC_OK || (which != DC_X && which != DC_DY)) return -1;
    return which == DC_X ? g.x_halo : g.dy_halo;
}

dc_status dc_required_halo(const dc_problem* prob, int32_t which, int32_t lohi[2]) {
    if (!lohi) return DC_ERR_NULL;
    dc_problem q;
    if (!prob) return DC_ERR_NULL;
    q = *prob;
    // the requirement does not depend on the halo field: evaluate with a
    // margin wide enough to pass the width check
    q.halo = std::max(std::max(q.R, q.S) + q.pad, 0);
    Geo g;
    dc_status st = make_geo(&q, &g);
    if (st != DC_OK && st != DC_ERR_HALO) return st;
    if (st == DC_ERR_HALO) {
        // tile narrower than the probe margin: recompute the margins directly
        q.halo = 0;
        st = make_geo(&q, &g);
        if (st != DC_OK && st != DC_ERR_HALO) return st;
    }
    if (which == DC_X) {
        lohi[0] = std::max(g.need_x_lo_r, g.need_x_lo_s);
        lohi[1] = std::max(g.need_x_hi_r, g.need_x_hi_s);
    } else if (which == DC_DY) {
        lohi[0] = std::max(g.need_dy_lo_r, g.need_dy_lo_s);
        lohi[1] = std::max(g.need_dy_hi_r, g.need_dy_hi_s);
    } else {
        return DC_ERR_ARG;
    }
    return DC_OK;
}

dc_status dc_tile_dims(const dc_problem* prob, int32_t dims[4]) {
    if (!dims) return DC_ERR_NULL;
    Geo g;
    dc_status st = make_geo(prob, &g);
    if (st != DC_OK) return st;
    dims[0] = g.Ht; dims[1] = g.Wt; dims[2] = g.Hot; dims[3] = g.Wot;
    return DC_OK;
}

const char* dc_status_string(int32_t s) {
    switch (s) {
        case DC_OK: return "ok";
        case DC_ERR_NULL: return "null pointer";
        case DC_ERR_SHAPE: return "invalid shape";
        case DC_ERR_DTYPE: return "invalid dtype";
        case DC_ERR_HALO: return "halo width does not fit the layer or the tiles";
        case DC_ERR_UNSUPPORTED: return "unsupported decomposition";
        case DC_ERR_WORKSPACE: return "workspace missing or too small";
        case DC_ERR_ALIGN: return "device pointer not 16-byte aligned";
        case DC_ERR_HIP: return "HIP runtime error";
        case DC_ERR_TILE: return "tile index out of range";
        case DC_ERR_ARG: return "invalid argument";
        case DC_ERR_TOO_LARGE: return "tensor too large for 32-bit element indexing";
        default: return "unknown status";
    }
}

dc_status dc_halo_pack(const dc_problem* prob, int32_t tile, int32_t which,
                       const void* t_pad, void* send, void* stream) {
    return halo_common(prob, tile, which, DC_BAND_ALL, t_pad, send, false, stream);
}

dc_status dc_halo_unpack(const dc_problem* prob, int32_t tile, int32_t which,
                         const void* recv, void* t_pad, void* stream) {
    return halo_common(prob, tile, which, DC_BAND_ALL, recv, t_pad, true, stream);
}

dc_status dc_halo_pack_bands(const dc_problem* prob, int32_t tile, int32_t which, int32_t bands,
                             const void* t_pad, void* send, void* stream) {
    return halo_common(prob, tile, which, bands, t_pad, send, false, stream);
}

dc_status dc_halo_unpack_bands(const dc_problem* prob, int32_t tile, int32_t which, int32_t bands,
                               const void* recv, void* t_pad, void* stream) {
    return halo_common(prob, tile, which, bands, recv, t_pad, true, stream);
}

dc_status dc_halo_bands(const dc_problem* prob, int32_t which, int32_t bw[4]) {
    if (!bw) return DC_ERR_NULL;
    Geo g;
    dc_status st = make_geo(prob, &g);
    if (st != DC_OK) return st;
    if (which != DC_X && which != DC_DY) return DC_ERR_ARG;
    for (int i = 0; i < 4; ++i) bw[i] = which == DC_X ? g.bw_x[i] : g.bw_dy[i];
    return DC_OK;
}

dc_status dc_conv_fwd(const dc_problem* prob, int32_t tile, const void* x_pad,
                      const void* w, float* y, void* stream) {
    return dc_conv_fwd_region(prob, tile, DC_REGION_ALL, x_pad, w, y, stream);
}

dc_status dc_conv_fwd_region(const dc_problem* prob, int32_t tile, int32_t region, const void* x_pad,
                             const void* w, float* y, void* stream) {
    Geo g;
    dc_status st = make_geo_tile(prob, tile, &g);
    if (st != DC_OK) return st;
    if (region != DC_REGION_ALL && region != DC_REGION_INTERIOR && region != DC_REGION_BOUNDARY)
        return DC_ERR_ARG;
    if (!x_pad || !w || !y) return DC_ERR_NULL;
    if (misaligned(x_pad) || misaligned(w) || misaligned(y)) return DC_ERR_ALIGN;
    if (region != DC_REGION_ALL && g.stride != 1) return DC_ERR_UNSUPPORTED;
    IgemmArgs a;
    igemm_common(g, tile, a);
    a.in = x_pad; a.w = w; a.out = y;
    a.in_tile = g.x_tile;
    a.out_tile = int64_t(g.N) * g.K * g.Hot * g.Wot;
    a.Cin = g.C; a.Cout = g.K;
    a.in_rows = g.x_rows; a.in_cols = g.x_cols; a.in_pitch = g.x_pitch;
    a.Uo = g.Hot; a.Vo = g.Wot;
    a.out_rows = g.Hot; a.out_cols = g.Wot;
    a.ostr = 1; a.oph_r = 0; a.oph_c = 0;
    a.istr = g.stride;
    a.Tr = g.R; a.Ts = g.S;
    a.base_r = g.h - g.pad; a.base_c = g.h - g.pad;
    a.wr0 = 0; a.wrstep = 1; a.ws0 = 0; a.wsstep = 1;
    a.w_os = int64_t(g.C) * g.R * g.S; a.w_cs = int64_t(g.R) * g.S;
    a.wmode = 0;
    // stride 1: the outputs that read x's halo bands are the frame of those
    // widths (output row p reads input rows p - pad .. p - pad + R - 1)
    if (region == DC_REGION_BOUNDARY) igemm_set_frame(a, g.bw_x);
    std::vector<IgemmArgs> launches;
    if (!plan_groups(g, a, g.x_sample, g.y_sample, launches)) return DC_ERR_UNSUPPORTED;
    return launch_all(launches, g.dtype, static_cast<hipStream_t>(stream));
}

dc_status dc_conv_bwd_data(const dc_problem* prob, int32_t tile, const void* dy_pad,
                           const void* w, float* dx, void* stream) {
    return dc_conv_bwd_data_region(prob, tile, DC_REGION_ALL, dy_pad, w, dx, stream);
}

dc_status dc_conv_bwd_data_region(const dc_problem* prob, int32_t tile, int32_t region,
                                  const void* dy_pad, const void* w, float* dx, void* stream) {
    Geo g;
    dc_status st = make_geo_tile(prob, tile, &g);
    if (st != DC_OK) return st;
    if (region != DC_REGION_ALL && region != DC_REGION_INTERIOR && region != DC_REGION_BOUNDARY)
        return DC_ERR_ARG;
    if (!dy_pad || !w || !dx) return DC_ERR_NULL;
    if (misaligned(dy_pad) || misaligned(w) || misaligned(dx)) return DC_ERR_ALIGN;
    if (region != DC_REGION_ALL && g.stride != 1) return DC_ERR_UNSUPPORTED;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int st_ = g.stride;
    // Stride 2 with at most 8 channels: the four output phases below share
    // one stride-1 correlation over dy, whose window is the union of theirs;
    // one launch computes all of them (4 C rows of the MFMA block instead of
    // C per launch).
    if (st_ == 2 && g.dtype == DC_BF16 && 4 * g.C <= 32 && g.Ht % 2 == 0 && g.Wt % 2 == 0) {
        IgemmArgs a;
        igemm_common(g, tile, a);
        a.in = dy_pad; a.w = w; a.out = dx;
        a.in_tile = g.dy_tile;
        a.out_tile = int64_t(g.N) * g.C * g.Ht * g.Wt;
        a.Cin = g.K; a.Cout = 4 * g.C;
        a.in_rows = g.dy_rows; a.in_cols = g.dy_cols; a.in_pitch = g.dy_pitch;
        a.out_rows = g.Ht; a.out_cols = g.Wt;
        a.ostr = 2; a.istr = 1;
        a.Uo = g.Ht / 2; a.Vo = g.Wt / 2;
        int br[2], bc[2];
        bool ok = true;
        for (int ph = 0; ph < 2; ++ph) {
            const int rr = (ph + g.pad) % 2, rc = (ph + g.pad) % 2;
            const int tr = rr < g.R ? (g.R - rr + 1) / 2 : 0, ts = rc < g.S ? (g.S - rc + 1) / 2 : 0;
            if (tr == 0 || ts == 0) ok = false;
            a.bptr[ph] = tr; a.bpts[ph] = ts;
            br[ph] = g.h + (ph + g.pad - rr) / 2 - (tr - 1);
            bc[ph] = g.h + (ph + g.pad - rc) / 2 - (ts - 1);
            a.bpr0[ph] = rr + 2 * (tr - 1);
            a.bps0[ph] = rc + 2 * (ts - 1);
        }
        a.base_r = std::min(br[0], br[1]);
        a.base_c = std::min(bc[0], bc[1]);
        a.Tr = a.Ts = 0;
        for (int ph = 0; ph < 2; ++ph) {
            a.bpdr[ph] = br[ph] - a.base_r;
            a.bpdc[ph] = bc[ph] - a.base_c;
            a.Tr = std::max(a.Tr, a.bpdr[ph] + a.bptr[ph]);
            a.Ts = std::max(a.Ts, a.bpdc[ph] + a.bpts[ph]);
        }
        a.bp = 1; a.bpC = g.C;
        a.w_os = int64_t(g.R) * g.S; a.w_cs = int64_t(g.C) * g.R * g.S;
        a.wmode = 0;
        std::vector<IgemmArgs> launches;
        if (ok && a.base_r >= 0 && a.base_c >= 0 && plan_groups(g, a, g.dy_sample, g.dx_sample, launches))
            return launch_all(launches, g.dtype, s);
    }
    // Eq. (3) split by output phase (i mod stride, j mod stride): each phase
    // is a stride-1 correlation of dy with the taps r = (phase+pad) mod stride
    // + stride*t, visited in reverse.  At stride 1 there is one phase holding
    // the whole filter reversed.
    std::vector<IgemmArgs> phases;
    for (int phr = 0; phr < st_; ++phr) {
        for (int phc = 0; phc < st_; ++phc) {
            IgemmArgs a;
            igemm_common(g, tile, a);
            a.in = dy_pad; a.w = w; a.out = dx;
            a.in_tile = g.dy_tile;
            a.out_tile = int64_t(g.N) * g.C * g.Ht * g.Wt;
            a.Cin = g.K; a.Cout = g.C;
            a.in_rows = g.dy_rows; a.in_cols = g.dy_cols; a.in_pitch = g.dy_pitch;
            a.out_rows = g.Ht; a.out_cols = g.Wt;
            a.ostr = st_; a.oph_r = phr; a.oph_c = phc;
            a.istr = 1;
            const int rr = (phr + g.pad) % st_, rc = (phc + g.pad) % st_;
            a.Tr = rr < g.R ? (g.R - rr + st_ - 1) / st_ : 0;
            a.Ts = rc < g.S ? (g.S - rc + st_ - 1) / st_ : 0;
            a.Uo = g.Ht > phr ? (g.Ht - phr + st_ - 1) / st_ : 0;
            a.Vo = g.Wt > phc ? (g.Wt - phc + st_ - 1) / st_ : 0;
            if (a.Uo == 0 || a.Vo == 0) continue;
            a.base_r = g.h + (phr + g.pad - rr) / st_ - (a.Tr - 1);
            a.base_c = g.h + (phc + g.pad - rc) / st_ - (a.Ts - 1);
            a.wr0 = rr + st_ * (a.Tr - 1); a.wrstep = -st_;
            a.ws0 = rc + st_ * (a.Ts - 1); a.wsstep = -st_;
            if (a.Tr == 0 || a.Ts == 0) { a.Tr = 0; a.Ts = 0; a.base_r = 0; a.base_c = 0; }
            a.w_os = int64_t(g.R) * g.S; a.w_cs = int64_t(g.C) * g.R * g.S;
            a.wmode = 1;
            // stride 1: the inputs whose gradient reads dy's halo bands are the
            // frame of those widths (dx row i reads dy rows i + pad - R + 1 .. i + pad)
            if (region == DC_REGION_BOUNDARY) igemm_set_frame(a, g.bw_dy);
            if (!plan_groups(g, a, g.dy_sample, g.dx_sample, phases)) return DC_ERR_UNSUPPORTED;
        }
    }
    // every phase is planned before the first launch: an unsupported one
    // launches nothing
    return launch_all(phases, g.dtype, s);
}

size_t dc_bwd_filter_workspace_bytes(const dc_problem* prob, int32_t tile) {
    Geo g;
    if (make_geo_tile(prob, tile, &g) != DC_OK) return 0;
    return bwd_filter_need(g, tile);
}

}  // extern "C"

namespace dc {

// Checks shared by both weight-gradient entry points; *need = workspace bytes.
static dc_status bwd_filter_check(const dc_problem* prob, int32_t tile, const void* x_pad,
                                  const void* dy_pad, const float* dw, int32_t accumulate, Geo* g,
                                  size_t* need) {
    dc_status st = make_geo_tile(prob, tile, g);
    if (st != DC_OK) return st;
    if (accumulate != 0 && accumulate != 1) return DC_ERR_ARG;
    if (!x_pad || !dy_pad || !dw) return DC_ERR_NULL;
    if (misaligned(x_pad) || misaligned(dy_pad) || misaligned(dw)) return DC_ERR_ALIGN;
    *need = bwd_filter_need(*g, tile);
    return DC_OK;
}

static dc_status bwd_filter_launch(const Geo& g, int32_t tile, const void* x_pad, const void* dy_pad,
                                   float* dw, int32_t accumulate, void* workspace, void* stream) {
    const int nt = tile == DC_ALL_TILES ? g.ntiles : 1;
    // sample groups (one unless the tile exceeds 32-bit indexing) in order,
    // each adding its partial to dw after the first: a fixed summation order
    std::vector<WgradArgs> launches;
    for (int n0 = 0; n0 < g.N; n0 += g.spg) {
        WgradArgs a;
        std::memset(&a, 0, sizeof(a));
        a.x = static_cast<const char*>(x_pad) + n0 * g.x_sample * g.esize;
        a.dy = static_cast<const char*>(dy_pad) + n0 * g.dy_sample * g.esize;
        a.part = static_cast<float*>(workspace); a.dw = dw;
        a.x_tile = g.x_tile; a.dy_tile = g.dy_tile;
        a.ntiles = nt; a.Nn = std::min(g.spg, g.N - n0);
        a.C = g.C; a.K = g.K; a.R = g.R; a.S = g.S;
        a.x_rows = g.x_rows; a.x_cols = g.x_cols; a.x_pitch = g.x_pitch;
        a.dy_pitch = g.dy_pitch; a.dy_off = g.h;
        a.Hot = g.Hot; a.Wot = g.Wot;
        a.istr = g.stride;
        a.base_r = g.h - g.pad; a.base_c = g.h - g.pad;
        a.accumulate = n0 == 0 ? accumulate : 1;
        if (!wgrad_plan(a, g.dtype)) return DC_ERR_UNSUPPORTED;
        launches.push_back(a);
    }
    clear_stale_error();
    for (const WgradArgs& a : launches) {
        dc_status r = launched(launch_wgrad(a, g.dtype, static_cast<hipStream_t>(stream)));
        if (r != DC_OK) return r;
    }
    return DC_OK;
}

}  // namespace dc

extern "C" {

dc_status dc_conv_bwd_filter(const dc_problem* prob, int32_t tile, const void* x_pad,
                             const void* dy_pad, float* dw, int32_t accumulate,
                             void* workspace, size_t workspace_bytes, void* stream) {
    Geo g;
    size_t need = 0;
    dc_status st = bwd_filter_check(prob, tile, x_pad, dy_pad, dw, accumulate, &g, &need);
    if (st != DC_OK) return st;
    if (need > 0 && (!workspace || workspace_bytes < need)) return DC_ERR_WORKSPACE;
    if (need > 0 && misaligned(workspace)) return DC_ERR_ALIGN;
    return bwd_filter_launch(g, tile, x_pad, dy_pad, dw, accumulate, workspace, stream);
}

dc_status dc_conv_bwd_filter_noalloc(const dc_problem* prob, int32_t tile, const void* x_pad,
                                     const void* dy_pad, float* dw, int32_t accumulate,
                                     void* stream) {
    Geo g;
    size_t need = 0;
    dc_status st = bwd_filter_check(prob, tile, x_pad, dy_pad, dw, accumulate, &g, &need);
    if (st != DC_OK) return st;
    if (need > wgrad_scratch_capacity()) return DC_ERR_WORKSPACE;
    void* ws = nullptr;
    if (need > 0 && wgrad_scratch_ptr(&ws) != hipSuccess) return DC_ERR_HIP;
    return bwd_filter_launch(g, tile, x_pad, dy_pad, dw, accumulate, ws, stream);
}

}  // extern "C"
