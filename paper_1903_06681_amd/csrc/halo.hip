// Halo pack / unpack kernels (Sec. III-A; message terms of Sec. V-A).
//
// A tile's margin ring is split into the bands a neighbour supplies: rows
// above and below the owned block (N, S), columns left and right of it (W,
// E) and the four corner blocks.  Band widths are per side: the margins the
// convolution passes actually read (with stride > 1 one side may need fewer
// rows than the other, or none, Sec. III-A).  Packed buffers hold eight
// regions [planes][rows][cols] in the order N, S, W, E, NW, NE, SW, SE; region
// d of a receive buffer has the shape of margin d, region d of a send buffer
// the shape of the neighbour's margin opposite to d.  Unpack writes the whole
// margin ring: received bands where the neighbour exists, zeros elsewhere
// (the convolution's zero padding, and any margin wider than the band).
//
// A workgroup handles a run of planes of one tile (one plane for a single
// tile; several when the grid is large, so that a launch does not consist of
// thousands of tiny workgroups).  Each thread first loads every element it
// moves in a pass and then stores them, so a workgroup pays one memory round
// trip per pass.  N/S rows travel as aligned 16-byte vectors: the side of the
// copy that is not 16-byte aligned (the owned block starts h columns into a
// padded row) is read as two aligned vectors and shifted.  W/E columns and
// corners are single elements.  Copies are bitwise (2- or 4-byte elements).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace dc {

static constexpr int kHaloThreads = 256;
static constexpr int kVecItems = 4;    // 16-byte vectors per thread and pass
static constexpr int kElemItems = 16;  // single elements per thread and pass

__device__ __forceinline__ int dir_di(int d) { return (d == 0 || d == 4 || d == 5) ? -1 : (d == 1 || d == 6 || d == 7) ? 1 : 0; }
__device__ __forceinline__ int dir_dj(int d) { return (d == 2 || d == 4 || d == 6) ? -1 : (d == 3 || d == 5 || d == 7) ? 1 : 0; }
__device__ __forceinline__ int dir_of(int di, int dj) {
    return di == 0 ? (dj < 0 ? 2 : 3) : dj == 0 ? (di < 0 ? 0 : 1) : (di < 0 ? (dj < 0 ? 4 : 5) : (dj < 0 ? 6 : 7));
}
__device__ __forceinline__ int opposite(int d) { return d < 4 ? (d ^ 1) : 11 - d; }

// bytes [bs, bs + 16) of the 32 bytes lo:hi (bs < 16, uniform)
__device__ __forceinline__ uint4 shift_bytes(uint4 lo, uint4 hi, int bs) {
    const uint64_t w0 = uint64_t(lo.x) | (uint64_t(lo.y) << 32), w1 = uint64_t(lo.z) | (uint64_t(lo.w) << 32);
    const uint64_t w2 = uint64_t(hi.x) | (uint64_t(hi.y) << 32), w3 = uint64_t(hi.z) | (uint64_t(hi.w) << 32);
    const bool q = bs >= 8;
    const int b = (bs & 7) * 8;
    const uint64_t a0 = q ? w1 : w0, a1 = q ? w2 : w1, a2 = q ? w3 : w2;
    const uint64_t o0 = b ? (a0 >> b) | (a1 << (64 - b)) : a0;
    const uint64_t o1 = b ? (a1 >> b) | (a2 << (64 - b)) : a1;
    return make_uint4(uint32_t(o0), uint32_t(o0 >> 32), uint32_t(o1), uint32_t(o1 >> 32));
}

struct TileCtx {
    int ti, tj, slot;
    __device__ bool has(const HaloArgs& a, int di, int dj) const {
        const int ni = ti + di, nj = tj + dj;
        return ni >= 0 && ni < a.P && nj >= 0 && nj < a.Q;
    }
};

__device__ __forceinline__ TileCtx tile_ctx(const HaloArgs& a) {
    TileCtx c;
    const int t = a.tile0 + blockIdx.y;
    c.ti = t / a.Q;
    c.tj = t - c.ti * a.Q;
    c.slot = a.all_tiles ? t : 0;   // single-tile calls pass one buffer
    return c;
}

// ---------------------------------------------------------------- pack

template <typename T>
__global__ __launch_bounds__(kHaloThreads) void halo_pack_kernel(HaloArgs a) {
    constexpr int VE = 16 / int(sizeof(T));
    const TileCtx tc = tile_ctx(a);
    const int p0 = blockIdx.x * a.ppw, np = min(a.ppw, a.planes - p0);
    const int h = a.h, ht = a.ht, wt = a.wt;
    const int bN = a.bw[0], bS = a.bw[1], bW = a.bw[2], bE = a.bw[3];
    const T* __restrict__ src0 = static_cast<const T*>(a.src) + int64_t(tc.slot) * a.tile_elems;
    T* __restrict__ dst = static_cast<T*>(a.dst) + int64_t(tc.slot) * a.halo_elems;
    int plane = p0;
    const T* src = src0;
    // send region d: shape of the neighbour's margin opposite(d); origin in the tile
    auto srows = [&](int di) { return di < 0 ? bS : di > 0 ? bN : ht; };
    auto scols = [&](int dj) { return dj < 0 ? bE : dj > 0 ? bW : wt; };
    auto sr0 = [&](int di) { return di > 0 ? h + ht - bN : h; };
    auto sc0 = [&](int dj) { return dj > 0 ? h + wt - bW : h; };
    auto region = [&](int d) -> T* {
        const int di = dir_di(d), dj = dir_dj(d);
        return dst + a.soff[d] + int64_t(plane) * srows(di) * scols(dj);
    };
    const bool ns = (a.bands & DC_BAND_NS) != 0, we = (a.bands & DC_BAND_WE) != 0,
               co = (a.bands & DC_BAND_CORNERS) != 0;
    const bool vec = ns && a.vec;
    const int kpr = wt / VE;                                   // vectors per N/S row
    const int nV = vec ? (bS + bN) * kpr : 0;                  // rows sent north, then south
    const int nNS = ns && !vec ? (bS + bN) * wt : 0;
    const int nWE = we ? ht * (bE + bW) : 0;                   // per row: cols sent west, then east
    const int nC = co ? (bS + bN) * (bE + bW) : 0;
    const int nE = nNS + nWE + nC;
    const int bs = (h % VE) * int(sizeof(T));                  // source misalignment (bytes)
    const int tV = np * nV, tE = np * nE;                      // items of the workgroup's planes

    for (int pv = 0, pe = 0; pv < tV || pe < tE; pv += kHaloThreads * kVecItems, pe += kHaloThreads * kElemItems) {
        uint4 vv[kVecItems];
        T* vdst[kVecItems];
        T ev[kElemItems];
        T* edst[kElemItems];
#pragma unroll
        for (int u = 0; u < kVecItems; ++u) {
            int v = pv + u * kHaloThreads + threadIdx.x;
            vdst[u] = nullptr;
            if (v < tV) {
                const int pl = v / nV;
                v -= pl * nV;
                plane = p0 + pl;
                src = src0 + int64_t(plane) * a.rows * a.pitch;
                const int rr_all = v / kpr, k = v - rr_all * kpr;
                const int di = rr_all < bS ? -1 : 1;
                const int rr = di < 0 ? rr_all : rr_all - bS;
                if (tc.has(a, di, 0)) {
                    const T* row = src + int64_t(sr0(di) + rr) * a.pitch;
                    const int c = h + VE * k, a0 = c & ~(VE - 1);
                    const uint4 lo = *reinterpret_cast<const uint4*>(row + a0);
                    // the second vector stays inside the padded row (pitch >= wt + 2h, rounded to 16 bytes)
                    vv[u] = bs ? shift_bytes(lo, *reinterpret_cast<const uint4*>(row + a0 + VE), bs) : lo;
                    vdst[u] = region(dir_of(di, 0)) + int64_t(rr) * wt + VE * k;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kElemItems; ++u) {
            int e = pe + u * kHaloThreads + threadIdx.x;
            edst[u] = nullptr;
            if (e >= tE) continue;
            const int pl = e / nE;
            e -= pl * nE;
            plane = p0 + pl;
            src = src0 + int64_t(plane) * a.rows * a.pitch;
            int di, dj, rr, cc;
            if (e < nNS) {
                const int ra = e / wt;
                cc = e - ra * wt;
                di = ra < bS ? -1 : 1;
                rr = di < 0 ? ra : ra - bS;
                dj = 0;
            } else if ((e -= nNS) < nWE) {
                const int wdt = bE + bW;
                rr = e / wdt;
                const int k = e - rr * wdt;
                di = 0;
                dj = k < bE ? -1 : 1;
                cc = dj < 0 ? k : k - bE;
            } else {
                e -= nWE;
                const int wdt = bE + bW;
                const int ra = e / wdt, k = e - ra * wdt;
                di = ra < bS ? -1 : 1;
                rr = di < 0 ? ra : ra - bS;
                dj = k < bE ? -1 : 1;
                cc = dj < 0 ? k : k - bE;
            }
            if (!tc.has(a, di, dj)) continue;   // nothing is sent where no neighbour exists
            ev[u] = src[int64_t(sr0(di) + rr) * a.pitch + sc0(dj) + cc];
            edst[u] = region(dir_of(di, dj)) + int64_t(rr) * scols(dj) + cc;
        }
#pragma unroll
        for (int u = 0; u < kVecItems; ++u)
            if (vdst[u]) *reinterpret_cast<uint4*>(vdst[u]) = vv[u];
#pragma unroll
        for (int u = 0; u < kElemItems; ++u)
            if (edst[u]) *edst[u] = ev[u];
    }
}

// ---------------------------------------------------------------- unpack

template <typename T>
__global__ __launch_bounds__(kHaloThreads) void halo_unpack_kernel(HaloArgs a) {
    constexpr int VE = 16 / int(sizeof(T));
    const TileCtx tc = tile_ctx(a);
    const int p0 = blockIdx.x * a.ppw, np = min(a.ppw, a.planes - p0);
    const int h = a.h, ht = a.ht, wt = a.wt;
    const int bN = a.bw[0], bS = a.bw[1], bW = a.bw[2], bE = a.bw[3];
    T* __restrict__ dst0 = static_cast<T*>(a.dst) + int64_t(tc.slot) * a.tile_elems;
    const T* __restrict__ src = static_cast<const T*>(a.src);
    int plane = p0;
    T* dst = dst0;
    // margin d: rows/cols of its band and the band's origin in the tile
    auto mrows = [&](int di) { return di < 0 ? bN : di > 0 ? bS : ht; };
    auto mcols = [&](int dj) { return dj < 0 ? bW : dj > 0 ? bE : wt; };
    auto mr0 = [&](int di) { return di < 0 ? h - bN : di > 0 ? h + ht : h; };
    auto mc0 = [&](int dj) { return dj < 0 ? h - bW : dj > 0 ? h + wt : h; };
    // offset (in src) of this plane's block of the band received from direction d:
    // all tiles: the neighbour's send buffer, its region facing this tile;
    // one tile: this tile's receive buffer, region d
    auto band = [&](int di, int dj) -> int64_t {
        const int d = dir_of(di, dj);
        const int64_t inplane = int64_t(plane) * mrows(di) * mcols(dj);
        if (a.all_tiles)
            return int64_t((tc.ti + di) * a.Q + tc.tj + dj) * a.halo_elems + a.soff[opposite(d)] + inplane;
        return a.roff[d] + inplane;
    };
    // ring cell (r, c): offset of its value in src, or -1 for zero
    auto source = [&](int r, int c) -> int64_t {
        const int di = r < h ? -1 : r >= h + ht ? 1 : 0;
        const int dj = c < h ? -1 : c >= h + wt ? 1 : 0;
        const bool in_band = (di < 0 ? r >= h - bN : di > 0 ? r < h + ht + bS : true) &&
                             (dj < 0 ? c >= h - bW : dj > 0 ? c < h + wt + bE : true);
        if (!in_band || !tc.has(a, di, dj)) return -1;
        return band(di, dj) + int64_t(r - mr0(di)) * mcols(dj) + (c - mc0(dj));
    };
    const bool ns = (a.bands & DC_BAND_NS) != 0, we = (a.bands & DC_BAND_WE) != 0,
               co = (a.bands & DC_BAND_CORNERS) != 0;
    const bool vec = ns && a.vec;
    // aligned vectors of a margin row lying inside columns [h, h + wt)
    const int ka = vec ? (h + VE - 1) / VE : 0, kb = vec ? (h + wt) / VE : 0;
    const int kpr = kb > ka ? kb - ka : 0;
    const int nV = vec ? 2 * h * kpr : 0;
    const int lead = kpr ? VE * ka - h : wt, tail = kpr ? h + wt - VE * kb : 0;   // elements outside the vectors
    const int ne1 = lead + tail;
    const int nNS = ns ? 2 * h * ne1 : 0;
    const int nWE = we ? ht * 2 * h : 0;
    const int nC = co ? 4 * h * h : 0;
    const int nE = nNS + nWE + nC;
    const int bs = ((VE - h % VE) % VE) * int(sizeof(T));   // source misalignment of a vector (bytes)
    auto mrow = [&](int i) { return i < h ? i : ht + i; };  // i-th margin row of the 2h above/below
    const int tV = np * nV, tE = np * nE;                   // items of the workgroup's planes

    for (int pv = 0, pe = 0; pv < tV || pe < tE; pv += kHaloThreads * kVecItems, pe += kHaloThreads * kElemItems) {
        uint4 vv[kVecItems];
        T* vdst[kVecItems];
        T ev[kElemItems];
        T* edst[kElemItems];
#pragma unroll
        for (int u = 0; u < kVecItems; ++u) {
            int v = pv + u * kHaloThreads + threadIdx.x;
            vdst[u] = nullptr;
            if (v >= tV) continue;
            const int pl = v / nV;
            v -= pl * nV;
            plane = p0 + pl;
            dst = dst0 + int64_t(plane) * a.rows * a.pitch;
            const int i = v / kpr, k = ka + (v - i * kpr);
            const int r = mrow(i), c = VE * k;
            vdst[u] = dst + int64_t(r) * a.pitch + c;
            const int64_t o = source(r, c);   // the whole vector shares the row's band and neighbour
            if (o < 0) {
                vv[u] = make_uint4(0, 0, 0, 0);
                continue;
            }
            // region rows are 16-byte aligned (host check); o - shift is the aligned vector below
            const int64_t a0 = o - bs / int(sizeof(T));
            const uint4 lo = *reinterpret_cast<const uint4*>(src + a0);
            if (bs == 0) {
                vv[u] = lo;
            } else if (a0 + 2 * VE <= a.src_elems) {
                vv[u] = shift_bytes(lo, *reinterpret_cast<const uint4*>(src + a0 + VE), bs);
            } else {   // the last vector of the buffer: elements one by one
                T t[VE];
#pragma unroll
                for (int j = 0; j < VE; ++j) t[j] = src[o + j];
                vv[u] = *reinterpret_cast<const uint4*>(t);
            }
        }
#pragma unroll
        for (int u = 0; u < kElemItems; ++u) {
            int e = pe + u * kHaloThreads + threadIdx.x;
            edst[u] = nullptr;
            if (e >= tE) continue;
            const int pl = e / nE;
            e -= pl * nE;
            plane = p0 + pl;
            dst = dst0 + int64_t(plane) * a.rows * a.pitch;
            int r, c;
            if (e < nNS) {
                const int i = e / ne1, k = e - i * ne1;
                r = mrow(i);
                c = k < lead ? h + k : VE * kb + (k - lead);
            } else if ((e -= nNS) < nWE) {
                const int i = e / (2 * h), k = e - i * (2 * h);
                r = h + i;
                c = k < h ? k : wt + k;
            } else {
                e -= nWE;
                const int blk = e / (h * h), in = e - blk * (h * h);
                const int rr = in / h, cc = in - rr * h;
                r = (blk & 2) ? h + ht + rr : rr;
                c = (blk & 1) ? h + wt + cc : cc;
            }
            const int64_t o = source(r, c);
            ev[u] = o < 0 ? T(0) : src[o];
            edst[u] = dst + int64_t(r) * a.pitch + c;
        }
#pragma unroll
        for (int u = 0; u < kVecItems; ++u)
            if (vdst[u]) *reinterpret_cast<uint4*>(vdst[u]) = vv[u];
#pragma unroll
        for (int u = 0; u < kElemItems; ++u)
            if (edst[u]) *edst[u] = ev[u];
    }
}

hipError_t launch_halo_pack(const HaloArgs& a, int esize, hipStream_t s) {
    dim3 grid((a.planes + a.ppw - 1) / a.ppw, a.ntiles), block(kHaloThreads);
    if (esize == 2)
        hipLaunchKernelGGL(halo_pack_kernel<uint16_t>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(halo_pack_kernel<uint32_t>, grid, block, 0, s, a);
    return hipGetLastError();
}

hipError_t launch_halo_unpack(const HaloArgs& a, int esize, hipStream_t s) {
    dim3 grid((a.planes + a.ppw - 1) / a.ppw, a.ntiles), block(kHaloThreads);
    if (esize == 2)
        hipLaunchKernelGGL(halo_unpack_kernel<uint16_t>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(halo_unpack_kernel<uint32_t>, grid, block, 0, s, a);
    return hipGetLastError();
}

}  // namespace dc
