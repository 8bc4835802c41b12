// Halo pack / unpack kernels (Sec. III-A; message terms of Sec. V-A).
//
// One workgroup handles one (tile, sample*channel) plane.  The eight regions
// of the plane (order N, S, W, E, NW, NE, SW, SE) are flattened into one
// index space and each thread gathers all of its elements before storing
// any, so a workgroup pays the memory latency once.  Region geometry is
// computed from the direction with selects on wave-uniform values (no table
// lookups).  Bands along a row put consecutive threads on consecutive
// columns; east/west bands are h-wide column strips.  Copies are bitwise
// (2- or 4-byte elements).  Unpack zero-fills margins that have no
// neighbour: the convolution's zero padding.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace dc {

static constexpr int kHaloThreads = 256;
static constexpr int kUnroll = 4;   // elements in flight per thread

struct Region {
    int d, i;          // region index and element index inside the region's plane block
    int di, dj;        // direction of the neighbour
    int rows, cols;
    int prefix;        // elements of the regions before d, per plane
};

__device__ __forceinline__ Region locate(int e, int Ht, int Wt, int h) {
    const int nNS = h * Wt, nWE = Ht * h, nC = h * h;
    // prefix sums of the per-plane region sizes
    const int p1 = nNS, p2 = 2 * nNS, p3 = p2 + nWE, p4 = p3 + nWE;
    Region r;
    r.d = e < p2 ? (e < p1 ? 0 : 1) : e < p4 ? (e < p3 ? 2 : 3) : 4 + (e - p4) / nC;
    const int d = r.d;
    r.prefix = d == 0 ? 0 : d == 1 ? p1 : d == 2 ? p2 : d == 3 ? p3 : p4 + (d - 4) * nC;
    r.i = e - r.prefix;
    r.di = (d == 0 || d == 4 || d == 5) ? -1 : (d == 1 || d == 6 || d == 7) ? 1 : 0;
    r.dj = (d == 2 || d == 4 || d == 6) ? -1 : (d == 3 || d == 5 || d == 7) ? 1 : 0;
    r.rows = r.di == 0 ? Ht : h;
    r.cols = r.dj == 0 ? Wt : h;
    return r;
}

__device__ __forceinline__ int opposite(int d) { return d < 4 ? (d ^ 1) : 11 - d; }

__device__ __forceinline__ int region_prefix(int d, int Ht, int Wt, int h) {
    const int nNS = h * Wt, nWE = Ht * h, nC = h * h;
    return d == 0 ? 0 : d == 1 ? nNS : d == 2 ? 2 * nNS : d == 3 ? 2 * nNS + nWE
                                                                  : 2 * nNS + 2 * nWE + (d - 4) * nC;
}

template <typename T>
__global__ __launch_bounds__(kHaloThreads) void halo_pack_kernel(HaloArgs a) {
    const int plane = blockIdx.x;
    const int t = a.tile0 + blockIdx.y;          // tile index in the grid
    const int slot = a.all_tiles ? t : 0;        // buffer index: single-tile calls pass one buffer
    const int ti = t / a.Q, tj = t % a.Q;
    const int Ht = a.ht, Wt = a.wt, h = a.h;
    const T* __restrict__ src = static_cast<const T*>(a.src) + int64_t(slot) * a.tile_elems +
                                int64_t(plane) * a.rows * a.pitch;
    T* __restrict__ dst = static_cast<T*>(a.dst) + int64_t(slot) * a.halo_elems;
    const int total = 2 * h * (Ht + Wt) + 4 * h * h;
    for (int base = 0; base < total; base += kHaloThreads * kUnroll) {
        T v[kUnroll];
        int64_t at[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int e = base + u * kHaloThreads + threadIdx.x;
            at[u] = -1;
            if (e < total) {
                const Region r = locate(e, Ht, Wt, h);
                const int ni = ti + r.di, nj = tj + r.dj;
                if (ni >= 0 && ni < a.P && nj >= 0 && nj < a.Q) {   // else: nothing sent
                    const int rr = r.i / r.cols, cc = r.i - rr * r.cols;
                    // band of the owned block next to the neighbour
                    const int tr0 = r.di > 0 ? Ht : h, tc0 = r.dj > 0 ? Wt : h;
                    v[u] = src[(tr0 + rr) * a.pitch + tc0 + cc];
                    at[u] = int64_t(a.planes) * r.prefix + int64_t(plane) * r.rows * r.cols + r.i;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (at[u] >= 0) dst[at[u]] = v[u];
    }
}

template <typename T>
__global__ __launch_bounds__(kHaloThreads) void halo_unpack_kernel(HaloArgs a) {
    const int plane = blockIdx.x;
    const int t = a.tile0 + blockIdx.y;          // tile index in the grid
    const int slot = a.all_tiles ? t : 0;        // buffer index: single-tile calls pass one buffer
    const int ti = t / a.Q, tj = t % a.Q;
    const int Ht = a.ht, Wt = a.wt, h = a.h;
    T* __restrict__ dst = static_cast<T*>(a.dst) + int64_t(slot) * a.tile_elems +
                          int64_t(plane) * a.rows * a.pitch;
    const T* __restrict__ src = static_cast<const T*>(a.src);
    const int total = 2 * h * (Ht + Wt) + 4 * h * h;
    for (int base = 0; base < total; base += kHaloThreads * kUnroll) {
        T v[kUnroll];
        int at[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int e = base + u * kHaloThreads + threadIdx.x;
            at[u] = -1;
            v[u] = T(0);   // no neighbour: zero padding
            if (e < total) {
                const Region r = locate(e, Ht, Wt, h);
                const int rr = r.i / r.cols, cc = r.i - rr * r.cols;
                // margin on side d
                const int tr0 = r.di < 0 ? 0 : r.di > 0 ? h + Ht : h;
                const int tc0 = r.dj < 0 ? 0 : r.dj > 0 ? h + Wt : h;
                at[u] = (tr0 + rr) * a.pitch + tc0 + cc;
                const int ni = ti + r.di, nj = tj + r.dj;
                if (ni >= 0 && ni < a.P && nj >= 0 && nj < a.Q) {
                    const int64_t inplane = int64_t(plane) * r.rows * r.cols + r.i;
                    // all tiles: the neighbour's send buffer, its region facing this tile;
                    // one tile: this tile's receive buffer, region d
                    const int64_t off =
                        a.all_tiles ? int64_t(ni * a.Q + nj) * a.halo_elems +
                                          int64_t(a.planes) * region_prefix(opposite(r.d), Ht, Wt, h) + inplane
                                    : int64_t(a.planes) * r.prefix + inplane;
                    v[u] = src[off];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (at[u] >= 0) dst[at[u]] = v[u];
    }
}

hipError_t launch_halo_pack(const HaloArgs& a, int esize, hipStream_t s) {
    dim3 grid(a.planes, a.ntiles), block(kHaloThreads);
    if (esize == 2)
        hipLaunchKernelGGL(halo_pack_kernel<uint16_t>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(halo_pack_kernel<uint32_t>, grid, block, 0, s, a);
    return hipGetLastError();
}

hipError_t launch_halo_unpack(const HaloArgs& a, int esize, hipStream_t s) {
    dim3 grid(a.planes, a.ntiles), block(kHaloThreads);
    if (esize == 2)
        hipLaunchKernelGGL(halo_unpack_kernel<uint16_t>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(halo_unpack_kernel<uint32_t>, grid, block, 0, s, a);
    return hipGetLastError();
}

}  // namespace dc
