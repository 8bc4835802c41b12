// Halo pack / unpack kernels (Sec. III-A; message terms of Sec. V-A).
//
// One workgroup handles one (tile, sample*channel) plane and all eight
// regions of it.  North/south bands and corners are row segments, copied with
// consecutive lanes on consecutive columns; east/west bands are h-wide column
// strips, one lane per element with rows spread over the wave.  Copies are
// bitwise (2- or 4-byte elements).  Unpack zero-fills margins that have no
// neighbour: the convolution's zero padding.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace dc {

static constexpr int kHaloThreads = 256;

template <typename T>
__global__ __launch_bounds__(kHaloThreads) void halo_pack_kernel(HaloArgs a) {
    const int plane = blockIdx.x;
    const int t = a.tile0 + blockIdx.y;          // tile index in the grid
    const int slot = a.all_tiles ? t : 0;        // buffer index: single-tile calls pass one buffer
    const int ti = t / a.Q, tj = t % a.Q;
    const T* src = static_cast<const T*>(a.src) + int64_t(slot) * a.tile_elems +
                   int64_t(plane) * a.rows * a.pitch;
    T* dst = static_cast<T*>(a.dst) + int64_t(slot) * a.halo_elems;
#pragma unroll 1
    for (int d = 0; d < 8; ++d) {
        const HaloRegion& r = a.reg[d];
        const int ni = ti + r.di, nj = tj + r.dj;
        if (ni < 0 || ni >= a.P || nj < 0 || nj >= a.Q) continue;  // no neighbour: nothing sent
        const int n = r.rows * r.cols;
        T* out = dst + r.off + int64_t(plane) * n;
        for (int e = threadIdx.x; e < n; e += kHaloThreads) {
            const int rr = e / r.cols, cc = e - rr * r.cols;
            out[e] = src[(r.tr0 + rr) * a.pitch + r.tc0 + cc];
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kHaloThreads) void halo_unpack_kernel(HaloArgs a) {
    const int plane = blockIdx.x;
    const int t = a.tile0 + blockIdx.y;          // tile index in the grid
    const int slot = a.all_tiles ? t : 0;        // buffer index: single-tile calls pass one buffer
    const int ti = t / a.Q, tj = t % a.Q;
    T* dst = static_cast<T*>(a.dst) + int64_t(slot) * a.tile_elems +
             int64_t(plane) * a.rows * a.pitch;
#pragma unroll 1
    for (int d = 0; d < 8; ++d) {
        const HaloRegion& r = a.reg[d];
        const int ni = ti + r.di, nj = tj + r.dj;
        const bool exists = ni >= 0 && ni < a.P && nj >= 0 && nj < a.Q;
        const int n = r.rows * r.cols;
        const T* in = nullptr;
        if (exists) {
            if (a.all_tiles) {
                // the neighbour's send buffer, its region facing this tile
                const int nb = ni * a.Q + nj;
                in = static_cast<const T*>(a.src) + int64_t(nb) * a.halo_elems +
                     a.reg[r.opp].off + int64_t(plane) * n;
            } else {
                in = static_cast<const T*>(a.src) + r.off + int64_t(plane) * n;
            }
        }
        for (int e = threadIdx.x; e < n; e += kHaloThreads) {
            const int rr = e / r.cols, cc = e - rr * r.cols;
            dst[(r.tr0 + rr) * a.pitch + r.tc0 + cc] = exists ? in[e] : T(0);
        }
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
