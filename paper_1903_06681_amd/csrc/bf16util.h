// Small device helpers shared by the bf16 kernels: MFMA operand types,
// 16-byte register packs, and unaligned 8-element row reads built from
// aligned 16-byte loads.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

namespace dc {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

// v_mfma_f32_32x32x16_bf16 written out so that the register class of the A
// operand is chosen here: AG = true reads it from AGPRs (the 512-entry
// register file of a wave holds a weight operand larger than the 256 VGPRs
// that way), ZERO = true starts a new accumulation (C = 0).  The accumulator
// lives in AGPRs.  The hardware interlocks back-to-back MFMAs that accumulate
// into the same registers; any other reader of the accumulator must come after
// mfma_drain(), and an A/B operand must not be written by a VALU instruction
// in the two instructions before the MFMA (A/B here come from loads).  The
// statements are volatile: memory operations keep their source order around
// them, which fixes how far loads run ahead and where stores interleave.
template <bool AG, bool ZERO>
__device__ __forceinline__ void mfma32x32x16(floatx16& acc, const bf16x8& a, const bf16x8& b) {
    if constexpr (ZERO) {
        if constexpr (AG)
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&a"(acc) : "a"(a), "v"(b));
        else
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&a"(acc) : "v"(a), "v"(b));
    } else {
        if constexpr (AG)
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "a"(a), "v"(b));
        else
            asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
    }
}

// Wait states between the last MFMA writing `acc` and any non-MFMA reader of
// it (32 >= passes + 4 for every 32x32 shape).
__device__ __forceinline__ void mfma_drain(floatx16& acc) {
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" : "+a"(acc));
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

union Pack8 {
    uint4 v;
    uint32_t d[4];
    uint16_t h[8];
    bf16x8 b;
};

// Elements [sh, sh+8) of the 16-element window d[0..7] (two aligned 16-byte chunks).
template <int SH>
__device__ __forceinline__ uint4 window8(const uint32_t (&d)[8]) {
    uint4 r;
    uint32_t* o = reinterpret_cast<uint32_t*>(&r);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if ((SH & 1) == 0)
            o[i] = d[SH / 2 + i];
        else
            o[i] = __builtin_amdgcn_alignbyte(d[SH / 2 + i + 1], d[SH / 2 + i], 2);
    }
    return r;
}

__device__ __forceinline__ uint4 window8_rt(const uint32_t (&d)[8], int sh) {
    switch (sh) {
        case 0: return window8<0>(d);
        case 1: return window8<1>(d);
        case 2: return window8<2>(d);
        case 3: return window8<3>(d);
        case 4: return window8<4>(d);
        case 5: return window8<5>(d);
        case 6: return window8<6>(d);
        default: return window8<7>(d);
    }
}

// The same window for a shift known only at run time (0..7, equal on every
// lane), without branches: selects pick the whole dwords, a byte-align the
// odd element.  Straight-line code lets the scheduler interleave it with
// matrix instructions.
__device__ __forceinline__ uint4 window8_sel(const uint32_t (&d)[8], int sh) {
    const int k = sh >> 1;
    const uint32_t bs = uint32_t(sh & 1) * 2u;
    uint32_t w[5];
#pragma unroll
    for (int j = 0; j < 5; ++j) {
        const uint32_t a = k & 1 ? d[j + 1] : d[j];
        const uint32_t b = k & 1 ? d[j + 3] : d[j + 2];
        w[j] = k & 2 ? b : a;
    }
    uint4 r;
    r.x = __builtin_amdgcn_alignbyte(w[1], w[0], bs);
    r.y = __builtin_amdgcn_alignbyte(w[2], w[1], bs);
    r.z = __builtin_amdgcn_alignbyte(w[3], w[2], bs);
    r.w = __builtin_amdgcn_alignbyte(w[4], w[3], bs);
    return r;
}

// 8 consecutive bf16 of a row starting at column g0 + sh, where g0 is a
// multiple of 8 and sh (0..7) is the same for the whole wave; columns outside
// [0, ncols) read as zero.  `row` is 16-byte aligned with `pitch` (a multiple
// of 8, >= ncols) readable elements.  Loads are unconditional 16-byte loads
// from clamped, always-valid addresses; out-of-range data is masked after.
__device__ __forceinline__ uint4 load_row8(const uint16_t* row, int g0, int sh, int ncols,
                                           int pitch, bool row_ok) {
    const int g = g0 + sh;
    const bool ok0 = row_ok && g < ncols;
    uint4 v = *reinterpret_cast<const uint4*>(row + (ok0 ? g0 : 0));
    if (sh != 0) {
        const bool ok1 = ok0 && g0 + 8 < pitch;
        uint4 v1 = *reinterpret_cast<const uint4*>(row + (ok1 ? g0 + 8 : 0));
        if (!ok1) v1 = make_uint4(0, 0, 0, 0);
        const uint32_t d[8] = {v.x, v.y, v.z, v.w, v1.x, v1.y, v1.z, v1.w};
        v = window8_rt(d, sh);
    }
    const int nv = ok0 ? ncols - g : 0;   // valid elements of this group of 8
    uint32_t* w = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t m = (2 * i < nv ? 0x0000ffffu : 0u) | (2 * i + 1 < nv ? 0xffff0000u : 0u);
        w[i] &= m;
    }
    return v;
}

// Keep the first nv (clamped to 0..8) elements of a group of 8, zero the rest.
__device__ __forceinline__ uint4 mask8(uint4 v, int nv) {
    uint32_t* w = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t m = (2 * i < nv ? 0x0000ffffu : 0u) | (2 * i + 1 < nv ? 0xffff0000u : 0u);
        w[i] &= m;
    }
    return v;
}

}  // namespace dc
