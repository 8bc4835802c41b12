/*
 * Drives every entry point of libdc's C ABI over a few thousand seeded
 * random problems (valid or not), tile indices, regions and band masks, with
 * fake 16-byte-aligned device addresses: the host code (validation, tile
 * geometry, halo bands, plans, sample groups, launch configuration) runs
 * under AddressSanitizer / UndefinedBehaviorSanitizer against the stub
 * runtime of hip_stub.c, which checks each launch's configuration.  Exit 0 if
 * no sanitizer or launch check fired.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "dc.h"

extern long stub_launches;

static uint64_t rs = 0x9e3779b97f4a7c15ull;
static int rnd(int n) { rs ^= rs << 13; rs ^= rs >> 7; rs ^= rs << 17; return (int)(rs % (uint64_t)n); }
static int pick(const int* v, int n) { return v[rnd(n)]; }

int main(void)
{
    static const int Ns[] = {1, 2, 3, 4, 32};
    static const int Cs[] = {1, 3, 5, 8, 16, 18, 32, 48, 64, 96, 256};
    static const int Hs[] = {1, 7, 8, 16, 26, 31, 32, 56, 64, 96, 130, 224, 256, 1024};
    static const int Rs[] = {1, 2, 3, 4, 5, 7, 9};
    static const int Gs[] = {1, 1, 2, 3, 4};
    void* X = (void*)(uintptr_t)0x100000, * Wt = (void*)(uintptr_t)0x200000;
    float* Y = (float*)(uintptr_t)0x300000;
    void* WS = (void*)(uintptr_t)0x400000;
    long valid = 0, calls = 0;
    for (int it = 0; it < 4000; ++it) {
        dc_problem p;
        p.N = pick(Ns, 5); p.C = pick(Cs, 11); p.K = pick(Cs, 11);
        p.H = pick(Hs, 14); p.W = rnd(3) ? p.H : pick(Hs, 14);
        p.R = pick(Rs, 7); p.S = rnd(4) ? p.R : pick(Rs, 7);
        p.stride = 1 + rnd(3); p.pad = rnd(4);
        p.P = pick(Gs, 5); p.Q = pick(Gs, 5); p.halo = rnd(5);
        p.dtype = rnd(2);
        if (it % 2 == 1) {   /* a valid decomposed layer: odd filter, 'same' padding, even tiles */
            p.R = p.S = 1 + 2 * rnd(3); p.pad = p.R / 2; p.halo = p.pad + rnd(2);
            p.stride = 1 + (p.R > 1 && rnd(3) == 0);
            p.H = p.P * p.stride * (p.halo + 1 + rnd(40)); p.W = p.Q * p.stride * (p.halo + 1 + rnd(40));
            if (p.stride == 2 && (p.R == 1 || (p.H + 2 * p.pad - p.R) / 2 + 1 != p.H / 2)) p.stride = 1;
        }
        if (it % 50 == 0) { p.N = 32; p.C = p.K = 64; p.H = p.W = 1024; p.R = p.S = 3; p.stride = 1; p.pad = 1;
                            p.P = p.Q = 1; p.halo = 1; p.dtype = DC_BF16; }   /* sample groups */
        if (it % 97 == 0) { p.N = -rnd(2); }                                  /* invalid sizes */
        const int ntiles = p.P * p.Q;
        for (int t = -2; t <= (ntiles > 0 ? ntiles : 1); ++t) {
            const int tile = t == -2 ? DC_ALL_TILES : t;
            dc_status v = dc_validate(&p, tile);
            int32_t lohi[2], bw[4], dims[4];
            (void)dc_required_halo(&p, DC_X, lohi);
            (void)dc_required_halo(&p, DC_DY, lohi);
            (void)dc_halo_bands(&p, rnd(3), bw);
            (void)dc_tile_dims(&p, dims);
            (void)dc_tile_pitch(&p, DC_X);
            (void)dc_tile_elems(&p, DC_DY);
            (void)dc_halo_elems(&p, DC_X);
            size_t ws = dc_bwd_filter_workspace_bytes(&p, tile);
            (void)dc_status_string(v);
            calls += 9;
            if (v == DC_OK) ++valid;
            (void)dc_conv_fwd(&p, tile, X, Wt, Y, NULL);
            (void)dc_conv_bwd_data(&p, tile, X, Wt, Y, NULL);
            (void)dc_conv_bwd_filter(&p, tile, X, X, Y, rnd(2), WS, ws, NULL);
            (void)dc_conv_bwd_filter_noalloc(&p, tile, X, X, Y, rnd(2), NULL);
            (void)dc_conv_fwd_region(&p, tile, rnd(4), X, Wt, Y, NULL);
            (void)dc_conv_bwd_data_region(&p, tile, rnd(4), X, Wt, Y, NULL);
            (void)dc_halo_pack(&p, tile, rnd(2), X, WS, NULL);
            (void)dc_halo_unpack(&p, tile, rnd(2), WS, X, NULL);
            (void)dc_halo_pack_bands(&p, tile, rnd(2), rnd(9), X, WS, NULL);
            (void)dc_halo_unpack_bands(&p, tile, rnd(2), rnd(9), WS, X, NULL);
            calls += 10;
        }
    }
    printf("host checks: %ld calls, %ld valid problem/tile pairs, %ld launches\n", calls, valid, stub_launches);
    return valid > 0 && stub_launches > 0 ? 0 : 1;
}
