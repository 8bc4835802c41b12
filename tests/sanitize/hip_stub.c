/*
 * A stand-in for the HIP runtime, for a CPU build of libdc's host code under
 * AddressSanitizer / UndefinedBehaviorSanitizer (no GPU involved).  Kernel
 * registration does nothing; a launch only checks its configuration (grid
 * and block extents, dynamic LDS) and counts; device queries answer as an
 * MI355X would.  Linked only into the test driver, never into the library.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct { uint32_t x, y, z; } dim3;
typedef void* hipStream_t;

static dim3 cfg_grid, cfg_block;
static size_t cfg_shmem;
static hipStream_t cfg_stream;
long stub_launches = 0;

void** __hipRegisterFatBinary(const void* data) { (void)data; static void* h; return &h; }
void __hipUnregisterFatBinary(void** m) { (void)m; }
void __hipRegisterFunction(void** m, const void* host, char* dev, const char* name, unsigned limit,
                           void* tid, void* bid, void* bdim, void* gdim, int* wsize)
{ (void)m; (void)host; (void)dev; (void)name; (void)limit; (void)tid; (void)bid; (void)bdim; (void)gdim; (void)wsize; }
void __hipRegisterVar(void** m, void* var, char* hv, char* dv, int ext, size_t size, int cnst, int glob)
{ (void)m; (void)var; (void)hv; (void)dv; (void)ext; (void)size; (void)cnst; (void)glob; }

int __hipPushCallConfiguration(dim3 g, dim3 b, size_t shmem, hipStream_t s)
{ cfg_grid = g; cfg_block = b; cfg_shmem = shmem; cfg_stream = s; return 0; }
int __hipPopCallConfiguration(dim3* g, dim3* b, size_t* shmem, hipStream_t* s)
{ *g = cfg_grid; *b = cfg_block; *shmem = cfg_shmem; *s = cfg_stream; return 0; }

int hipLaunchKernel(const void* f, dim3 g, dim3 b, void** args, size_t shmem, hipStream_t s)
{
    (void)f; (void)args; (void)s;
    const uint64_t threads = (uint64_t)b.x * b.y * b.z;
    if (g.x < 1 || g.y < 1 || g.z < 1 || g.y > 65535 || g.z > 65535 || threads < 1 || threads > 1024 ||
        (uint64_t)g.x * threads > 0xffffffffull || shmem > 160 * 1024) {
        fprintf(stderr, "bad launch: grid %u %u %u block %u %u %u lds %zu\n", g.x, g.y, g.z, b.x, b.y, b.z, shmem);
        abort();
    }
    ++stub_launches;
    return 0;
}

int hipGetDevice(int* d) { *d = 0; return 0; }
int hipDeviceGetAttribute(int* v, int attr, int dev) { (void)attr; (void)dev; *v = 160 * 1024; return 0; }
int hipFuncSetAttribute(const void* f, int attr, int v) { (void)f; (void)attr; (void)v; return 0; }
int hipGetLastError(void) { return 0; }
int hipGetSymbolAddress(void** p, const void* sym) { *p = (void*)sym; return 0; }
