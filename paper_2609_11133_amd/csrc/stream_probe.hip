// HBM streaming reference for the roofline: how fast this GPU reads (and copies)
// large buffers with the access shapes the expert kernels use.  Not part of the
// library; built as a separate executable and used by the measurement scripts.
//
//   stream_probe <mode> <MiB> <iters>
//   modes: read      grid-stride 16-byte loads over a contiguous buffer
//          read_nt   the same with non-temporal loads
//          tiles     16-row x 128-byte tiles of 4096-byte rows, each lane two 16-byte
//                    pieces (the FP8 MFMA operand shape), rows streamed in K order
//          tiles_nt  the same with non-temporal loads
//          deep_nt   contiguous, each workgroup sixteen 4 KB pieces in flight (16 loads per
//                    lane), non-temporal, 512 workgroups walking the buffer
//          packed_nt 16-row tiles stored as contiguous 2 KB K blocks (the packed weight
//                    layout): each lane 16 bytes at 16l and 1024 + 16l of a block, eight
//                    blocks in flight, non-temporal
//          copy      contiguous 16-byte copy (reads and writes MiB each)
//          tilestream <MiB> <iters> <tile KiB> <depth>
//                    one launch streams MiB as packed tiles of <tile KiB> per wave (2 KB
//                    blocks, <depth> of them in flight per wave, 4 or 8), non-temporal;
//                    successive launches read different regions of a 4 GiB arena, so no
//                    launch finds its bytes in the MALL: the time of one cold launch of that
//                    shape, ramp and tail included
//          chain <iters>
//                    the launch floor of one decode step: four empty kernels back to back
//                    in the grid shapes of the 235B-shaped layer's step at one token
//                    (routing 32, gate/up 432, down 288, combine 4 workgroups of 256)
// Prints one line: mode, bytes moved per launch, mean ms, GB/s.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ inline u32x4 ld(const u32x4 *p)
{
    if constexpr (NT)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}

template <bool NT>
__global__ __launch_bounds__(256) void read_kernel(const u32x4 *__restrict__ a, size_t n, uint32_t *__restrict__ sink)
{
    u32x4 acc = {0, 0, 0, 0};
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const u32x4 v0 = ld<NT>(a + i), v1 = ld<NT>(a + i + stride), v2 = ld<NT>(a + i + 2 * stride),
                    v3 = ld<NT>(a + i + 3 * stride);
        acc ^= v0 ^ v1 ^ v2 ^ v3;
    }
    for (; i < n; i += stride) acc ^= ld<NT>(a + i);
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[0] = 1;  // keeps the loads alive
}

// Each wave streams one tile of 16 rows (row length 4096 bytes) in 128-byte K blocks.
template <bool NT>
__global__ __launch_bounds__(256) void tiles_kernel(const uint8_t *__restrict__ a, size_t n_tiles,
                                                    uint32_t *__restrict__ sink)
{
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
    u32x4 acc = {0, 0, 0, 0};
    for (size_t t = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < n_tiles; t += (size_t)gridDim.x * 4) {
        const uint8_t *row = a + t * 16 * 4096 + (size_t)r * 4096;
#pragma unroll 4
        for (int kb = 0; kb < 32; ++kb) {
            acc ^= ld<NT>(reinterpret_cast<const u32x4 *>(row + kb * 128 + 16 * g));
            acc ^= ld<NT>(reinterpret_cast<const u32x4 *>(row + kb * 128 + 64 + 16 * g));
        }
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[0] = 1;
}

// Workgroup b of G takes pieces b, b+G, ... of U*256 16-byte elements, all U loads of
// a piece in flight together.
template <int U>
__global__ __launch_bounds__(256) void deep_kernel(const u32x4 *__restrict__ a, size_t n, uint32_t *__restrict__ sink)
{
    const size_t per = (size_t)U * 256, pieces = n / per;
    u32x4 acc = {0, 0, 0, 0};
    for (size_t pc = blockIdx.x; pc < pieces; pc += gridDim.x) {
        const u32x4 *q = a + pc * per + threadIdx.x;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = ld<true>(q + 256 * u);
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u];
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[0] = 1;
}

// Each wave streams one packed tile (64 KB: 32 K blocks of 2 KB), eight blocks in flight.
__global__ __launch_bounds__(256) void packed_kernel(const uint8_t *__restrict__ a, size_t n_tiles,
                                                     uint32_t *__restrict__ sink)
{
    const int lane = threadIdx.x & 63;
    u32x4 acc = {0, 0, 0, 0};
    for (size_t t = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < n_tiles; t += (size_t)gridDim.x * 4) {
        const uint8_t *tile = a + t * 16 * 4096 + 16 * lane;
        for (int kb0 = 0; kb0 < 32; kb0 += 8) {
            u32x4 v[8][2];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                v[u][0] = ld<true>(reinterpret_cast<const u32x4 *>(tile + (kb0 + u) * 2048));
                v[u][1] = ld<true>(reinterpret_cast<const u32x4 *>(tile + (kb0 + u) * 2048 + 1024));
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) acc ^= v[u][0] ^ v[u][1];
        }
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[0] = 1;
}

// Wave w streams tile w (tile_blocks 2 KB blocks at 2048 * tile_blocks * w), lane l
// reading 16 bytes at 16l and 1024 + 16l of each block, D blocks in flight.
template <int D>
__global__ __launch_bounds__(256) void tilestream_kernel(const uint8_t *__restrict__ a, int tile_blocks,
                                                         uint32_t *__restrict__ sink)
{
    const int lane = threadIdx.x & 63;
    const size_t wave = (size_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const uint8_t *tile = a + wave * (size_t)tile_blocks * 2048 + 16 * lane;
    u32x4 acc = {0, 0, 0, 0};
    u32x4 v[D][2];
#pragma unroll
    for (int u = 0; u < D - 1; ++u) {
        v[u][0] = ld<true>(reinterpret_cast<const u32x4 *>(tile + u * 2048));
        v[u][1] = ld<true>(reinterpret_cast<const u32x4 *>(tile + u * 2048 + 1024));
    }
    for (int kb = 0; kb < tile_blocks; kb += D) {  // tile_blocks is a multiple of D
#pragma unroll
        for (int u = 0; u < D; ++u) {
            const int nb = kb + u + D - 1;  // block loaded now; past the tile: reload the last one
            const int b = nb < tile_blocks ? nb : tile_blocks - 1;
            v[(u + D - 1) % D][0] = ld<true>(reinterpret_cast<const u32x4 *>(tile + (size_t)b * 2048));
            v[(u + D - 1) % D][1] = ld<true>(reinterpret_cast<const u32x4 *>(tile + (size_t)b * 2048 + 1024));
            acc ^= v[u][0] ^ v[u][1];
        }
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9E3779B9u) sink[0] = 1;
}

__global__ void empty_kernel(uint32_t *__restrict__ sink, int never)
{
    if (never == 1) sink[0] = 1;
}

__global__ __launch_bounds__(256) void copy_kernel(const u32x4 *__restrict__ a, u32x4 *__restrict__ b, size_t n)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) b[i] = a[i];
}

#define CHECK(x)                                                                             \
    do {                                                                                     \
        hipError_t e = (x);                                                                  \
        if (e != hipSuccess) {                                                               \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e));                           \
            exit(1);                                                                         \
        }                                                                                    \
    } while (0)

static int run_tilestream(size_t bytes, int iters, int tile_kib, int depth)
{
    if (tile_kib < 2 || tile_kib % 2 || (depth != 4 && depth != 8) || (tile_kib / 2) % depth ||
        bytes % ((size_t)tile_kib * 1024 * 4)) {
        fprintf(stderr, "tilestream: tile KiB even, (tile KiB / 2) a multiple of depth (4 or 8), MiB a "
                        "multiple of 4 tiles\n");
        return 2;
    }
    const size_t arena = (size_t)4 << 30;
    if (bytes > arena / 4) {
        fprintf(stderr, "tilestream: at most 1 GiB per launch\n");
        return 2;
    }
    const int regions = (int)(arena / bytes);
    uint8_t *a = nullptr;
    uint32_t *sink = nullptr;
    CHECK(hipMalloc(&a, arena));
    CHECK(hipMalloc(&sink, 4));
    CHECK(hipMemset(a, 1, arena));
    const int tile_blocks = tile_kib / 2;
    const int grid = (int)(bytes / ((size_t)tile_kib * 1024) / 4);
    auto launch = [&](int i) {
        const uint8_t *p = a + (size_t)(i % regions) * bytes;
        if (depth == 4)
            tilestream_kernel<4><<<grid, 256>>>(p, tile_blocks, sink);
        else
            tilestream_kernel<8><<<grid, 256>>>(p, tile_blocks, sink);
        CHECK(hipGetLastError());
    };
    for (int i = 0; i < regions; ++i) launch(i);
    CHECK(hipDeviceSynchronize());
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    float total = 0.f;
    for (int i = 0; i < iters; ++i) {  // one launch between two events, each launch cold
        CHECK(hipEventRecord(e0, 0));
        launch(i);
        CHECK(hipEventRecord(e1, 0));
        CHECK(hipEventSynchronize(e1));
        float ms = 0.f;
        CHECK(hipEventElapsedTime(&ms, e0, e1));
        total += ms;
    }
    const float ms = total / iters;
    printf("tilestream bytes=%zu tile_kib=%d depth=%d waves=%zu ms=%.4f GBps=%.1f\n", bytes, tile_kib, depth,
           bytes / ((size_t)tile_kib * 1024), ms, bytes / (ms * 1e-3) / 1e9);
    CHECK(hipFree(a));
    CHECK(hipFree(sink));
    return 0;
}

static int run_chain(int iters)
{
    uint32_t *sink = nullptr;
    CHECK(hipMalloc(&sink, 4));
    const int grids[4] = {32, 432, 288, 4};
    auto step = [&]() {
        for (int g : grids) empty_kernel<<<g, 256>>>(sink, 0);
        CHECK(hipGetLastError());
    };
    for (int i = 0; i < 10; ++i) step();
    CHECK(hipDeviceSynchronize());
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    CHECK(hipEventRecord(e0, 0));
    for (int i = 0; i < iters; ++i) step();
    CHECK(hipEventRecord(e1, 0));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    printf("chain kernels=4 us_per_step=%.2f us_per_launch=%.2f\n", ms * 1e3 / iters, ms * 1e3 / iters / 4);
    CHECK(hipFree(sink));
    return 0;
}

int main(int argc, char **argv)
{
    if (argc >= 3 && !strcmp(argv[1], "chain")) return run_chain(atoi(argv[2]) > 0 ? atoi(argv[2]) : 1000);
    if (argc >= 6 && !strcmp(argv[1], "tilestream"))
        return run_tilestream((size_t)atol(argv[2]) << 20, atoi(argv[3]) > 0 ? atoi(argv[3]) : 1, atoi(argv[4]),
                              atoi(argv[5]));
    if (argc < 4) {
        fprintf(stderr, "usage: %s read|read_nt|tiles|tiles_nt|deep_nt|packed_nt|copy MiB iters\n", argv[0]);
        return 2;
    }
    const char *mode = argv[1];
    const size_t bytes = (size_t)atol(argv[2]) << 20;
    const int iters = atoi(argv[3]);
    if (bytes == 0 || bytes % (16 * 4096) != 0 || iters < 1) {
        fprintf(stderr, "MiB must be positive (multiple of 64 KiB) and iters >= 1\n");
        return 2;
    }
    int cus = 0;
    CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
    uint8_t *a = nullptr, *b = nullptr;
    uint32_t *sink = nullptr;
    CHECK(hipMalloc(&a, bytes));
    CHECK(hipMalloc(&sink, 4));
    CHECK(hipMemset(a, 1, bytes));
    const bool copy = strcmp(mode, "copy") == 0;
    if (copy) CHECK(hipMalloc(&b, bytes));
    const size_t n16 = bytes / 16, n_tiles = bytes / (16 * 4096);
    const int grid = cus * 8;
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    auto launch = [&]() {
        if (!strcmp(mode, "read"))
            read_kernel<false><<<grid, 256>>>((const u32x4 *)a, n16, sink);
        else if (!strcmp(mode, "read_nt"))
            read_kernel<true><<<grid, 256>>>((const u32x4 *)a, n16, sink);
        else if (!strcmp(mode, "tiles"))
            tiles_kernel<false><<<grid, 256>>>(a, n_tiles, sink);
        else if (!strcmp(mode, "tiles_nt"))
            tiles_kernel<true><<<grid, 256>>>(a, n_tiles, sink);
        else if (!strcmp(mode, "deep_nt"))
            deep_kernel<16><<<512, 256>>>((const u32x4 *)a, n16, sink);
        else if (!strcmp(mode, "packed_nt"))
            packed_kernel<<<cus * 4, 256>>>(a, n_tiles, sink);
        else if (copy)
            copy_kernel<<<grid, 256>>>((const u32x4 *)a, (u32x4 *)b, n16);
        else {
            fprintf(stderr, "unknown mode %s\n", mode);
            exit(2);
        }
        CHECK(hipGetLastError());
    };
    launch();
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(e0, 0));
    for (int i = 0; i < iters; ++i) launch();
    CHECK(hipEventRecord(e1, 0));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    ms /= iters;
    const double moved = copy ? 2.0 * bytes : (double)bytes;
    printf("%s bytes=%zu ms=%.4f GBps=%.1f\n", mode, (size_t)moved, ms, moved / (ms * 1e-3) / 1e9);
    CHECK(hipFree(a));
    if (b) CHECK(hipFree(b));
    CHECK(hipFree(sink));
    return 0;
}
