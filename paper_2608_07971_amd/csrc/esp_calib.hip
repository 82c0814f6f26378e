// Streaming-ceiling probe of the structure-of-arrays table layout: a
// measurement kernel, not part of the method.  It reads a table laid out as
// the packer lays out one cluster (ncol fp32 columns of `tiles` 256-entry
// tiles, col_len floats apart) with exactly the access pattern of the fused
// dense kernel's one-pass launch: a workgroup of 4 wavefronts per block,
// tiles grid-strided over the wavefronts, one 128-bit non-temporal load per
// lane per column per tile, three tiles in registers (two in flight while one
// is consumed), loads past the end clamped to the last tile.  Its only work
// per tile is one fp32 add per loaded value, so a launch takes as long as
// streaming the table takes: the ceiling the fused kernel's pass time is
// compared with.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/esp_calib.h"

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
constexpr int kTile = 256;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

template <int NCOL>
__global__ __launch_bounds__(kThreads) void k_stream_probe(const float *col, size_t col_len, int tiles, float *sink) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int stride = gridDim.x * kWaves;
    const int tile0 = blockIdx.x * kWaves + wave;
    const int last = tiles - 1;
    const size_t lane_off = static_cast<size_t>(lane) * 4;
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    auto load = [&](int t, f4 (&v)[NCOL]) {
        const float *p = col + static_cast<size_t>(t) * kTile + lane_off;
#pragma unroll
        for (int c = 0; c < NCOL; ++c)
            v[c] = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p + c * col_len));
    };
    auto use = [&](const f4 (&v)[NCOL]) {
#pragma unroll
        for (int c = 0; c < NCOL; ++c) acc += v[c];
    };
    f4 a[NCOL], b[NCOL], c[NCOL];
    load(min(tile0, last), a);
    load(min(tile0 + stride, last), b);
    for (int t = tile0; t < tiles; t += 3 * stride) {
        const int t1 = t + stride, t2 = t + 2 * stride;
        load(min(t2, last), c);
        use(a);
        load(min(t2 + stride, last), a);
        if (t1 < tiles) use(b);
        load(min(t2 + 2 * stride, last), b);
        if (t2 < tiles) use(c);
    }
    sink[static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

template <int NCOL>
hipError_t launch(const float *col, size_t col_len, int tiles, int blocks, float *sink, hipStream_t s) {
    hipLaunchKernelGGL((k_stream_probe<NCOL>), dim3(blocks), dim3(kThreads), 0, s, col, col_len, tiles, sink);
    return hipGetLastError();
}

}  // namespace

extern "C" int esp_calib_stream(const float *table, int ncol, size_t col_len, int tiles, int blocks, float *sink,
                                void *stream) {
    if (table == nullptr || sink == nullptr || tiles < 1 || blocks < 1 ||
        col_len < static_cast<size_t>(tiles) * kTile)
        return 1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    switch (ncol) {
        case 1: e = launch<1>(table, col_len, tiles, blocks, sink, s); break;
        case 2: e = launch<2>(table, col_len, tiles, blocks, sink, s); break;
        case 3: e = launch<3>(table, col_len, tiles, blocks, sink, s); break;
        case 4: e = launch<4>(table, col_len, tiles, blocks, sink, s); break;
        case 5: e = launch<5>(table, col_len, tiles, blocks, sink, s); break;
        case 6: e = launch<6>(table, col_len, tiles, blocks, sink, s); break;
        case 7: e = launch<7>(table, col_len, tiles, blocks, sink, s); break;
        case 8: e = launch<8>(table, col_len, tiles, blocks, sink, s); break;
        case 9: e = launch<9>(table, col_len, tiles, blocks, sink, s); break;
        case 10: e = launch<10>(table, col_len, tiles, blocks, sink, s); break;
        default: return 1;
    }
    return e == hipSuccess ? 0 : 8;
}
