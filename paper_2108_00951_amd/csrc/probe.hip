// Streaming bandwidth probes (measurement aids, not part of the method):
// the same tile shape and cache hints as the hard-threshold kernel, so that
// their rates are the ceilings the compression passes are compared with.
// Each launches either the hard threshold's persistent grid (two
// workgroups per CU striding over the tiles, XCD by XCD for long sweeps) or
// one workgroup per 4096-element tile, dispatched in tile order; a plain
// stream runs faster in the second shape, which the compression passes
// cannot take (their one payload atomic per workgroup would then serialise
// on a single address).
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

// Same tile shape, grid sizing and cache hints as the hard-threshold kernel:
// four 16-byte non-temporal loads per thread in flight, then four
// non-temporal stores.
__global__ __launch_bounds__(kBlock) void copy_kernel(const float *__restrict__ src,
                                                      float *__restrict__ dst, int64_t n,
                                                      uint32_t ntiles, bool by_xcd) {
    const int tid = threadIdx.x;
    const TileWalk walk = tile_walk(ntiles, by_xcd);
    for (uint32_t tile = walk.first; tile < walk.end; tile += walk.stride) {
        const int64_t tile0 = int64_t(tile) * kTile;
        if (tile0 + kTile <= n) {
            const f32x4 *s4 = reinterpret_cast<const f32x4 *>(src + tile0);
            f32x4 *d4 = reinterpret_cast<f32x4 *>(dst + tile0);
            f32x4 v[kVecPerThread];
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) v[j] = __builtin_nontemporal_load(s4 + j * kBlock + tid);
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) __builtin_nontemporal_store(v[j], d4 + j * kBlock + tid);
        } else {
            for (int64_t i = tile0 + tid; i < n; i += kBlock) dst[i] = src[i];
        }
    }
}

// Streaming ceilings with the same tile shape and grid: read only (a sum
// whose result is written only if it equals an impossible value), write only
// (a constant fill with default caching, so that it also serves to evict the
// Infinity Cache), and two reads plus one write in place (y = y + 0.5 x, the
// access pattern and cache hints of the error-feedback passes).
template <int kMode>
__global__ __launch_bounds__(kBlock) void stream_probe_kernel(const float *__restrict__ x,
                                                              float *__restrict__ y, int64_t n,
                                                              uint32_t ntiles, bool by_xcd) {
    const int tid = threadIdx.x;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    const TileWalk walk = tile_walk(ntiles, by_xcd);
    for (uint32_t tile = walk.first; tile < walk.end; tile += walk.stride) {
        const int64_t tile0 = int64_t(tile) * kTile;
        if (tile0 + kTile > n) continue;  // the probe covers whole tiles only
        const f32x4 *x4 = reinterpret_cast<const f32x4 *>(x + tile0);
        f32x4 *y4 = reinterpret_cast<f32x4 *>(y + tile0);
        if (kMode == 1) {
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) acc += __builtin_nontemporal_load(x4 + j * kBlock + tid);
        } else if (kMode == 2) {
            const f32x4 c = {1.0f, 2.0f, 3.0f, 4.0f};
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) y4[j * kBlock + tid] = c;
        } else {
            f32x4 a[kVecPerThread], b[kVecPerThread];
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
                a[j] = __builtin_nontemporal_load(x4 + j * kBlock + tid);
                b[j] = __builtin_nontemporal_load(y4 + j * kBlock + tid);
            }
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j)
                __builtin_nontemporal_store(b[j] + 0.5f * a[j], y4 + j * kBlock + tid);
        }
    }
    if (kMode == 1 && acc.x == -1234.5f) y[tid] = acc.y;
}

}  // namespace

// The persistent grid of the hard threshold (with its XCD-by-XCD walk of
// long sweeps), or one workgroup per tile.
struct ProbeGrid {
    uint32_t grid;
    bool by_xcd;
};

ProbeGrid probe_grid(int64_t tiles, bool per_tile) {
    if (per_tile) return ProbeGrid{uint32_t(tiles), false};
    const uint32_t grid = balanced_grid(tiles, kHtWorkgroupsPerCU);
    return ProbeGrid{grid, tiles >= int64_t(kXcdWalkMinTiles) * grid};
}

hipError_t launch_stream_probe(const float *x, float *y, int64_t n, int mode, bool per_tile,
                               hipStream_t stream) {
    const int64_t tiles = n > 0 ? (n + kTile - 1) / kTile : 1;
    const ProbeGrid pg = probe_grid(tiles, per_tile);
    const uint32_t nt = uint32_t(tiles);
    if (mode == 1)
        stream_probe_kernel<1><<<pg.grid, kBlock, 0, stream>>>(x, y, n, nt, pg.by_xcd);
    else if (mode == 2)
        stream_probe_kernel<2><<<pg.grid, kBlock, 0, stream>>>(x, y, n, nt, pg.by_xcd);
    else
        stream_probe_kernel<3><<<pg.grid, kBlock, 0, stream>>>(x, y, n, nt, pg.by_xcd);
    return hipGetLastError();
}

hipError_t launch_copy(const float *src, float *dst, int64_t n, bool per_tile,
                       hipStream_t stream) {
    const int64_t tiles = n > 0 ? (n + kTile - 1) / kTile : 1;
    const ProbeGrid pg = probe_grid(tiles, per_tile);
    copy_kernel<<<pg.grid, kBlock, 0, stream>>>(src, dst, n, uint32_t(tiles), pg.by_xcd);
    return hipGetLastError();
}

}  // namespace efs
