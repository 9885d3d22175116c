// Exchange-and-average of n workers' sparse payloads on one device
// (Algorithm 1: the average (1/n) sum_i Delta_i of the compressed updates).
//
//   zero     out = +0 (16-byte stores)
//   scatter  one launch per worker, in worker order: out[i] += v for every
//            (i, v) of that payload.  Indices are distinct within a payload,
//            so no two lanes of one launch touch the same coordinate and no
//            atomics are needed; stream order between launches fixes the
//            summation order, so the result is the same on every run.  The
//            first launch knows out[i] is +0 and stores +0 + v without
//            reading it.
//   scale    out = out / n (IEEE division), skipped for n == 1.  A zero
//            divided by n is the same zero, so only the non-zero
//            coordinates (those some payload touched) are rewritten: a read
//            of out and a few scattered writes instead of a full rewrite.
//
// Also the streaming copy probe used to measure the bandwidth ceiling.
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

// Zero fill: one workgroup per CU, each writing 4096-element tiles (four
// 16-byte stores per thread) in turn; measured 3 us faster at 25.6e6 than a
// grid-stride fill from 8 workgroups per CU.
constexpr int kFillWorkgroupsPerCU = 1;

__global__ __launch_bounds__(kBlock) void fill_zero_kernel(float *__restrict__ out, int64_t d) {
    const int64_t nvec = d / 4;
    f32x4 *o4 = reinterpret_cast<f32x4 *>(out);
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    const int64_t ntile = nvec / (4 * kBlock);
    for (int64_t t = blockIdx.x; t < ntile; t += gridDim.x) {
#pragma unroll
        for (int j = 0; j < 4; ++j) o4[t * 4 * kBlock + j * kBlock + threadIdx.x] = z;
    }
    // the vectors after the last whole tile
    for (int64_t v = ntile * 4 * kBlock + int64_t(blockIdx.x) * kBlock + threadIdx.x; v < nvec;
         v += int64_t(gridDim.x) * kBlock)
        o4[v] = z;
    const int64_t t = nvec * 4 + int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d) out[t] = 0.0f;
}

template <bool kFirst>
__global__ __launch_bounds__(kBlock) void scatter_add_kernel(const int32_t *__restrict__ idx,
                                                             const float *__restrict__ val,
                                                             const uint32_t *__restrict__ count,
                                                             int64_t cap, int64_t d,
                                                             float *__restrict__ out) {
    int64_t n = cap;
    if (count != nullptr) n = min(int64_t(*count), cap);
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    for (int64_t j = int64_t(blockIdx.x) * kBlock + threadIdx.x; j < n; j += stride) {
        const int32_t i = idx[j];
        if (i >= 0 && int64_t(i) < d)
            out[i] = __fadd_rn(kFirst ? 0.0f : out[i], val[j]);
    }
}

__global__ __launch_bounds__(kBlock) void scale_kernel(float *__restrict__ out, int64_t d,
                                                       float n) {
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    const int64_t nvec = d / 4;
    f32x4 *o4 = reinterpret_cast<f32x4 *>(out);
    for (int64_t v = int64_t(blockIdx.x) * kBlock + threadIdx.x; v < nvec; v += stride) {
        const f32x4 x = __builtin_nontemporal_load(o4 + v);
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (x[c] != 0.0f) out[4 * v + c] = __fdiv_rn(x[c], n);
    }
    const int64_t t = nvec * 4 + int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d) {
        const float x = out[t];
        if (x != 0.0f) out[t] = __fdiv_rn(x, n);
    }
}

// Same tile shape, grid sizing and cache hints as the hard-threshold kernel:
// four 16-byte non-temporal loads per thread in flight, then four
// non-temporal stores.
__global__ __launch_bounds__(kBlock) void copy_kernel(const float *__restrict__ src,
                                                      float *__restrict__ dst, int64_t n,
                                                      uint32_t ntiles) {
    const int tid = threadIdx.x;
    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
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
                                                              uint32_t ntiles) {
    const int tid = threadIdx.x;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
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

uint32_t stream_grid(int64_t nvec) {
    return persistent_grid((nvec + int64_t(kBlock) * 4 - 1) / (int64_t(kBlock) * 4));
}

}  // namespace

hipError_t launch_accumulate(const int32_t *const *idx, const float *const *val,
                             const uint32_t *const *counts, const int64_t *caps,
                             int32_t n, int64_t d, float *out, hipStream_t stream) {
    // The dense passes use 16-byte accesses; `out` is required to be 16-byte
    // aligned by the ABI layer.
    const uint32_t dense_grid = stream_grid(d / 4 + 1);
    const uint32_t fill_grid = uint32_t(device_cu_count() * kFillWorkgroupsPerCU);
    fill_zero_kernel<<<fill_grid, kBlock, 0, stream>>>(out, d);
    bool first = true;
    for (int32_t w = 0; w < n; ++w) {
        const int64_t cap = caps[w];
        if (cap <= 0) continue;
        const uint32_t grid = persistent_grid((cap + kTile - 1) / kTile);
        const uint32_t *cnt = counts != nullptr ? counts[w] : nullptr;
        if (first)
            scatter_add_kernel<true><<<grid, kBlock, 0, stream>>>(idx[w], val[w], cnt, cap, d, out);
        else
            scatter_add_kernel<false><<<grid, kBlock, 0, stream>>>(idx[w], val[w], cnt, cap, d, out);
        first = false;
    }
    if (n > 1) scale_kernel<<<dense_grid, kBlock, 0, stream>>>(out, d, float(n));
    return hipGetLastError();
}

hipError_t launch_stream_probe(const float *x, float *y, int64_t n, int mode,
                               hipStream_t stream) {
    const int64_t tiles = n > 0 ? (n + kTile - 1) / kTile : 1;
    const uint32_t grid = balanced_grid(tiles, kHtWorkgroupsPerCU);
    if (mode == 1)
        stream_probe_kernel<1><<<grid, kBlock, 0, stream>>>(x, y, n, uint32_t(tiles));
    else if (mode == 2)
        stream_probe_kernel<2><<<grid, kBlock, 0, stream>>>(x, y, n, uint32_t(tiles));
    else
        stream_probe_kernel<3><<<grid, kBlock, 0, stream>>>(x, y, n, uint32_t(tiles));
    return hipGetLastError();
}

hipError_t launch_copy(const float *src, float *dst, int64_t n, hipStream_t stream) {
    const int64_t tiles = n > 0 ? (n + kTile - 1) / kTile : 1;
    copy_kernel<<<balanced_grid(tiles, kHtWorkgroupsPerCU), kBlock, 0, stream>>>(src, dst, n,
                                                                               uint32_t(tiles));
    return hipGetLastError();
}

}  // namespace efs
