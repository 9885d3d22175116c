// Device-side building blocks shared by the efsparse kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace efs {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;              // threads per workgroup (4 waves)
constexpr int kWave = 64;
constexpr int kWaves = kBlock / kWave;
constexpr int kVecPerThread = 4;         // float4 per thread per tile
constexpr int kTile = kBlock * kVecPerThread * 4;   // 4096 elements per tile

// Resident workgroups per compute unit assumed by the grid sizing
// (balanced_grid): the hard-threshold pass (two 4-wave workgroups per CU
// measured fastest), kernels staging pairs in LDS (up to 33 KiB each), and
// histogram / scan passes.
constexpr int kHtWorkgroupsPerCU = 2;
constexpr int kStageWorkgroupsPerCU = 4;
constexpr int kScanWorkgroupsPerCU = 8;

// The tiles a workgroup of a persistent grid takes: first, first + stride,
// ... below end.  Plain: tile b, b + G, b + 2G, ... (the resident workgroups
// sweep one window of the vector together).  By XCD: workgroups b with the
// same b % 8 run on one XCD (workgroups are dispatched to the 8 XCDs in
// turn), so each XCD takes a contiguous share of the tiles in proportion to
// its workgroups, and its workgroups stride through that share.
constexpr int kXcds = 8;
// Tiles per workgroup from which a sweep walks the vector by XCD.  Measured
// on the hard threshold (2 workgroups per CU): by XCD is 1-2 % faster from
// 6e8 elements (290 tiles per workgroup) up to 1.5e9, and 1-9 % slower at
// 4e8 and below (110e6: 224.5 against 239.3 us).
constexpr int kXcdWalkMinTiles = 256;

struct TileWalk {
    uint32_t first, end, stride;
};

__device__ __forceinline__ TileWalk tile_walk(uint32_t ntiles, bool by_xcd) {
    const uint32_t G = gridDim.x, b = blockIdx.x;
    if (!by_xcd) return TileWalk{b, ntiles, G};
    const uint32_t x = b % kXcds;
    const uint32_t n_x = (G - x + kXcds - 1) / kXcds;                 // workgroups on this XCD
    const uint32_t before = x * (G / kXcds) + min(x, G % kXcds);     // on the XCDs before it
    const uint32_t lo = uint32_t(uint64_t(ntiles) * before / G);
    const uint32_t hi = uint32_t(uint64_t(ntiles) * (before + n_x) / G);
    return TileWalk{lo + b / kXcds, hi, n_x};
}

// Counter word layout used for single-launch stream compaction: the low 40
// bits accumulate the number of emitted pairs, the high 24 bits count
// workgroups that have finished (a ticket, so the last one is known).
constexpr int kTicketShift = 40;
constexpr uint64_t kCountMask = (uint64_t(1) << kTicketShift) - 1;
constexpr uint64_t kTicketOne = uint64_t(1) << kTicketShift;

// p = e + lr*g with two separately rounded fp32 operations.
__device__ __forceinline__ float ef_accumulate(float e, float lr, float g) {
    return __fadd_rn(e, __fmul_rn(lr, g));
}

__device__ __forceinline__ uint32_t magnitude_key(float p) {
    return __float_as_uint(p) & 0x7fffffffu;
}

// Number of set bits of `mask` held by lanes below the calling lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi(uint32_t(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo(uint32_t(mask), 0u));
}

// Exclusive prefix over the wave of a small per-lane count c (0 <= c < 32),
// from five ballots of its bits; also returns the wave total.
__device__ __forceinline__ uint32_t wave_prefix_small(uint32_t c, uint32_t &total) {
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int b = 0; b < 5; ++b) {
        const uint64_t m = __ballot((c >> b) & 1u);
        pre += lanes_below(m) << b;
        tot += uint32_t(__popcll(m)) << b;
    }
    total = tot;
    return pre;
}

// Exclusive prefix over the block of a per-thread count c (< 32), and the
// block total.  Uses kWaves words of LDS; contains two barriers.
__device__ __forceinline__ uint32_t block_prefix_small(uint32_t c, uint32_t *s_wave,
                                                       uint32_t &block_total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    uint32_t wtot;
    uint32_t pre = wave_prefix_small(c, wtot);
    if (lane == 0) s_wave[wave] = wtot;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        const uint32_t v = s_wave[w];
        off += (w < wave) ? v : 0u;
        tot += v;
    }
    __syncthreads();
    block_total = tot;
    return pre + off;
}

// Sum of a per-thread value over the workgroup (every thread gets it).
// Uses kWaves words of LDS; contains two barriers.
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t *s_wave) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & (kWave - 1)) == 0) s_wave[threadIdx.x / kWave] = v;
    __syncthreads();
    uint32_t tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += s_wave[w];
    __syncthreads();
    return tot;
}

// Sum of a per-thread double over the workgroup (thread 0's result is the
// total).  Uses kWaves doubles of LDS; contains two barriers.
__device__ __forceinline__ double block_sum_f64(double v, double *s_wave) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & (kWave - 1)) == 0) s_wave[threadIdx.x / kWave] = v;
    __syncthreads();
    double tot = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += s_wave[w];
    __syncthreads();
    return tot;
}

// Maximum of a per-thread value over the workgroup (every thread gets it).
__device__ __forceinline__ uint32_t block_max(uint32_t v, uint32_t *s_wave) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v = max(v, uint32_t(__shfl_xor(int(v), off)));
    if ((threadIdx.x & (kWave - 1)) == 0) s_wave[threadIdx.x / kWave] = v;
    __syncthreads();
    uint32_t m = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) m = max(m, s_wave[w]);
    __syncthreads();
    return m;
}

// Workgroup-local staging of (index, value) pairs in LDS.  Kept pairs of
// successive tiles are appended here and written to the global payload in
// coalesced runs, one atomic per flush instead of one per tile.
template <int N>
struct PairStageN {
    int32_t idx[N];
    float val[N];
    uint32_t wave[kWaves];
    unsigned long long base;
};
using PairStage = PairStageN<kTile>;

// Flushes the `fill` staged pairs to payload slots reserved by one atomic on
// `word`.  With `last` the workgroup also takes its ticket; the workgroup
// holding the final ticket (all others have added their pairs by then)
// publishes the total to *count when count is non-null, and returns `word`
// to zero for the next call.  Slots at or past `cap` are not written.
// Called by every thread of the workgroup; contains barriers.
// Error-feedback telemetry accumulated across calls (layout of the C ABI's
// telemetry object): the total error sum_t ||e_{t+1}||^2 as kTelemetryParts
// partial sums (workgroup b adds into part b mod kTelemetryParts: one binary64
// atomic per workgroup on a single word serialises at the end of the pass),
// total pairs sent sum_t k_t, running max of |e_{t+1}| as a bit pattern,
// number of calls.
constexpr int kTelemetryParts = 32;
struct Telemetry {
    double err2_part[kTelemetryParts];
    double sent_total;
    uint32_t max_abs_bits;
    uint32_t calls;
    uint64_t reserved[2];
};
static_assert(sizeof(Telemetry) == 288, "telemetry object layout");

template <int N>
__device__ __forceinline__ void stage_flush(PairStageN<N> &st, uint32_t fill, bool last,
                                            unsigned long long *word, uint32_t *count,
                                            uint64_t cap, int32_t *__restrict__ idx,
                                            float *__restrict__ val,
                                            Telemetry *tel = nullptr) {
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint64_t add = (last ? kTicketOne : 0ull) | fill;
        const uint64_t old = add ? atomicAdd(word, (unsigned long long)add) : 0ull;
        const uint64_t base = old & kCountMask;
        if (last && (old >> kTicketShift) == uint64_t(gridDim.x - 1)) {
            if (count != nullptr) *count = uint32_t(base + fill);
            if (tel != nullptr) {
                atomicAdd(&tel->sent_total, double(base + fill));
                atomicAdd(&tel->calls, 1u);
            }
            __hip_atomic_store(word, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        st.base = base;
    }
    __syncthreads();
    const uint64_t base = st.base;
    for (uint32_t j = threadIdx.x; j < fill; j += kBlock) {
        const uint64_t o = base + j;
        if (o < cap) {
            idx[o] = st.idx[j];
            val[o] = st.val[j];
        }
    }
    __syncthreads();
}

// Appends the elements of one tile selected by `mask` (bit 4*j + c for
// element (j, c) of this thread; index tile0 + (j*kBlock + tid)*4 + c, value
// v[j][c]) to the stage, flushing first when they might not fit.  A tile
// with more selected elements than the stage holds is written straight to
// the payload behind its own atomic.  `fill` is identical in all threads.
// Called by every thread of the workgroup; contains barriers.
template <int N>
__device__ __forceinline__ void stage_mask(PairStageN<N> &st, uint32_t &fill, uint32_t mask,
                                           const float (&v)[kVecPerThread][4], int64_t tile0,
                                           unsigned long long *word, uint64_t cap,
                                           int32_t *__restrict__ idx, float *__restrict__ val) {
    uint32_t total;
    const uint32_t pos = block_prefix_small(__popc(mask), st.wave, total);
    if (total == 0) return;
    const bool direct = total > uint32_t(N);
    if (direct || fill + total > uint32_t(N)) {
        stage_flush(st, fill, false, word, nullptr, cap, idx, val);
        fill = 0;
    }
    uint64_t o = fill + pos;
    if (direct) {
        // stage_flush ended with a barrier, so st.base is free to reuse
        if (threadIdx.x == 0) st.base = atomicAdd(word, (unsigned long long)total) & kCountMask;
        __syncthreads();
        o += st.base;
    }
#pragma unroll
    for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if ((mask >> (4 * j + c)) & 1u) {
                const int32_t i = int32_t(tile0 + int64_t(j * kBlock + int(threadIdx.x)) * 4 + c);
                if (direct) {
                    if (o < cap) {
                        idx[o] = i;
                        val[o] = v[j][c];
                    }
                } else {
                    st.idx[o] = i;
                    st.val[o] = v[j][c];
                }
                ++o;
            }
        }
    }
    if (direct)
        __syncthreads();  // st.base is read above before any later flush rewrites it
    else
        fill += total;
}

}  // namespace efs
