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

// Counter word layout used for single-launch stream compaction: the low 40
// bits accumulate the number of emitted pairs, the high 24 bits count tiles
// that have reserved their slice (a ticket, so the last tile is known).
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

__device__ __forceinline__ uint32_t atomic_load_u32(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Last-workgroup election.  Every thread fences its own global writes
// (release), the block synchronises, one thread takes a ticket; the block
// holding the last ticket fences again (acquire) before reading what the
// other blocks produced.  Returns true in all threads of the last block.
__device__ __forceinline__ bool last_block_done(uint32_t *ticket, uint32_t nblocks,
                                                uint32_t *s_flag) {
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) *s_flag = (atomicAdd(ticket, 1u) == nblocks - 1u) ? 1u : 0u;
    __syncthreads();
    const bool last = *s_flag != 0u;
    if (last) __threadfence();
    return last;
}

}  // namespace efs
