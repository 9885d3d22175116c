// Hard-threshold sparsifier with error feedback, one fused pass.
//
// Algorithm 1 (distributed EF SGD) with the hard-threshold compressor of
// section 4.2, S_lambda(p) = { i : |p_i| >= lambda }:
//   p = e + lr*g ;  payload = { (i, p_i) : |p_i| >= lambda } ;  e' = p - kept.
//
// One workgroup owns one 4096-element tile.  Each thread loads four 16-byte
// vectors of g and of e (every wave instruction touches 1 KiB of contiguous
// memory), forms p with a separately rounded multiply and add, writes e'
// straight back, and keeps a 16-bit mask of its kept elements.  The tile's
// kept pairs are then compacted without a second pass over memory: ballot
// prefix sums give each thread its offset inside the tile, and one 64-bit
// atomic per tile on the caller's counter object reserves the tile's slice of
// the payload and, in its upper bits, counts finished tiles, so the last
// tile publishes k_t and returns the counter to zero.  Bytes moved per
// element: 4 (g) + 4 (e) + 4 (e') + 8 per kept pair.
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

template <bool kVector>
__global__ __launch_bounds__(kBlock) void ht_fused_kernel(
    const float *__restrict__ g, float *__restrict__ e, int64_t d, float lr, float lambda,
    int32_t *__restrict__ idx, float *__restrict__ val, int64_t cap,
    uint32_t *__restrict__ counter, uint32_t ntiles) {
    __shared__ uint32_t s_wave[kWaves];
    __shared__ uint64_t s_base;

    const int tid = threadIdx.x;
    const int64_t tile0 = int64_t(blockIdx.x) * kTile;
    float p[kVecPerThread][4];
    uint32_t keep = 0;  // bit 4*j + c: element (j, c) of this thread is sent

    if (kVector && tile0 + kTile <= d) {
        const f32x4 *g4 = reinterpret_cast<const f32x4 *>(g + tile0);
        f32x4 *e4 = reinterpret_cast<f32x4 *>(e + tile0);
        f32x4 gv[kVecPerThread], ev[kVecPerThread];
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
            gv[j] = __builtin_nontemporal_load(g4 + j * kBlock + tid);
            ev[j] = e4[j * kBlock + tid];
        }
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
            f32x4 out;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float a = ef_accumulate(ev[j][c], lr, gv[j][c]);
                const bool k = fabsf(a) >= lambda;
                p[j][c] = a;
                keep |= uint32_t(k) << (4 * j + c);
                out[c] = k ? 0.0f : a;
            }
            e4[j * kBlock + tid] = out;
        }
    } else {
        // Ragged last tile, or g/e not 16-byte aligned: same element-to-thread
        // map, scalar accesses with a bound check.
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t i = tile0 + int64_t(j * kBlock + tid) * 4 + c;
                p[j][c] = 0.0f;
                if (i < d) {
                    const float a = ef_accumulate(e[i], lr, g[i]);
                    const bool k = fabsf(a) >= lambda;
                    p[j][c] = a;
                    keep |= uint32_t(k) << (4 * j + c);
                    e[i] = k ? 0.0f : a;
                }
            }
        }
    }

    // Stream compaction of this tile's kept pairs.
    const uint32_t cnt = __popc(keep);
    uint32_t total;
    const uint32_t pos = block_prefix_small(cnt, s_wave, total);
    if (tid == 0) {
        unsigned long long *word = reinterpret_cast<unsigned long long *>(counter + 2);
        const uint64_t old = atomicAdd(word, (unsigned long long)(kTicketOne | total));
        const uint64_t base = old & kCountMask;
        if ((old >> kTicketShift) == uint64_t(ntiles - 1)) {
            // Every other tile has reserved its slice: publish k_t and leave
            // the counter at zero for the next call.
            counter[0] = uint32_t(base + total);
            __hip_atomic_store(word, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        s_base = base;
    }
    __syncthreads();
    if (cnt) {
        uint64_t o = s_base + pos;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((keep >> (4 * j + c)) & 1u) {
                    if (o < uint64_t(cap)) {
                        idx[o] = int32_t(tile0 + int64_t(j * kBlock + tid) * 4 + c);
                        val[o] = p[j][c];
                    }
                    ++o;
                }
            }
        }
    }
}

hipError_t launch_ht(const float *g, float *e, int64_t d, float lr, float lambda,
                     int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                     hipStream_t stream) {
    const int64_t tiles = d > 0 ? (d + kTile - 1) / kTile : 1;
    const uint32_t ntiles = uint32_t(tiles);
    const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(e)) & 15u) == 0;
    if (vec)
        ht_fused_kernel<true><<<ntiles, kBlock, 0, stream>>>(g, e, d, lr, lambda, idx, val, cap,
                                                            counter, ntiles);
    else
        ht_fused_kernel<false><<<ntiles, kBlock, 0, stream>>>(g, e, d, lr, lambda, idx, val,
                                                             cap, counter, ntiles);
    return hipGetLastError();
}

}  // namespace efs
