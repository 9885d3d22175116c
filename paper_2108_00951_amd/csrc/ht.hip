// Hard-threshold sparsifier with error feedback, one fused pass.
//
// Algorithm 1 (distributed EF SGD) with the hard-threshold compressor of
// section 4.2, S_lambda(p) = { i : |p_i| >= lambda }:
//   p = e + lr*g ;  payload = { (i, p_i) : |p_i| >= lambda } ;  e' = p - kept.
//
// A persistent grid of workgroups strides over 4096-element tiles (for
// long sweeps, each XCD through a contiguous share of them).  Per tile
// each thread loads four 16-byte vectors of g and of e (every wave
// instruction covers 1 KiB of contiguous memory), forms p with a separately
// rounded multiply and add, writes e' straight back, and keeps a 16-bit mask
// of its kept elements.  Ballot prefix sums place the tile's kept pairs in an
// LDS stage; the stage is written to the payload in coalesced runs when it
// could overflow and once at the end, each time behind a single 64-bit
// atomic on the caller's counter object.  The atomic's upper bits count
// finished workgroups so the last one publishes k_t and zeroes the counter:
// one launch per call, no host synchronisation.
//
// Bytes per element: 4 (g) + 4 (e) + 4 (e'), plus 8 per kept pair.  g and e
// are read and e' written with the non-temporal hint: every byte is touched
// once, and with g and e coming from HBM the launch is 7 % (25.6e6 elements)
// to 10 % (110e6) faster than with default caching.
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

// With kStats, every workgroup also sums ||e'||^2 (binary64) and the max of
// |e'| over its elements and adds them to the telemetry object with one
// atomic each (the sum into one of the 32 partial sums, spreading the
// atomics over 32 words); the last workgroup adds k_t and counts the call.
template <bool kVector, bool kStats>
__global__ __launch_bounds__(kBlock) void ht_fused_kernel(
    const float *__restrict__ g, float *__restrict__ e, int64_t d, float lr, float lambda,
    int32_t *__restrict__ idx, float *__restrict__ val, int64_t cap,
    uint32_t *__restrict__ counter, Telemetry *__restrict__ tel, uint32_t ntiles, bool by_xcd) {
    __shared__ PairStage st;
    __shared__ double s_f64[kWaves];
    unsigned long long *word = reinterpret_cast<unsigned long long *>(counter + 2);
    const int tid = threadIdx.x;
    uint32_t fill = 0;  // pairs staged; identical in every thread
    double err2 = 0.0;  // kStats: sum of e'^2 over this thread's elements
    uint32_t max_bits = 0u;

    const TileWalk walk = tile_walk(ntiles, by_xcd);
    for (uint32_t tile = walk.first; tile < walk.end; tile += walk.stride) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float p[kVecPerThread][4];
        uint32_t keep = 0;  // bit 4*j + c: element (j, c) of this thread is sent

        if (kVector && tile0 + kTile <= d) {
            const f32x4 *g4 = reinterpret_cast<const f32x4 *>(g + tile0);
            f32x4 *e4 = reinterpret_cast<f32x4 *>(e + tile0);
            f32x4 gv[kVecPerThread], ev[kVecPerThread];
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
                gv[j] = __builtin_nontemporal_load(g4 + j * kBlock + tid);
                ev[j] = __builtin_nontemporal_load(e4 + j * kBlock + tid);
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
                    if (kStats) {
                        err2 += double(out[c]) * double(out[c]);
                        max_bits = max(max_bits, magnitude_key(out[c]));
                    }
                }
                __builtin_nontemporal_store(out, e4 + j * kBlock + tid);
            }
        } else {
            // Ragged last tile, or g/e not 16-byte aligned: same element map,
            // scalar accesses with a bound check.
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
                        const float r = k ? 0.0f : a;
                        e[i] = r;
                        if (kStats) {
                            err2 += double(r) * double(r);
                            max_bits = max(max_bits, magnitude_key(r));
                        }
                    }
                }
            }
        }

        uint32_t total;
        const uint32_t pos = block_prefix_small(__popc(keep), st.wave, total);
        if (total == 0) continue;
        if (fill + total > uint32_t(kTile)) {
            stage_flush(st, fill, false, word, nullptr, uint64_t(cap), idx, val);
            fill = 0;
        }
        uint32_t o = fill + pos;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((keep >> (4 * j + c)) & 1u) {
                    st.idx[o] = int32_t(tile0 + int64_t(j * kBlock + tid) * 4 + c);
                    st.val[o] = p[j][c];
                    ++o;
                }
            }
        }
        fill += total;
    }
    if (kStats) {
        const double wg_err2 = block_sum_f64(err2, s_f64);
        const uint32_t wg_max = block_max(max_bits, st.wave);
        if (tid == 0) {
            atomicAdd(&tel->err2_part[blockIdx.x % kTelemetryParts], wg_err2);
            atomicMax(&tel->max_abs_bits, wg_max);
        }
    }
    stage_flush(st, fill, true, word, counter, uint64_t(cap), idx, val, kStats ? tel : nullptr);
}

hipError_t launch_ht(const float *g, float *e, int64_t d, float lr, float lambda,
                     int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                     void *telemetry, hipStream_t stream) {
    const int64_t tiles = d > 0 ? (d + kTile - 1) / kTile : 1;
    const uint32_t ntiles = uint32_t(tiles);
    const uint32_t grid = balanced_grid(tiles, kHtWorkgroupsPerCU);
    // long sweeps go XCD by XCD
    const bool by_xcd = tiles >= int64_t(kXcdWalkMinTiles) * grid;
    const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(e)) & 15u) == 0;
    Telemetry *tel = static_cast<Telemetry *>(telemetry);
    if (tel != nullptr) {
        if (vec)
            ht_fused_kernel<true, true><<<grid, kBlock, 0, stream>>>(g, e, d, lr, lambda, idx, val,
                                                                    cap, counter, tel, ntiles, by_xcd);
        else
            ht_fused_kernel<false, true><<<grid, kBlock, 0, stream>>>(g, e, d, lr, lambda, idx, val,
                                                                     cap, counter, tel, ntiles, by_xcd);
    } else {
        if (vec)
            ht_fused_kernel<true, false><<<grid, kBlock, 0, stream>>>(g, e, d, lr, lambda, idx, val,
                                                                     cap, counter, tel, ntiles, by_xcd);
        else
            ht_fused_kernel<false, false><<<grid, kBlock, 0, stream>>>(g, e, d, lr, lambda, idx,
                                                                      val, cap, counter, tel, ntiles, by_xcd);
    }
    return hipGetLastError();
}

}  // namespace efs
