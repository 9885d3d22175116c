// Exchange-and-average of n workers' payloads fused with the model update
// that follows it (Algorithm 1: x <- x - avg; Appendix C.6.2, Algorithm 2:
// m <- beta m + avg, x <- x - gamma (avg + m)), in one dense or sparse pass.
//
// The index space is cut into ranges of kRange coordinates.  The pairs of
// every payload are first grouped in a workspace into one segment per
// (range, worker), range-major and worker-minor; then one workgroup per
// range sums its pairs into an LDS tile worker by worker (the summation
// order of the definition) and applies the update to its coordinates:
//
//   zero     one counter per (range, worker) = 0
//   count    counters += pairs per segment (one atomic per run of equal
//            ranges within a wave)
//   scan     exclusive prefix of the counters in place, per 4096-counter
//            chunk; with more than one chunk, `top` then scans the chunk
//            totals (one workgroup)
//   scatter  every pair to a slot of its segment; afterwards each counter
//            holds the end of its segment
//   range    per range: LDS sum in worker order, then
//              average   out = sum / n                       (dense write)
//              sgd       x -= sum / n at touched coordinates  (sparse)
//              momentum  m, x updated at every coordinate      (dense)
//
// Indices are distinct within a payload, so no two lanes adding one
// worker's pairs touch the same LDS word; a barrier separates workers.
//
// With one worker the sum is a single term, so grouping buys nothing: the
// average is the plain fill-and-scatter of sparse_accumulate, and the SGD
// update one scatter x[i] = x[i] - (+0 + v) over the payload (the same bits:
// the sum starts from +0 and the division by 1 is exact).
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

constexpr int kRangeLog = 13;
constexpr int kRange = 1 << kRangeLog;             // coordinates per range (32 KB of LDS)
constexpr int kScanPerThread = 16;
constexpr int kScanChunk = kBlock * kScanPerThread; // counters per scan workgroup
static_assert(kRange % (4 * kBlock) == 0, "range must split into float4 per thread");

struct Payloads {
    const int32_t *idx[kMaxApplyWorkers];
    const float *val[kMaxApplyWorkers];
    const uint32_t *count[kMaxApplyWorkers];
    int64_t cap[kMaxApplyWorkers];
};

struct Layout {
    size_t cnt_off, part_off, pair_off, bytes;
    int64_t ranges, entries, chunks;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

Layout make_layout(int32_t n, int64_t d, int64_t total_cap) {
    Layout L;
    L.ranges = (d + kRange - 1) / kRange;
    L.entries = L.ranges * n;
    L.chunks = (L.entries + kScanChunk - 1) / kScanChunk;
    L.cnt_off = 0;
    L.part_off = round_up(size_t(L.entries) * 4 + 4, 256);
    L.pair_off = L.part_off + round_up(size_t(L.chunks) * 4 + 4, 256);
    L.bytes = L.pair_off + size_t(total_cap) * 8;
    return L;
}

__device__ __forceinline__ int64_t payload_len(const Payloads &p, int w) {
    const int64_t cap = p.cap[w];
    if (p.count[w] == nullptr) return cap;
    return min(int64_t(*p.count[w]), cap);
}

__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t o = __shfl_up(v, off);
        if (lane >= off) v += o;
    }
    return v;
}

__global__ __launch_bounds__(kBlock) void apply_zero_kernel(uint32_t *__restrict__ cnt,
                                                            int64_t entries) {
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    for (int64_t j = int64_t(blockIdx.x) * kBlock + threadIdx.x; j < entries; j += stride)
        cnt[j] = 0u;
}

// Walks the pairs of worker blockIdx.y in wave-sized groups.  Each lane
// with a valid pair (index in [0, d)) finds the range of its pair; the first
// lane of every run of lanes with equal ranges adds the run length to the
// counter of (range, worker).  kScatter also places the pairs: slot =
// segment start + the counter value the run's atomic returned + the lane's
// place in the run.  A slot holds (worker << kRangeLog | index in range,
// value bits).
template <bool kScatter>
__global__ __launch_bounds__(kBlock) void apply_group_kernel(Payloads p, int32_t n, int64_t d,
                                                             uint32_t *__restrict__ cnt,
                                                             const uint32_t *__restrict__ part,
                                                             uint2 *__restrict__ pairs,
                                                             int64_t pair_cap) {
    const int w = blockIdx.y;
    const int64_t c = payload_len(p, w);
    const int32_t *__restrict__ idx = p.idx[w];
    const float *__restrict__ val = p.val[w];
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    for (int64_t base = int64_t(blockIdx.x) * kBlock; base < c; base += stride) {
        const int64_t j = base + threadIdx.x;
        int32_t i = -1;
        if (j < c) i = idx[j];
        const bool valid = i >= 0 && int64_t(i) < d;
        // invalid lanes get keys no valid lane has and that differ from
        // their neighbours', so each is a run of its own and never counted
        const uint32_t key = valid ? uint32_t(i) >> kRangeLog : 0x80000000u + uint32_t(lane);
        const uint32_t prev = __shfl_up(key, 1);
        const bool start = lane == 0 || key != prev;
        const uint64_t starts = __ballot(start);
        // run leader of this lane: highest start at or below it
        const uint64_t at_or_below = lane == 63 ? ~uint64_t(0) : ((uint64_t(2) << lane) - 1);
        const int leader = 63 - __clzll(starts & at_or_below);
        uint32_t old = 0;
        if (valid && start) {
            const uint64_t above = lane == 63 ? 0 : (starts >> (lane + 1));
            const int next = above == 0 ? 64 : lane + __ffsll((long long)above);
            old = atomicAdd(&cnt[int64_t(key) * n + w], uint32_t(next - lane));
        }
        if (kScatter) {
            const uint32_t run_base = __shfl(old, leader);
            if (valid) {
                const int64_t e = int64_t(key) * n + w;
                const int64_t pos = int64_t(part[e / kScanChunk]) + run_base + (lane - leader);
                const uint32_t tag = (uint32_t(w) << kRangeLog) | (uint32_t(i) & (kRange - 1));
                if (pos < pair_cap) pairs[pos] = make_uint2(tag, __float_as_uint(val[j]));
            }
        }
    }
}

// Exclusive prefix of one chunk of counters in place; part[chunk] = the
// chunk total, or 0 (the exclusive prefix) when there is only one chunk.
__global__ __launch_bounds__(kBlock) void apply_scan_kernel(uint32_t *__restrict__ cnt,
                                                            int64_t entries,
                                                            uint32_t *__restrict__ part) {
    __shared__ uint32_t s_wave[kWaves];
    const int64_t first = int64_t(blockIdx.x) * kScanChunk + int64_t(threadIdx.x) * kScanPerThread;
    uint32_t v[kScanPerThread];
    uint32_t sum = 0;
#pragma unroll
    for (int q = 0; q < kScanPerThread; ++q) {
        v[q] = first + q < entries ? cnt[first + q] : 0u;
        sum += v[q];
    }
    const uint32_t incl = wave_inclusive_sum(sum);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    if (lane == kWave - 1) s_wave[wave] = incl;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
        off += q < wave ? s_wave[q] : 0u;
        tot += s_wave[q];
    }
    uint32_t run = off + incl - sum;
#pragma unroll
    for (int q = 0; q < kScanPerThread; ++q) {
        if (first + q < entries) cnt[first + q] = run;
        run += v[q];
    }
    if (threadIdx.x == 0) part[blockIdx.x] = gridDim.x == 1 ? 0u : tot;
}

// Exclusive prefix of the chunk totals in place (a single workgroup).
__global__ __launch_bounds__(kBlock) void apply_top_kernel(uint32_t *__restrict__ part,
                                                           int64_t chunks) {
    __shared__ uint32_t s_wave[kWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    uint32_t carry = 0;
    for (int64_t base = 0; base < chunks; base += kBlock) {
        const int64_t j = base + threadIdx.x;
        const uint32_t v = j < chunks ? part[j] : 0u;
        const uint32_t incl = wave_inclusive_sum(v);
        if (lane == kWave - 1) s_wave[wave] = incl;
        __syncthreads();
        uint32_t off = 0, tot = 0;
#pragma unroll
        for (int q = 0; q < kWaves; ++q) {
            off += q < wave ? s_wave[q] : 0u;
            tot += s_wave[q];
        }
        __syncthreads();
        if (j < chunks) part[j] = carry + off + incl - v;
        carry += tot;
    }
}

__device__ __forceinline__ float average_of(float s, int32_t n, float fn) {
    return n > 1 ? __fdiv_rn(s, fn) : s;
}

__device__ __forceinline__ int64_t segment_end(const uint32_t *cnt, const uint32_t *part,
                                               int64_t e) {
    return int64_t(part[e / kScanChunk]) + cnt[e];
}

template <int kMode>
__global__ __launch_bounds__(kBlock) void apply_range_kernel(const uint32_t *__restrict__ cnt,
                                                             const uint32_t *__restrict__ part,
                                                             const uint2 *__restrict__ pairs,
                                                             int64_t pair_cap, int32_t n,
                                                             int64_t d, float *__restrict__ x,
                                                             float *__restrict__ m, float beta,
                                                             float gamma) {
    __shared__ f32x4 acc4[kRange / 4];
    __shared__ uint32_t claim[kRange / 32];
    __shared__ int64_t bound[kMaxApplyWorkers + 1];
    float *acc = reinterpret_cast<float *>(acc4);
    const int tid = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int64_t r0 = b * kRange;
    const int64_t len = min(int64_t(kRange), d - r0);
    // bound[w] .. bound[w+1] is worker w's segment of this range; all n + 1
    // bounds are loaded at once.  They are clamped to the pair slots so that
    // no read can leave the workspace even if a payload changed between the
    // passes.
    const int64_t e0 = b * n;
    if (tid <= n) {
        const int64_t e = e0 - 1 + tid;
        bound[tid] = e < 0 ? 0 : min(segment_end(cnt, part, e), pair_cap);
    }
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int q = tid; q < kRange / 4; q += kBlock) acc4[q] = z;
    if (kMode == 1)
        for (int q = tid; q < kRange / 32; q += kBlock) claim[q] = 0u;
    __syncthreads();
    const int64_t first = bound[0];
    const int64_t last = max(first, bound[n]);

    // Pairs are loaded kBatch at a time, all loads of a batch in flight
    // together; the batch is then added worker by worker with a barrier
    // between workers.  Segments are ordered by worker, so this keeps the
    // worker order of every coordinate's sum.
    constexpr int kPer = 4;
    constexpr int64_t kBatch = int64_t(kPer) * kBlock;
    const bool one_batch = last - first <= kBatch;
    uint2 pr[kPer];
    for (int64_t base = first; base < last; base += kBatch) {
#pragma unroll
        for (int p = 0; p < kPer; ++p) {
            const int64_t q = base + p * kBlock + tid;
            pr[p] = q < last ? pairs[q] : make_uint2(0xFFFFFFFFu, 0u);
        }
        const int64_t qhi = min(last, base + kBatch) - 1;
        int wlo = 0, whi = 0;
        while (wlo < n - 1 && base >= bound[wlo + 1]) ++wlo;
        while (whi < n - 1 && qhi >= bound[whi + 1]) ++whi;
        for (int w = wlo; w <= whi; ++w) {
#pragma unroll
            for (int p = 0; p < kPer; ++p) {
                if ((pr[p].x >> kRangeLog) != uint32_t(w)) continue;
                const uint32_t li = pr[p].x & (kRange - 1);
                acc[li] = __fadd_rn(acc[li], __uint_as_float(pr[p].y));
            }
            __syncthreads();
        }
    }
    const float fn = float(n);

    if (kMode == 1) {
        // x -= avg at each coordinate some payload touched, once
        for (int64_t base = first; base < last; base += kBatch) {
#pragma unroll
            for (int p = 0; p < kPer; ++p) {
                const int64_t q = base + p * kBlock + tid;
                if (q >= last) continue;
                const uint32_t li = (one_batch ? pr[p].x : pairs[q].x) & (kRange - 1);
                if (li >= uint32_t(len)) continue;
                const uint32_t bit = 1u << (li & 31u);
                const uint32_t was = atomicOr(&claim[li >> 5], bit);
                if ((was & bit) == 0u) {
                    const int64_t i = r0 + li;
                    x[i] = __fsub_rn(x[i], average_of(acc[li], n, fn));
                }
            }
        }
        return;
    }

    if (len == kRange) {
        constexpr int kVec = kRange / 4 / kBlock;
        f32x4 *x4 = reinterpret_cast<f32x4 *>(x + r0);
        if (kMode == 0) {
#pragma unroll
            for (int q = 0; q < kVec; ++q) {
                f32x4 a = acc4[q * kBlock + tid];
#pragma unroll
                for (int c = 0; c < 4; ++c) a[c] = average_of(a[c], n, fn);
                x4[q * kBlock + tid] = a;
            }
        } else {
            // x and m stream through once: non-temporal loads and stores (with
            // x and m coming from HBM, 16 % faster than default caching)
            f32x4 *m4 = reinterpret_cast<f32x4 *>(m + r0);
            f32x4 xv[kVec], mv[kVec];
#pragma unroll
            for (int q = 0; q < kVec; ++q) {
                xv[q] = __builtin_nontemporal_load(x4 + q * kBlock + tid);
                mv[q] = __builtin_nontemporal_load(m4 + q * kBlock + tid);
            }
#pragma unroll
            for (int q = 0; q < kVec; ++q) {
                const f32x4 a = acc4[q * kBlock + tid];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const float avg = average_of(a[c], n, fn);
                    const float mn = __fadd_rn(__fmul_rn(beta, mv[q][c]), avg);
                    mv[q][c] = mn;
                    xv[q][c] = __fsub_rn(xv[q][c], __fmul_rn(gamma, __fadd_rn(avg, mn)));
                }
                __builtin_nontemporal_store(mv[q], m4 + q * kBlock + tid);
                __builtin_nontemporal_store(xv[q], x4 + q * kBlock + tid);
            }
        }
    } else {
        for (int64_t q = tid; q < len; q += kBlock) {
            const float avg = average_of(acc[q], n, fn);
            if (kMode == 0) {
                x[r0 + q] = avg;
            } else {
                const float mn = __fadd_rn(__fmul_rn(beta, m[r0 + q]), avg);
                m[r0 + q] = mn;
                x[r0 + q] = __fsub_rn(x[r0 + q], __fmul_rn(gamma, __fadd_rn(avg, mn)));
            }
        }
    }
}

// One worker's SGD update: x[i] -= (+0 + v) for each pair (i, v); indices
// outside [0, d) are ignored, as everywhere.
__global__ __launch_bounds__(kBlock) void apply_sgd_one_kernel(const int32_t *__restrict__ idx,
                                                               const float *__restrict__ val,
                                                               const uint32_t *__restrict__ count,
                                                               int64_t cap, int64_t d,
                                                               float *__restrict__ x) {
    int64_t n = cap;
    if (count != nullptr) n = min(int64_t(*count), cap);
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    for (int64_t j = int64_t(blockIdx.x) * kBlock + threadIdx.x; j < n; j += stride) {
        const int32_t i = idx[j];
        if (i >= 0 && int64_t(i) < d) x[i] = __fsub_rn(x[i], __fadd_rn(0.0f, val[j]));
    }
}

}  // namespace

size_t apply_workspace_size(int32_t n, int64_t d, int64_t total_cap) {
    return make_layout(n, d, total_cap).bytes;
}

hipError_t launch_apply(const int32_t *const *idx, const float *const *val,
                        const uint32_t *const *counts, const int64_t *caps, int32_t n,
                        int64_t d, int mode, float *x, float *m, float beta, float gamma,
                        void *workspace, hipStream_t stream) {
    if (d == 0) return hipSuccess;
    if (n == 1 && mode == 0) return launch_accumulate(idx, val, counts, caps, 1, d, x, stream);
    if (n == 1 && mode == 1) {
        if (caps[0] > 0) {
            const uint32_t grid = persistent_grid((caps[0] + kTile - 1) / kTile);
            apply_sgd_one_kernel<<<grid, kBlock, 0, stream>>>(
                idx[0], val[0], counts != nullptr ? counts[0] : nullptr, caps[0], d, x);
        }
        return hipGetLastError();
    }
    Payloads p{};
    int64_t total = 0, max_cap = 0;
    for (int32_t w = 0; w < n; ++w) {
        p.idx[w] = idx[w];
        p.val[w] = val[w];
        p.count[w] = counts != nullptr ? counts[w] : nullptr;
        p.cap[w] = caps[w];
        total += caps[w];
        max_cap = caps[w] > max_cap ? caps[w] : max_cap;
    }
    const Layout L = make_layout(n, d, total);
    char *ws = static_cast<char *>(workspace);
    uint32_t *cnt = reinterpret_cast<uint32_t *>(ws + L.cnt_off);
    uint32_t *part = reinterpret_cast<uint32_t *>(ws + L.part_off);
    uint2 *pairs = reinterpret_cast<uint2 *>(ws + L.pair_off);

    apply_zero_kernel<<<persistent_grid((L.entries + kBlock - 1) / kBlock), kBlock, 0, stream>>>(
        cnt, L.entries);
    // a few hundred workgroups per worker: payloads are usually far shorter
    // than their capacity, and a grid-stride loop covers the rest
    const int64_t group_tiles = (max_cap + kBlock - 1) / kBlock;
    const int64_t group_cap = int64_t(device_cu_count()) * 2;
    const dim3 group_grid(uint32_t(group_tiles < group_cap ? group_tiles : group_cap), uint32_t(n));
    if (max_cap > 0)
        apply_group_kernel<false><<<group_grid, kBlock, 0, stream>>>(p, n, d, cnt, part, pairs, total);
    apply_scan_kernel<<<uint32_t(L.chunks), kBlock, 0, stream>>>(cnt, L.entries, part);
    if (L.chunks > 1) apply_top_kernel<<<1, kBlock, 0, stream>>>(part, L.chunks);
    if (max_cap > 0)
        apply_group_kernel<true><<<group_grid, kBlock, 0, stream>>>(p, n, d, cnt, part, pairs, total);
    const uint32_t grid = uint32_t(L.ranges);
    if (mode == 0)
        apply_range_kernel<0><<<grid, kBlock, 0, stream>>>(cnt, part, pairs, total, n, d, x, m,
                                                            beta, gamma);
    else if (mode == 1)
        apply_range_kernel<1><<<grid, kBlock, 0, stream>>>(cnt, part, pairs, total, n, d, x, m,
                                                            beta, gamma);
    else
        apply_range_kernel<2><<<grid, kBlock, 0, stream>>>(cnt, part, pairs, total, n, d, x, m,
                                                            beta, gamma);
    return hipGetLastError();
}

}  // namespace efs
