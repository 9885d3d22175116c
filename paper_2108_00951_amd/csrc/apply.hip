// Exchange-and-average of n workers' payloads (Algorithm 1: the average
// (1/n) sum_i Delta_i of the compressed updates), alone or fused with the
// model update that follows it (Algorithm 1: x <- x - avg; Appendix C.6.2,
// Algorithm 2: m <- beta m + avg, x <- x - gamma (avg + m)).
//
// The index space is cut into ranges of kRange coordinates.  The pairs of
// every payload are grouped in a workspace into one segment per (range,
// worker), range-major and worker-minor; then each range with pairs is
// summed in an LDS tile worker by worker (the summation order of the
// definition) and written.  Four launches:
//
//   count    counters += pairs per segment (one atomic per run of equal
//            ranges within a wave); payload counts above their capacity and
//            indices outside [0, d) are noted.  Each counter carries a tag
//            of the call's epoch, so a counter left by an earlier call (or
//            any other content) reads as zero and no clearing pass is needed.
//   scan     one workgroup: the exclusive prefix of the counters (the
//            segment starts), the list of ranges with pairs, the status word
//            of the call, and the counters tagged for the next epoch with
//            count 0 (the next call on the workspace then adds to them
//            without checking tags)
//   scatter  every pair to a slot of its segment (an atomic on the segment
//            start returns the slot); afterwards start[e] is the end of
//            segment e
//   range    a persistent grid takes the listed ranges in turn, adds each
//            one's pairs into an LDS tile worker by worker, then
//              average   out = sum / n over the whole tile
//              sgd       x -= sum / n at the touched coordinates
//            and, for the momentum update, every range (m, x at every
//            coordinate, a zero average where no pair falls).
// The average's zeros stream from extra workgroups of the count and scatter
// launches (their own work is small and latency-bound) and from the range
// launch, which writes them over the empty ranges of the second half.
//
// Indices are distinct within a payload, so no two lanes adding one
// worker's pairs touch the same LDS word.
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

constexpr int kRangeLog = 13;
constexpr int kRange = 1 << kRangeLog;             // coordinates per range (32 KB of LDS)
static_assert(kRange % (4 * kBlock) == 0, "range must split into float4 per thread");
// range kernel workgroups per CU (33 KB of LDS each)
constexpr int kRangeWorkgroupsPerCU = 4;
static_assert(kMaxApplyWorkers <= 64, "a pair's worker fits the tag");

struct Payloads {
    const int32_t *idx[kMaxApplyWorkers];
    const float *val[kMaxApplyWorkers];
    const uint32_t *count[kMaxApplyWorkers];
    int64_t cap[kMaxApplyWorkers];
};

// Counter words: a tag in the bits above kEpochShift, the count below (a
// segment holds at most kRange pairs of one worker, whose indices are
// distinct).  The tag of counter e in the call of epoch E is E xor a
// multiplicative hash of e, so that neither a counter of an earlier call
// nor a workspace filled with any one byte value carries the current tag (a
// constant fill would otherwise give every counter the control block's
// epoch bits).
constexpr int kEpochShift = 24;
constexpr uint64_t kCountBits = (uint64_t(1) << kEpochShift) - 1;
constexpr uint64_t kEpochMask = (uint64_t(1) << (64 - kEpochShift)) - 1;

__device__ __forceinline__ uint64_t counter_tag(uint64_t epoch, uint64_t e) {
    return (epoch ^ ((e + 1) * 0x9E3779B97F4A7C15ull >> 17)) & kEpochMask;
}
constexpr uint64_t kFlagsTagIndex = ~uint64_t(0) - 1;

struct ApplyCtl {
    unsigned long long epoch;  // epoch of the next call (40 bits)
    unsigned long long flags;  // status bits noted during a call, tagged with its epoch
    unsigned long long clean;  // clean_key(epoch, entries) when the counters hold that
                               // epoch's tags with count 0 (set by the scan)
    uint32_t status;           // status bits of the last completed call
    uint32_t nonempty;         // ranges with pairs in this call (listed by the scan)
    uint32_t pad[56];
};
static_assert(sizeof(ApplyCtl) == 256, "control block is 256 bytes");

// The value of ApplyCtl::clean that says every counter e < entries holds
// counter_tag(epoch, e) with count 0, so that the passes may add to and read
// the counters without checking their tags.
__device__ __forceinline__ unsigned long long clean_key(uint64_t epoch, int64_t entries) {
    return 0x436C65616E000000ull ^ (counter_tag(epoch ^ 0x5A5A5A5A5Aull, uint64_t(entries)) << 8);
}

struct Layout {
    size_t cnt_off, start_off, list_off, pair_off, bytes;
    int64_t ranges, entries;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

Layout make_layout(int32_t n, int64_t d, int64_t total_cap) {
    Layout L;
    L.ranges = (d + kRange - 1) / kRange;
    L.entries = L.ranges * n;
    L.cnt_off = sizeof(ApplyCtl);
    L.start_off = L.cnt_off + round_up(size_t(L.entries) * 8, 256);
    L.list_off = L.start_off + round_up(size_t(L.entries + 1) * 4, 256);
    L.pair_off = L.list_off + round_up(size_t(L.ranges) * 4, 256);
    L.bytes = L.pair_off + size_t(total_cap) * 8;
    return L;
}

// Pairs of payload w to read, and whether its count exceeded its capacity.
__device__ __forceinline__ int64_t payload_len(const Payloads &p, int w, bool &truncated) {
    const int64_t cap = p.cap[w];
    truncated = false;
    if (p.count[w] == nullptr) return cap;
    const int64_t c = int64_t(*p.count[w]);
    truncated = c > cap;
    return c < cap ? c : cap;
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

// Adds `len` to a tagged counter word: a word with another tag counts as
// zero.  Returns the count before the addition.
__device__ __forceinline__ uint64_t tagged_add(unsigned long long *w, uint64_t tag, uint64_t len) {
    unsigned long long cur = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (;;) {
        const uint64_t base = (cur >> kEpochShift) == tag ? (cur & kCountBits) : 0;
        const unsigned long long want = (tag << kEpochShift) | ((base + len) & kCountBits);
        const unsigned long long got = atomicCAS(w, cur, want);
        if (got == cur) return base;
        cur = got;
    }
}

// The run of lanes with equal keys that this lane belongs to: its leader
// (first lane) and its length (set for leaders only).  Invalid lanes carry
// keys of their own and form runs of one.
struct Run {
    int leader, len;
};

__device__ __forceinline__ Run lane_run(uint32_t key) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint32_t prev = __shfl_up(key, 1);
    const bool start = lane == 0 || key != prev;
    const uint64_t starts = __ballot(start);
    const uint64_t at_or_below = lane == 63 ? ~uint64_t(0) : ((uint64_t(2) << lane) - 1);
    Run r;
    r.leader = 63 - __clzll(starts & at_or_below);
    r.len = 0;
    if (start) {
        const uint64_t above = lane == 63 ? 0 : (starts >> (lane + 1));
        r.len = (above == 0 ? 64 : lane + __ffsll((long long)above)) - lane;
    }
    return r;
}

// Zeroes x[lo, hi) with workgroups wg of nwg, kThreads threads each
// (16-byte stores in tiles of kThreads * 16 elements; lo is a multiple of
// kRange and x is 16-byte aligned).
template <int kThreads>
__device__ __forceinline__ void zero_share(float *__restrict__ x, int64_t lo, int64_t hi,
                                           int64_t wg, int64_t nwg) {
    if (x == nullptr || hi <= lo) return;
    constexpr int64_t kZeroTile = int64_t(kThreads) * 16;
    const int64_t tiles = (hi - lo) / kZeroTile;
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int64_t t = wg; t < tiles; t += nwg) {
        f32x4 *x4 = reinterpret_cast<f32x4 *>(x + lo + t * kZeroTile);
#pragma unroll
        for (int j = 0; j < 4; ++j) x4[j * kThreads + threadIdx.x] = z;
    }
    if (wg == nwg - 1)
        for (int64_t i = lo + tiles * kZeroTile + threadIdx.x; i < hi; i += kThreads) x[i] = 0.0f;
}

// Rows blockIdx.y < n: count the pairs of worker blockIdx.y per (range,
// worker) segment and note payload counts above their capacity and indices
// outside [0, d).  The rows after them zero x[zlo, zhi) meanwhile.
__global__ __launch_bounds__(kBlock) void apply_count_kernel(Payloads p, int32_t n, int64_t d,
                                                             unsigned long long *__restrict__ cnt,
                                                             int64_t entries,
                                                             ApplyCtl *__restrict__ ctl,
                                                             float *__restrict__ zx, int64_t zlo,
                                                             int64_t zhi) {
    __shared__ uint32_t s_flags;
    if (int(blockIdx.y) >= n) {
        zero_share<kBlock>(zx, zlo, zhi, int64_t(blockIdx.y - n) * gridDim.x + blockIdx.x,
                           int64_t(gridDim.y - n) * gridDim.x);
        return;
    }
    const int w = blockIdx.y;
    const uint64_t epoch = ctl->epoch & kEpochMask;
    // the last call on this workspace left every counter tagged for this
    // epoch with count 0: plain atomic adds suffice
    const bool clean = ctl->clean == clean_key(epoch, entries);
    if (threadIdx.x == 0) s_flags = 0u;
    __syncthreads();
    bool truncated;
    const int64_t c = payload_len(p, w, truncated);
    if (truncated && blockIdx.x == 0 && threadIdx.x == 0) s_flags |= kSparseTruncated;
    const int32_t *__restrict__ idx = p.idx[w];
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    bool bad = false;
    for (int64_t base = int64_t(blockIdx.x) * kBlock; base < c; base += stride) {
        const int64_t j = base + threadIdx.x;
        int32_t i = -1;
        const bool in = j < c;
        if (in) i = idx[j];
        const bool valid = i >= 0 && int64_t(i) < d;
        bad = bad || (in && !valid);
        const uint32_t key = valid ? uint32_t(i) >> kRangeLog : 0x80000000u + uint32_t(lane);
        const Run r = lane_run(key);
        if (valid && r.len > 0) {
            const int64_t e = int64_t(key) * n + w;
            if (clean)
                atomicAdd(&cnt[e], (unsigned long long)r.len);
            else
                tagged_add(&cnt[e], counter_tag(epoch, uint64_t(e)), uint64_t(r.len));
        }
    }
    if (bad) atomicOr(&s_flags, kSparseBadIndex);
    __syncthreads();
    if (threadIdx.x == 0 && s_flags) {
        // a flags word with another tag reads as 0
        tagged_add(&ctl->flags, counter_tag(epoch, kFlagsTagIndex), 0);
        atomicOr(&ctl->flags, (unsigned long long)s_flags);
    }
}

// One workgroup: the exclusive prefix of the counters into the segment
// starts (start[e] = pairs of all segments before e; start[entries] =
// total), the list of ranges with pairs in ascending order, the status word
// of this call, and the counters set up for the next call (tagged for the
// next epoch, count 0).  It takes the counters in tiles of kScanPer per
// thread (consecutive threads, consecutive groups), the next tile's loads in
// flight while the current one is scanned; cnt and start begin on 256-byte
// boundaries of the 16-byte aligned workspace, so every group is 16-byte
// aligned.  The chain of dependent rounds is the launch's cost, so each
// round covers as much as the registers allow.
constexpr int kScanBlock = 1024;
constexpr int kScanWaves = kScanBlock / kWave;
constexpr int kScanPer = 8;
constexpr int64_t kScanTile = int64_t(kScanPer) * kScanBlock;

struct Group {
    unsigned long long c[kScanPer];
};

__device__ __forceinline__ Group load_group(const unsigned long long *cnt, int64_t j, int64_t n) {
    Group q;
    if (j + kScanPer <= n) {
#pragma unroll
        for (int h = 0; h < kScanPer / 2; ++h) {
            const ulonglong2 a = reinterpret_cast<const ulonglong2 *>(cnt + j)[h];
            q.c[2 * h] = a.x;
            q.c[2 * h + 1] = a.y;
        }
    } else {
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) q.c[i] = j + i < n ? cnt[j + i] : 0ull;
    }
    return q;
}

// Block-wide exclusive prefix of v over kScanBlock threads (plus the total);
// uses `s` (kScanWaves words); two barriers.
__device__ __forceinline__ uint32_t scan_block(uint32_t v, uint32_t *s, uint32_t &total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint32_t incl = wave_inclusive_sum(v);
    if (lane == kWave - 1) s[wave] = incl;
    __syncthreads();
    uint32_t run = incl - v, tot = 0;
#pragma unroll
    for (int w = 0; w < kScanWaves; ++w) {
        run += w < wave ? s[w] : 0u;
        tot += s[w];
    }
    __syncthreads();
    total = tot;
    return run;
}

__global__ __launch_bounds__(kScanBlock) void apply_scan_kernel(unsigned long long *__restrict__ cnt,
                                                                uint32_t *__restrict__ start,
                                                                int32_t n, int64_t ranges,
                                                                uint32_t *__restrict__ list,
                                                                ApplyCtl *__restrict__ ctl) {
    __shared__ uint32_t s_wave[kScanWaves];
    const int64_t entries = ranges * n;
    const uint64_t epoch = ctl->epoch & kEpochMask;
    const uint64_t next = (epoch + 1) & kEpochMask;
    const bool clean = ctl->clean == clean_key(epoch, entries);
    uint32_t carry = 0;
    Group q = load_group(cnt, kScanPer * int64_t(threadIdx.x), entries);
    for (int64_t t0 = 0; t0 < entries; t0 += kScanTile) {
        const int64_t j = t0 + kScanPer * int64_t(threadIdx.x);
        const Group cur = q;
        if (t0 + kScanTile < entries) q = load_group(cnt, j + kScanTile, entries);
        uint32_t v[kScanPer], sum = 0;
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            const unsigned long long w = cur.c[i];
            v[i] = (clean || (w >> kEpochShift) == counter_tag(epoch, uint64_t(j + i)))
                       ? uint32_t(w & kCountBits) : 0u;
            sum += v[i];
        }
        // the counters, set up for the next call
        if (j + kScanPer <= entries) {
            ulonglong2 *c2 = reinterpret_cast<ulonglong2 *>(cnt + j);
#pragma unroll
            for (int h = 0; h < kScanPer / 2; ++h)
                c2[h] = make_ulonglong2(counter_tag(next, j + 2 * h) << kEpochShift,
                                        counter_tag(next, j + 2 * h + 1) << kEpochShift);
        } else {
            for (int i = 0; i < kScanPer; ++i)
                if (j + i < entries) cnt[j + i] = counter_tag(next, j + i) << kEpochShift;
        }
        uint32_t total;
        uint32_t run = carry + scan_block(sum, s_wave, total);
        if (j + kScanPer <= entries) {
            uint4 *s4 = reinterpret_cast<uint4 *>(start + j);
#pragma unroll
            for (int h = 0; h < kScanPer / 4; ++h) {
                uint4 o;
                o.x = run;
                run += v[4 * h];
                o.y = run;
                run += v[4 * h + 1];
                o.z = run;
                run += v[4 * h + 2];
                o.w = run;
                run += v[4 * h + 3];
                s4[h] = o;
            }
        } else {
            for (int i = 0; i < kScanPer; ++i) {
                if (j + i < entries) start[j + i] = run;
                run += v[i];
            }
        }
        carry += total;
    }
    if (threadIdx.x == 0) start[entries] = carry;
    __syncthreads();   // every start of this workgroup is written
    // the ranges with pairs (start[(r+1) n] > start[r n]), kScanPer per thread
    uint32_t listed = 0;
    for (int64_t r0 = 0; r0 < ranges; r0 += kScanTile) {
        const int64_t rb = r0 + kScanPer * int64_t(threadIdx.x);
        uint32_t has = 0, cntr = 0;
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            const int64_t r = rb + i;
            if (r < ranges && start[(r + 1) * n] > start[r * n]) {
                has |= 1u << i;
                ++cntr;
            }
        }
        uint32_t total;
        uint32_t pos = listed + scan_block(cntr, s_wave, total);
#pragma unroll
        for (int i = 0; i < kScanPer; ++i)
            if ((has >> i) & 1u) list[pos++] = uint32_t(rb + i);
        listed += total;
    }
    if (threadIdx.x == 0) {
        ctl->nonempty = listed;
        const unsigned long long f = ctl->flags;
        ctl->status = (f >> kEpochShift) == counter_tag(epoch, kFlagsTagIndex) ? uint32_t(f & 0xffu)
                                                                                : 0u;
        ctl->epoch = next;
        ctl->clean = clean_key(next, entries);
    }
}

// Rows blockIdx.y < n place every valid pair of worker blockIdx.y: the
// leader of each run of equal ranges in a wave reserves the run's slots
// with one atomic on the segment's start.  A slot holds (worker <<
// kRangeLog | index in range, value bits).  The rows after them zero
// x[zlo, zhi) meanwhile.
__global__ __launch_bounds__(kBlock) void apply_scatter_kernel(Payloads p, int32_t n, int64_t d,
                                                               uint32_t *__restrict__ start,
                                                               uint2 *__restrict__ pairs,
                                                               int64_t pair_cap,
                                                               float *__restrict__ zx, int64_t zlo,
                                                               int64_t zhi) {
    if (int(blockIdx.y) >= n) {
        zero_share<kBlock>(zx, zlo, zhi, int64_t(blockIdx.y - n) * gridDim.x + blockIdx.x,
                           int64_t(gridDim.y - n) * gridDim.x);
        return;
    }
    const int w = blockIdx.y;
    bool truncated;
    const int64_t c = payload_len(p, w, truncated);
    const int32_t *__restrict__ idx = p.idx[w];
    const float *__restrict__ val = p.val[w];
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    for (int64_t base = int64_t(blockIdx.x) * kBlock; base < c; base += stride) {
        const int64_t j = base + threadIdx.x;
        int32_t i = -1;
        if (j < c) i = idx[j];
        const bool valid = i >= 0 && int64_t(i) < d;
        const uint32_t key = valid ? uint32_t(i) >> kRangeLog : 0x80000000u + uint32_t(lane);
        const Run r = lane_run(key);
        uint32_t old = 0;
        if (valid && r.len > 0) old = atomicAdd(&start[int64_t(key) * n + w], uint32_t(r.len));
        const uint32_t run_base = __shfl(old, r.leader);
        if (valid) {
            const int64_t pos = int64_t(run_base) + (lane - r.leader);
            const uint32_t tag = (uint32_t(w) << kRangeLog) | (uint32_t(i) & (kRange - 1));
            if (pos < pair_cap) pairs[pos] = make_uint2(tag, __float_as_uint(val[j]));
        }
    }
}

__device__ __forceinline__ float average_of(float s, int32_t n, float fn) {
    return n > 1 ? __fdiv_rn(s, fn) : s;
}

// Momentum update of coordinates [r0, r0 + len) with the sums in acc4 (all
// of them, +0 where nothing was added).
__device__ __forceinline__ void momentum_range(const f32x4 *acc4, int64_t r0, int64_t len,
                                               int32_t n, float *__restrict__ x,
                                               float *__restrict__ m, float beta, float gamma) {
    const int tid = threadIdx.x;
    const float fn = float(n);
    const float *acc = reinterpret_cast<const float *>(acc4);
    if (len == kRange) {
        constexpr int kVec = kRange / 4 / kBlock;
        // x and m stream through once: non-temporal loads and stores
        f32x4 *x4 = reinterpret_cast<f32x4 *>(x + r0);
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
    } else {
        for (int64_t q = tid; q < len; q += kBlock) {
            const float avg = average_of(acc[q], n, fn);
            const float mn = __fadd_rn(__fmul_rn(beta, m[r0 + q]), avg);
            m[r0 + q] = mn;
            x[r0 + q] = __fsub_rn(x[r0 + q], __fmul_rn(gamma, __fadd_rn(avg, mn)));
        }
    }
}

// LDS state of one workgroup of the range launch.
struct RangeShared {
    f32x4 acc4[kRange / 4];
    uint32_t claim[kRange / 32];
    int64_t bound[kMaxApplyWorkers + 1];
};

// Range b: adds its pairs into the LDS tile worker by worker and writes the
// result: the average's whole tile (mode 0), x -= avg at the touched
// coordinates (mode 1), or the momentum update of every coordinate (mode
// 2).  Worker w's pairs are [end[b n + w - 1], end[b n + w]) with end =
// start after the scatter (end[-1] = 0), clamped to the pair slots so that
// no read can leave the workspace even if a payload changed between the
// passes.  Pairs are loaded kBatch at a time, all loads of a batch in
// flight together; the batch is then added worker by worker with a barrier
// between workers (segments are in worker order, so every coordinate's sum
// keeps it).  Called by every thread of the workgroup; starts and ends with
// a barrier.
template <int kMode>
__device__ void sum_range(RangeShared &sh, int64_t b, const uint32_t *__restrict__ end,
                          const uint2 *__restrict__ pairs, int64_t pair_cap, int32_t n, int64_t d,
                          float *__restrict__ x, float *__restrict__ m, float beta, float gamma) {
    constexpr int kPer = 4;
    constexpr int64_t kBatch = int64_t(kPer) * kBlock;
    constexpr int kVec = kRange / 4 / kBlock;
    float *acc = reinterpret_cast<float *>(sh.acc4);
    const int tid = threadIdx.x;
    const float fn = float(n);
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    const int64_t r0 = b * kRange;
    const int64_t len = min(int64_t(kRange), d - r0);
    __syncthreads();   // the previous range is done with the LDS state
    if (tid <= n) {
        const int64_t e = b * n - 1 + tid;
        sh.bound[tid] = e < 0 ? 0 : min(int64_t(end[e]), pair_cap);
    }
    for (int q = tid; q < kRange / 4; q += kBlock) sh.acc4[q] = z;
    if (kMode == 1)
        for (int q = tid; q < kRange / 32; q += kBlock) sh.claim[q] = 0u;
    __syncthreads();
    const int64_t first = sh.bound[0];
    const int64_t last = max(first, sh.bound[n]);
    const bool one_batch = last - first <= kBatch;
    uint2 pr[kPer];
    for (int64_t base = first; base < last; base += kBatch) {
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t s = base + q * kBlock + tid;
            pr[q] = s < last ? pairs[s] : make_uint2(0xFFFFFFFFu, 0u);
        }
        const int64_t shi = min(last, base + kBatch) - 1;
        int wlo = 0, whi = 0;
        while (wlo < n - 1 && base >= sh.bound[wlo + 1]) ++wlo;
        while (whi < n - 1 && shi >= sh.bound[whi + 1]) ++whi;
        for (int w = wlo; w <= whi; ++w) {
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                if ((pr[q].x >> kRangeLog) != uint32_t(w)) continue;
                const uint32_t li = pr[q].x & (kRange - 1);
                acc[li] = __fadd_rn(acc[li], __uint_as_float(pr[q].y));
            }
            __syncthreads();
        }
    }

    if (kMode == 2) {
        momentum_range(sh.acc4, r0, len, n, x, m, beta, gamma);
    } else if (kMode == 0) {
        // the whole tile (over any zeros written before)
        if (len == kRange) {
            f32x4 *x4 = reinterpret_cast<f32x4 *>(x + r0);
#pragma unroll
            for (int q = 0; q < kVec; ++q) {
                f32x4 a = sh.acc4[q * kBlock + tid];
#pragma unroll
                for (int c = 0; c < 4; ++c) a[c] = average_of(a[c], n, fn);
                x4[q * kBlock + tid] = a;
            }
        } else {
            for (int64_t q = tid; q < len; q += kBlock) x[r0 + q] = average_of(acc[q], n, fn);
        }
    } else {
        // x -= avg once at each touched coordinate
        for (int64_t base = first; base < last; base += kBatch) {
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int64_t s = base + q * kBlock + tid;
                if (s >= last) continue;
                const uint32_t li = (one_batch ? pr[q].x : pairs[s].x) & (kRange - 1);
                if (li >= uint32_t(len)) continue;
                const uint32_t bit = 1u << (li & 31u);
                const uint32_t was = atomicOr(&sh.claim[li >> 5], bit);
                if ((was & bit) == 0u) x[r0 + li] = __fsub_rn(x[r0 + li], average_of(acc[li], n, fn));
            }
        }
    }
    __syncthreads();
}

// Average and sgd: a persistent grid takes the listed ranges (those with
// pairs) in turn; then, for the average, writes zeros over the empty ranges
// from zdone on (the earlier launches zeroed everything below).  Momentum:
// every range in turn (a range without pairs has a zero average).
template <int kMode>
__global__ __launch_bounds__(kBlock) void apply_range_kernel(const uint32_t *__restrict__ end,
                                                             const uint32_t *__restrict__ list,
                                                             const ApplyCtl *__restrict__ ctl,
                                                             const uint2 *__restrict__ pairs,
                                                             int64_t pair_cap, int32_t n,
                                                             int64_t d, int64_t ranges,
                                                             int64_t zdone, float *__restrict__ x,
                                                             float *__restrict__ m, float beta,
                                                             float gamma) {
    __shared__ RangeShared sh;
    const int64_t G = gridDim.x;
    if (kMode == 2) {
        for (int64_t b = blockIdx.x; b < ranges; b += G)
            sum_range<2>(sh, b, end, pairs, pair_cap, n, d, x, m, beta, gamma);
        return;
    }
    const int64_t ne = ctl->nonempty;
    for (int64_t i = blockIdx.x; i < ne; i += G)
        sum_range<kMode>(sh, list[i], end, pairs, pair_cap, n, d, x, m, beta, gamma);
    if (kMode == 0) {
        constexpr int kVec = kRange / 4 / kBlock;
        const int tid = threadIdx.x;
        const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int64_t b = zdone / kRange + blockIdx.x; b < ranges; b += G) {
            const int64_t first = b == 0 ? 0 : min(int64_t(end[b * n - 1]), pair_cap);
            const int64_t last = min(int64_t(end[b * n + n - 1]), pair_cap);
            if (last > first) continue;   // written by its listed pass
            const int64_t r0 = b * kRange;
            const int64_t len = min(int64_t(kRange), d - r0);
            if (len == kRange) {
                f32x4 *x4 = reinterpret_cast<f32x4 *>(x + r0);
#pragma unroll
                for (int q = 0; q < kVec; ++q) x4[q * kBlock + tid] = z;
            } else {
                for (int64_t q = tid; q < len; q += kBlock) x[r0 + q] = 0.0f;
            }
        }
    }
}

}  // namespace

size_t apply_workspace_size(int32_t n, int64_t d, int64_t total_cap) {
    return make_layout(n, d, total_cap).bytes;
}

size_t apply_status_offset() { return offsetof(ApplyCtl, status); }

hipError_t launch_apply(const int32_t *const *idx, const float *const *val,
                        const uint32_t *const *counts, const int64_t *caps, int32_t n,
                        int64_t d, int mode, float *x, float *m, float beta, float gamma,
                        void *workspace, hipStream_t stream) {
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
    ApplyCtl *ctl = reinterpret_cast<ApplyCtl *>(ws);
    unsigned long long *cnt = reinterpret_cast<unsigned long long *>(ws + L.cnt_off);
    uint32_t *start = reinterpret_cast<uint32_t *>(ws + L.start_off);
    uint32_t *list = reinterpret_cast<uint32_t *>(ws + L.list_off);
    uint2 *pairs = reinterpret_cast<uint2 *>(ws + L.pair_off);

    // The average's zeros: x[0, z1) from the count launch, [z1, z2) from the
    // scatter launch (extra workgroups beside their own small, latency-bound
    // work), the empty ranges from z2 on from the range launch; the listed
    // ranges' tiles are written over them.  (The scan launch is one
    // workgroup's chain of dependent rounds: memory traffic beside it
    // lengthens every round.)
    float *zx = mode == 0 ? x : nullptr;
    const int64_t z1 = (d / 4) / kRange * kRange;
    const int64_t z2 = max_cap > 0 ? (d / 2) / kRange * kRange : z1;
    const int cus = device_cu_count();
    // about two workgroups per CU over all workers: payloads are usually
    // far shorter than their capacity, and a grid-stride loop covers the
    // rest (at least one workgroup per worker, so that every count is checked)
    const int64_t tiles = (max_cap + kBlock - 1) / kBlock;
    const int64_t per_worker = int64_t(cus) * 2 / n;
    int64_t gx = tiles < per_worker ? tiles : per_worker;
    gx = gx < 1 ? 1 : gx;
    // then rows of fill workgroups, about two per CU
    const int64_t fill_rows = zx != nullptr ? (int64_t(cus) * 2 + gx - 1) / gx : 0;
    const dim3 group_grid(uint32_t(gx), uint32_t(n + fill_rows));
    apply_count_kernel<<<group_grid, kBlock, 0, stream>>>(p, n, d, cnt, L.entries, ctl, zx, 0, z1);
    apply_scan_kernel<<<1, kScanBlock, 0, stream>>>(cnt, start, n, L.ranges, list, ctl);
    if (max_cap > 0)
        apply_scatter_kernel<<<group_grid, kBlock, 0, stream>>>(p, n, d, start, pairs, total, zx,
                                                                 z1, z2);
    const int64_t zdone = zx != nullptr ? z2 : 0;
    const int64_t rgrid_cap = int64_t(cus) * kRangeWorkgroupsPerCU;
    const uint32_t grid = uint32_t(L.ranges < rgrid_cap ? L.ranges : rgrid_cap);
    if (mode == 0)
        apply_range_kernel<0><<<grid, kBlock, 0, stream>>>(start, list, ctl, pairs, total, n, d,
                                                            L.ranges, zdone, x, m, beta, gamma);
    else if (mode == 1)
        apply_range_kernel<1><<<grid, kBlock, 0, stream>>>(start, list, ctl, pairs, total, n, d,
                                                            L.ranges, zdone, x, m, beta, gamma);
    else
        apply_range_kernel<2><<<grid, kBlock, 0, stream>>>(start, list, ctl, pairs, total, n, d,
                                                            L.ranges, zdone, x, m, beta, gamma);
    return hipGetLastError();
}

}  // namespace efs
