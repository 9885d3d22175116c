// Exchange-and-average of n workers' payloads (Algorithm 1: the average
// (1/n) sum_i Delta_i of the compressed updates), alone or fused with the
// model update that follows it (Algorithm 1: x <- x - avg; Appendix C.6.2,
// Algorithm 2: m <- beta m + avg, x <- x - gamma (avg + m)).
//
// The index space is cut into ranges (4096 coordinates in the bucketed
// layout, 8192 in the packed one); the pairs of one worker in one range form
// a segment.  Every range is summed in an LDS
// tile worker by worker (the summation order of the definition) and written
// once.  The pairs reach that pass through one of two layouts of the
// caller's workspace:
//
//   bucketed (two launches; about 8 n d bytes)
//     place    every pair to the next free slot of its segment's bucket (a
//              slot per coordinate of the range; one atomic per run of equal
//              ranges within a wave, on the segment's counter)
//     range    (below)
//   packed (four launches; about 8 bytes per pair of capacity)
//     count    counters += pairs per segment
//     scan     one workgroup: the exclusive prefix of the counters, i.e. the
//              segment starts in one array of pairs, range-major and
//              worker-minor
//     scatter  every pair to a slot of its segment (an atomic on the segment
//              start returns the slot); afterwards start[e] is the end of
//              segment e
//     range    (below)
//
// range: one workgroup per range adds the range's pairs into the LDS tile
// worker by worker (a barrier between workers), then writes
//     average   out = sum / n over the whole tile (zeros where no pair falls)
//     sgd       x -= sum / n at the touched coordinates
//     momentum  m and x at every coordinate (a zero average where no pair falls)
// and sets the range's counters up for the next call.  Its first workgroup
// publishes the call's status word and advances the epoch.
//
// Counters carry a tag of the call's epoch, so that a counter left by an
// earlier call (or any other content) reads as zero and no clearing pass is
// needed; once a call has completed, every counter holds the next epoch's
// tag with count 0 and the next call adds to them without checking tags.
// Payload counts above their capacity and indices outside [0, d) are noted
// in the status word.  Indices are distinct within a payload, so no two
// lanes adding one worker's pairs touch the same LDS word.
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

// Coordinates per range: 4096 in the bucketed layout (16 KB of LDS per
// range workgroup, eight of them per CU), 8192 in the packed one (half the
// counters for its one-workgroup scan).
constexpr int kBucketRangeLog = 12;
constexpr int kPackedRangeLog = 13;

template <bool kBucket>
struct Geom {
    static constexpr int kLog = kBucket ? kBucketRangeLog : kPackedRangeLog;
    static constexpr int kRange = 1 << kLog;
    static_assert(kRange % (4 * kBlock) == 0, "range must split into float4 per thread");
};
static_assert(kMaxApplyWorkers <= 64, "a pair's worker fits the tag; one wave reads the counts");

struct Payloads {
    const int32_t *idx[kMaxApplyWorkers];
    const float *val[kMaxApplyWorkers];
    const uint32_t *count[kMaxApplyWorkers];
    int64_t cap[kMaxApplyWorkers];
};

// Counter words: a tag in the bits above kEpochShift, the count below (a
// segment holds at most a range's worth of pairs of one worker, whose
// indices are distinct).  The tag of counter e in the call of epoch E is E xor a
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

// Each word of the control block has one writer launch and is read only by
// launches that run after that writer has finished:
//   epoch, clean   written by the range launch, read by the next call's first
//                  launch;
//   run_epoch, run_clean   the call's epoch and whether its counters were
//                  clean, written by the first launch for the later ones;
//   flags          added to by the first launch;
//   status         written by the range launch.
struct ApplyCtl {
    unsigned long long epoch;  // epoch of the next call (40 bits)
    unsigned long long flags;  // status bits noted during a call, tagged with its epoch
    unsigned long long clean;  // clean_key(epoch, entries) when the counters hold that
                               // epoch's tags with count 0
    uint32_t status;           // status bits of the last completed call
    uint32_t run_clean;        // 1 when this call's counters started clean
    unsigned long long run_epoch;   // epoch of the call in progress
    uint32_t pad[54];
};
static_assert(sizeof(ApplyCtl) == 256, "control block is 256 bytes");

// The value of ApplyCtl::clean that says every counter e < entries holds
// counter_tag(epoch, e) with count 0, so that the passes may add to and read
// the counters without checking their tags.
__device__ __forceinline__ unsigned long long clean_key(uint64_t epoch, int64_t entries) {
    return 0x436C65616E000000ull ^ (counter_tag(epoch ^ 0x5A5A5A5A5Aull, uint64_t(entries)) << 8);
}

struct Layout {
    size_t cnt_off, start_off, pair_off, bytes;
    int64_t ranges, entries, pair_slots;
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ctl | cnt[entries] | (packed: start[entries + 1]) | pair slots
Layout make_layout(int32_t n, int64_t d, int64_t total_cap, bool bucketed) {
    Layout L;
    const int64_t range = int64_t(1) << (bucketed ? kBucketRangeLog : kPackedRangeLog);
    L.ranges = (d + range - 1) / range;
    L.entries = L.ranges * n;
    L.cnt_off = sizeof(ApplyCtl);
    L.start_off = L.cnt_off + round_up(size_t(L.entries) * 8, 256);
    if (bucketed) {
        L.pair_off = L.start_off;
        L.pair_slots = L.entries * range;
    } else {
        L.pair_off = L.start_off + round_up(size_t(L.entries + 1) * 4, 256);
        L.pair_slots = total_cap;
    }
    L.bytes = L.pair_off + size_t(L.pair_slots) * 8;
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

// Adds `len` to counter e of the call of `epoch` and returns the count
// before the addition.
__device__ __forceinline__ uint32_t counter_add(unsigned long long *cnt, int64_t e, bool clean,
                                                uint64_t epoch, uint32_t len) {
    if (clean) return uint32_t(atomicAdd(&cnt[e], (unsigned long long)len) & kCountBits);
    return uint32_t(tagged_add(&cnt[e], counter_tag(epoch, uint64_t(e)), len));
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

// The status bits a workgroup noted, into the control block's flags word
// (tagged with the call's epoch: a flags word with another tag reads as 0).
__device__ __forceinline__ void note_flags(ApplyCtl *ctl, uint64_t epoch, uint32_t flags) {
    tagged_add(&ctl->flags, counter_tag(epoch, kFlagsTagIndex), 0);
    atomicOr(&ctl->flags, (unsigned long long)flags);
}

// A pair in a slot: (worker << kLog | index in range, value bits).
template <int kLog>
__device__ __forceinline__ uint2 make_pair(int w, int32_t i, float v) {
    return make_uint2((uint32_t(w) << kLog) | (uint32_t(i) & ((1u << kLog) - 1)), __float_as_uint(v));
}

// Workgroup (x, w) walks payload w in a grid-stride loop over kBlock pairs
// at a time.  kPlace: each valid pair goes to the next slot of its
// segment's bucket (bucketed layout); otherwise the pairs are only counted
// (packed layout).  Both note truncated payloads and indices outside
// [0, d); the first workgroup hands the call's epoch to the later launches.
template <bool kPlace>
__global__ __launch_bounds__(kBlock) void apply_group_kernel(Payloads p, int32_t n, int64_t d,
                                                             unsigned long long *__restrict__ cnt,
                                                             int64_t entries,
                                                             ApplyCtl *__restrict__ ctl,
                                                             uint2 *__restrict__ bucket) {
    constexpr int kLog = Geom<kPlace>::kLog;
    constexpr int kRange = Geom<kPlace>::kRange;
    __shared__ uint32_t s_flags;
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
    const float *__restrict__ val = p.val[w];
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t stride = int64_t(gridDim.x) * kBlock;
    bool bad = false;
    for (int64_t base = int64_t(blockIdx.x) * kBlock; base < c; base += stride) {
        const int64_t j = base + threadIdx.x;
        int32_t i = -1;
        float v = 0.0f;
        if (j < c) {
            i = idx[j];
            if (kPlace) v = val[j];
            bad = bad || i < 0 || int64_t(i) >= d;
        }
        const bool valid = i >= 0 && int64_t(i) < d;
        const uint32_t key = valid ? uint32_t(i) >> kLog : 0x80000000u + uint32_t(lane);
        const Run r = lane_run(key);
        const int64_t e = int64_t(key) * n + w;   // meaningful for valid lanes only
        uint32_t old = 0;
        if (valid && r.len > 0) old = counter_add(cnt, e, clean, epoch, uint32_t(r.len));
        if (kPlace) {
            const uint32_t slot = __shfl(old, r.leader) + uint32_t(lane - r.leader);
            // a slot past the bucket needs an index repeated within the payload
            if (valid && slot < uint32_t(kRange)) bucket[e * kRange + slot] = make_pair<kLog>(w, i, v);
        }
    }
    if (bad) atomicOr(&s_flags, kSparseBadIndex);
    __syncthreads();
    if (threadIdx.x == 0) {
        if (s_flags) note_flags(ctl, epoch, s_flags);
        if (blockIdx.x == 0 && w == 0) {
            ctl->run_epoch = epoch;
            ctl->run_clean = clean ? 1u : 0u;
        }
    }
}

// Packed layout, one workgroup: start[e] = the pairs of all segments before
// e (start[entries] = the total).  Tiles of kScanTile counters: coalesced
// loads (the next tile's in flight while the current one is scanned), the
// counts staged in LDS so that each thread scans kScanPer consecutive ones,
// the starts staged back and stored coalesced.  Two LDS buffers alternate,
// so one barrier per tile separates a tile's last reads from the next
// tile's writes.  The counters themselves are set up for the next call by
// the range pass.
constexpr int kScanBlock = 1024;
constexpr int kScanWaves = kScanBlock / kWave;
constexpr int kScanPer = 8;
constexpr int kScanTile = kScanPer * kScanBlock;

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

__global__ __launch_bounds__(kScanBlock) void apply_scan_kernel(
    const unsigned long long *__restrict__ cnt, uint32_t *__restrict__ start, int64_t entries,
    const ApplyCtl *__restrict__ ctl) {
    __shared__ __align__(16) uint32_t s_v[2][kScanTile];
    __shared__ uint32_t s_wave[kScanWaves];
    const int tid = threadIdx.x;
    const uint64_t epoch = ctl->run_epoch;
    const bool clean = ctl->run_clean != 0u;
    unsigned long long q[kScanPer];
#pragma unroll
    for (int i = 0; i < kScanPer; ++i) {
        const int64_t e = int64_t(i) * kScanBlock + tid;
        q[i] = e < entries ? cnt[e] : 0ull;
    }
    uint32_t carry = 0;
    int buf = 0;
    for (int64_t t0 = 0; t0 < entries; t0 += kScanTile, buf ^= 1) {
        uint32_t *sv = s_v[buf];
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            const int64_t e = t0 + int64_t(i) * kScanBlock + tid;
            const unsigned long long w = q[i];
            sv[i * kScanBlock + tid] =
                (e < entries && (clean || (w >> kEpochShift) == counter_tag(epoch, uint64_t(e))))
                    ? uint32_t(w & kCountBits) : 0u;
        }
        if (t0 + kScanTile < entries) {
#pragma unroll
            for (int i = 0; i < kScanPer; ++i) {
                const int64_t e = t0 + kScanTile + int64_t(i) * kScanBlock + tid;
                q[i] = e < entries ? cnt[e] : 0ull;
            }
        }
        __syncthreads();
        uint4 *mine = reinterpret_cast<uint4 *>(sv + kScanPer * tid);
        const uint4 a = mine[0], b = mine[1];
        uint32_t total;
        uint32_t run = carry + scan_block(a.x + a.y + a.z + a.w + b.x + b.y + b.z + b.w, s_wave,
                                          total);
        uint4 o;
        o.x = run;
        run += a.x;
        o.y = run;
        run += a.y;
        o.z = run;
        run += a.z;
        o.w = run;
        run += a.w;
        mine[0] = o;
        o.x = run;
        run += b.x;
        o.y = run;
        run += b.y;
        o.z = run;
        run += b.z;
        o.w = run;
        mine[1] = o;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kScanPer; ++i) {
            const int64_t e = t0 + int64_t(i) * kScanBlock + tid;
            if (e < entries) start[e] = sv[i * kScanBlock + tid];
        }
        carry += total;
    }
    if (tid == 0) start[entries] = carry;
}

// Packed layout: workgroup (x, w) places every valid pair of payload w: the
// leader of each run of equal ranges in a wave reserves the run's slots
// with one atomic on the segment's start.
__global__ __launch_bounds__(kBlock) void apply_scatter_kernel(Payloads p, int32_t n, int64_t d,
                                                               uint32_t *__restrict__ start,
                                                               uint2 *__restrict__ pairs,
                                                               int64_t pair_cap) {
    constexpr int kLog = Geom<false>::kLog;
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
        float v = 0.0f;
        if (j < c) {
            i = idx[j];
            v = val[j];
        }
        const bool valid = i >= 0 && int64_t(i) < d;
        const uint32_t key = valid ? uint32_t(i) >> kLog : 0x80000000u + uint32_t(lane);
        const Run r = lane_run(key);
        uint32_t old = 0;
        if (valid && r.len > 0) old = atomicAdd(&start[int64_t(key) * n + w], uint32_t(r.len));
        const uint32_t run_base = __shfl(old, r.leader);
        if (valid) {
            const int64_t pos = int64_t(run_base) + (lane - r.leader);
            if (pos < pair_cap) pairs[pos] = make_pair<kLog>(w, i, v);
        }
    }
}

__device__ __forceinline__ float average_of(float s, int32_t n, float fn) {
    return n > 1 ? __fdiv_rn(s, fn) : s;
}

// Momentum update of coordinates [r0, r0 + len) with the sums in acc4 (all
// of them, +0 where nothing was added); full ranges have kRange coordinates.
template <int kRange>
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

// LDS state of one workgroup of the range launch.  bound[w] .. bound[w + 1]
// are worker w's pairs of the range: slots of the packed array, or
// (bucketed) positions in the concatenation of the range's n buckets.
template <int kRange>
struct RangeShared {
    f32x4 acc4[kRange / 4];
    uint32_t claim[kRange / 32];
    int64_t bound[kMaxApplyWorkers + 1];
};

struct RangeArgs {
    const uint32_t *end;        // packed: segment ends after the scatter
    unsigned long long *cnt;    // the counters, set up here for the next call
    ApplyCtl *ctl;
    const uint2 *pairs;         // packed array or buckets
    int64_t pair_cap;           // slots of the packed array or of all buckets
    int32_t n;
    int64_t d, ranges;
    float *x, *m;
    float beta, gamma;
};

constexpr int kPairsPerThread = 4;
constexpr int64_t kPairBatch = int64_t(kPairsPerThread) * kBlock;

// The slot of the range's pair at position s of bound[0] .. bound[n].
template <bool kBucket>
__device__ __forceinline__ int64_t pair_slot(const int64_t *bound, int64_t s, int64_t b,
                                             int32_t n) {
    constexpr int kRange = Geom<kBucket>::kRange;
    if (!kBucket) return s;
    int lo = 0, hi = n;   // bound[lo] <= s < bound[hi]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (bound[mid] <= s)
            lo = mid;
        else
            hi = mid;
    }
    return (b * n + lo) * kRange + (s - bound[lo]);
}

// One workgroup per range b.  Wave 0 reads the range's bounds (its n
// counters, bucketed, or the segment ends around it, packed) and sets its
// counters up for the next call; the pairs are added into the LDS tile
// worker by worker, kPairBatch at a time with all loads of a batch in flight
// (a barrier between workers keeps every coordinate's sum in worker order),
// and the result is written: the average's whole tile (zeros where no pair
// falls), x -= avg at the touched coordinates, or the momentum update of
// every coordinate.  Workgroup 0 also publishes the call's status word and
// the next call's epoch: every launch that reads those words in this call
// has finished.
template <int kMode, bool kBucket>
__global__ __launch_bounds__(kBlock) void apply_range_kernel(RangeArgs a) {
    constexpr int kLog = Geom<kBucket>::kLog;
    constexpr int kRange = Geom<kBucket>::kRange;
    __shared__ RangeShared<kRange> sh;
    constexpr int kVec = kRange / 4 / kBlock;
    const int tid = threadIdx.x;
    const int32_t n = a.n;
    const float fn = float(n);
    const int64_t b = blockIdx.x;
    const uint64_t epoch = a.ctl->run_epoch;
    const uint64_t next = (epoch + 1) & kEpochMask;
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    float *acc = reinterpret_cast<float *>(sh.acc4);
    if (tid < kWave) {
        const int lane = tid;
        const int64_t e = b * n + lane;
        if (kBucket) {
            uint32_t c = 0;
            if (lane < n) {
                const unsigned long long word = a.cnt[e];
                if (a.ctl->run_clean != 0u || (word >> kEpochShift) == counter_tag(epoch, uint64_t(e)))
                    c = min(uint32_t(word & kCountBits), uint32_t(kRange));
            }
            const uint32_t incl = wave_inclusive_sum(c);
            if (lane < n) sh.bound[lane + 1] = incl;
            if (lane == 0) sh.bound[0] = 0;
        } else {
            if (lane < n) sh.bound[lane + 1] = min(int64_t(a.end[e]), a.pair_cap);
            if (lane == 0) sh.bound[0] = e > 0 ? min(int64_t(a.end[e - 1]), a.pair_cap) : 0;
        }
        if (lane < n) a.cnt[e] = counter_tag(next, uint64_t(e)) << kEpochShift;
        if (b == 0 && lane == 0) {
            ApplyCtl *ctl = a.ctl;
            const unsigned long long f = ctl->flags;
            ctl->status = (f >> kEpochShift) == counter_tag(epoch, kFlagsTagIndex)
                              ? uint32_t(f & 0xffu) : 0u;
            ctl->epoch = next;
            ctl->clean = clean_key(next, a.ranges * n);
        }
    }
    __syncthreads();
    const int64_t first = sh.bound[0];
    const int64_t last = max(first, sh.bound[n]);
    const bool sum = kMode == 2 || last > first;
    const int64_t r0 = b * kRange;
    const int64_t len = min(int64_t(kRange), a.d - r0);
    if (!sum) {
        if (kMode == 0) {
            if (len == kRange) {
                f32x4 *x4 = reinterpret_cast<f32x4 *>(a.x + r0);
#pragma unroll
                for (int q = 0; q < kVec; ++q) __builtin_nontemporal_store(z, x4 + q * kBlock + tid);
            } else {
                for (int64_t q = tid; q < len; q += kBlock) a.x[r0 + q] = 0.0f;
            }
        }
        return;
    }
    for (int q = tid; q < kRange / 4; q += kBlock) sh.acc4[q] = z;
    if (kMode == 1)
        for (int q = tid; q < kRange / 32; q += kBlock) sh.claim[q] = 0u;
    uint2 pr[kPairsPerThread];
    bool cleared = false;
    for (int64_t base = first; base < last; base += kPairBatch) {
#pragma unroll
        for (int q = 0; q < kPairsPerThread; ++q) {
            const int64_t s = base + q * kBlock + tid;
            pr[q] = s < last ? a.pairs[pair_slot<kBucket>(sh.bound, s, b, n)]
                             : make_uint2(0xFFFFFFFFu, 0u);
        }
        if (!cleared) {
            __syncthreads();   // the tile is clear
            cleared = true;
        }
        const int64_t shi = min(last, base + kPairBatch) - 1;
        int wlo = 0, whi = 0;
        while (wlo < n - 1 && base >= sh.bound[wlo + 1]) ++wlo;
        while (whi < n - 1 && shi >= sh.bound[whi + 1]) ++whi;
        for (int w = wlo; w <= whi; ++w) {
#pragma unroll
            for (int q = 0; q < kPairsPerThread; ++q) {
                if ((pr[q].x >> kLog) != uint32_t(w)) continue;
                const uint32_t li = pr[q].x & (kRange - 1);
                acc[li] = __fadd_rn(acc[li], __uint_as_float(pr[q].y));
            }
            __syncthreads();
        }
    }
    if (!cleared) __syncthreads();   // momentum of a range without pairs

    if (kMode == 2) {
        momentum_range<kRange>(sh.acc4, r0, len, n, a.x, a.m, a.beta, a.gamma);
    } else if (kMode == 0) {
        if (len == kRange) {
            f32x4 *x4 = reinterpret_cast<f32x4 *>(a.x + r0);
#pragma unroll
            for (int q = 0; q < kVec; ++q) {
                f32x4 v = sh.acc4[q * kBlock + tid];
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = average_of(v[c], n, fn);
                __builtin_nontemporal_store(v, x4 + q * kBlock + tid);
            }
        } else {
            for (int64_t q = tid; q < len; q += kBlock) a.x[r0 + q] = average_of(acc[q], n, fn);
        }
    } else {
        // x -= avg once at each touched coordinate
        const bool one_batch = last - first <= kPairBatch;
        for (int64_t base = first; base < last; base += kPairBatch) {
#pragma unroll
            for (int q = 0; q < kPairsPerThread; ++q) {
                const int64_t s = base + q * kBlock + tid;
                if (s >= last) continue;
                const uint32_t li =
                    (one_batch ? pr[q].x : a.pairs[pair_slot<kBucket>(sh.bound, s, b, n)].x) &
                    (kRange - 1);
                if (li >= uint32_t(len)) continue;
                const uint32_t bit = 1u << (li & 31u);
                const uint32_t was = atomicOr(&sh.claim[li >> 5], bit);
                if ((was & bit) == 0u)
                    a.x[r0 + li] = __fsub_rn(a.x[r0 + li], average_of(acc[li], n, fn));
            }
        }
    }
}

template <int kMode>
void launch_range(bool bucketed, uint32_t grid, const RangeArgs &a, hipStream_t stream) {
    if (bucketed)
        apply_range_kernel<kMode, true><<<grid, kBlock, 0, stream>>>(a);
    else
        apply_range_kernel<kMode, false><<<grid, kBlock, 0, stream>>>(a);
}

}  // namespace

size_t apply_workspace_size(int32_t n, int64_t d, int64_t total_cap) {
    return make_layout(n, d, total_cap, false).bytes;
}

size_t apply_bucket_workspace_size(int32_t n, int64_t d) {
    return make_layout(n, d, 0, true).bytes;
}

size_t apply_status_offset() { return offsetof(ApplyCtl, status); }

hipError_t launch_apply(const int32_t *const *idx, const float *const *val,
                        const uint32_t *const *counts, const int64_t *caps, int32_t n,
                        int64_t d, int mode, float *x, float *m, float beta, float gamma,
                        void *workspace, size_t workspace_bytes, hipStream_t stream) {
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
    const bool bucketed = workspace_bytes >= apply_bucket_workspace_size(n, d);
    const Layout L = make_layout(n, d, total, bucketed);
    char *ws = static_cast<char *>(workspace);
    ApplyCtl *ctl = reinterpret_cast<ApplyCtl *>(ws);
    unsigned long long *cnt = reinterpret_cast<unsigned long long *>(ws + L.cnt_off);
    uint32_t *start = reinterpret_cast<uint32_t *>(ws + L.start_off);
    uint2 *pairs = reinterpret_cast<uint2 *>(ws + L.pair_off);

    const int cus = device_cu_count();
    // about sixteen workgroups per CU over all workers, so that a payload's
    // chain of dependent accesses (count, pairs, counter atomic, slot) runs
    // once or twice per workgroup: payloads are usually far shorter than
    // their capacity, and a grid-stride loop covers the rest (at least one
    // workgroup per worker, so that every count is checked)
    const int64_t tiles = (max_cap + kBlock - 1) / kBlock;
    const int64_t per_worker = int64_t(cus) * 16 / n;
    int64_t gx = tiles < per_worker ? tiles : per_worker;
    gx = gx < 1 ? 1 : gx;
    const dim3 group_grid(static_cast<uint32_t>(gx), static_cast<uint32_t>(n));
    if (bucketed) {
        apply_group_kernel<true><<<group_grid, kBlock, 0, stream>>>(p, n, d, cnt, L.entries, ctl,
                                                                     pairs);
    } else {
        apply_group_kernel<false><<<group_grid, kBlock, 0, stream>>>(p, n, d, cnt, L.entries, ctl,
                                                                      nullptr);
        apply_scan_kernel<<<1, kScanBlock, 0, stream>>>(cnt, start, L.entries, ctl);
        if (max_cap > 0)
            apply_scatter_kernel<<<group_grid, kBlock, 0, stream>>>(p, n, d, start, pairs, total);
    }
    RangeArgs a;
    a.end = start;
    a.cnt = cnt;
    a.ctl = ctl;
    a.pairs = pairs;
    a.pair_cap = L.pair_slots;
    a.n = n;
    a.d = d;
    a.ranges = L.ranges;
    a.x = x;
    a.m = m;
    a.beta = beta;
    a.gamma = gamma;
    const uint32_t grid = uint32_t(L.ranges);
    if (mode == 0)
        launch_range<0>(bucketed, grid, a, stream);
    else if (mode == 1)
        launch_range<1>(bucketed, grid, a, stream);
    else
        launch_range<2>(bucketed, grid, a, stream);
    return hipGetLastError();
}

}  // namespace efs
