// Exact Top-k sparsifier with error feedback (Algorithm 1 with Top-k; the
// per-iteration optimum of Lemma 2).
//
// Keys are the 31-bit patterns of |p| (monotone in |p| for non-NaN values),
// ranked larger first and, on equal keys, lower index first.  Selection is a
// radix select (the paper notes radix select costs O(ceil(b/r) d), section 1)
// with a shortcut for error-feedback loops, where the k-th magnitude moves
// little from one iteration to the next.  Five launches, always all enqueued
// (work a call does not need returns at once):
//
//   reset  zero the control block and histograms; form the key bracket
//          [lo, hi] of 2^20 keys (about 3..6 % in magnitude either side;
//          2^21 keys for 16 calls after a threshold fell outside it)
//          around the threshold predicted from the previous two calls on
//          this workspace.
//   pass1  p = e + lr*g written into e (12 B/element, streamed with the
//          non-temporal hint); LDS histogram of key
//          bits 30..20; with a bracket, keys above it go straight to the
//          payload and keys inside it to a candidate buffer (staged
//          compaction) and into coarse (1024) and fine (one per key) histograms of
//          key - lo.
//   step3  every workgroup first decides the path: the bracket path only
//          when the counts prove the k-th key lies inside the bracket
//          (#(key > hi) <= k <= #(key >= lo), every bracket key collected),
//          and not when T is the key of zero with more ties to split than
//          the tie list holds (see below).
//          Bracket path: select T from the coarse then fine histogram, append
//          the candidates with key > T (all key == T too when no tie is
//          dropped), zero e at every kept coordinate.  Radix path: select the
//          top digit from the pass-1 histogram, then histogram bits 19..0 of
//          the keys under it (a 4 B/element read of p) into 1024 coarse and
//          2^20 fine bins.
//   step4  radix path: coarse then fine selection, so T is exact, then
//          one read of p that sends every key > T (and every key == T when
//          no tie is dropped).  When ties at T must be split
//          (0 < m < #(key == T)) and at most kTieList of them exist, they
//          are listed (radix path: in that read; bracket path: from the
//          candidates, which hold every key equal to T); with more, per-tile
//          counts of key == T.
//   emit   only the ties of index rank < m, when some are dropped: from the
//          list, one workgroup selects the m lowest indices; from per-tile
//          counts, a read of the tiles holding ties ranks them over the
//          vector (exclusive sums of the counts, each workgroup summing the
//          tiles before its own, then a block scan in index order inside
//          the tile); at T = 0 on the radix path that read covers every
//          tile and also clears e at the keys > T, which step 4 left as p.
//
// Selections made by every workgroup read the same histograms, so they agree;
// workgroup 0 records them in the control block.  Workgroups exchange data
// only through global atomics and kernel boundaries; none waits on another.
//
// Workspace (offsets 256-byte aligned):
//   control block (256 B) | histograms: 2048 top-digit bins, 1024 + 2^20
//   radix bins, 1024 + 2^21 bracket bins | per-tile tie counts | candidates
//   (int32 index, fp32 value) x ccap.
#include <stddef.h>

#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

constexpr int kBins1 = 2048;  // bits 30..20
constexpr int kCoarse = 1024; // coarse bins of a 20-bit range (1024 keys each)
constexpr int kFineBits = 20;
constexpr uint32_t kFine = 1u << kFineBits;        // radix path: bits 19..0
constexpr int kFinePerCoarse = int(kFine) / kCoarse;
// Bracket width in keys, one fine bin per key: kBracketNarrow, or
// kBracketWide for kWideCalls calls after a call whose threshold fell
// outside its bracket.  Under error feedback the threshold's step from one
// call to the next wanders by about half its size; a 2^20-key bracket
// missed it on 1 to 2 of 20 calls on the 25.6e6 and 1.5e9 workloads (each
// miss costs the radix path), a 2^21-key one on none after the first
// steps, at the price of twice the candidates (+3 us a call at 25.6e6).
constexpr uint32_t kBracketNarrow = 1u << 20;
constexpr uint32_t kBracketWide = 1u << 21;
constexpr uint32_t kWideCalls = 16;
// the extrapolated step is capped at kStepCap keys, or at kStepCapSteady
// when the step before went the same way and at least half as far
constexpr int64_t kStepCap = int64_t(1) << 18;
constexpr int64_t kStepCapSteady = int64_t(1) << 21;
constexpr uint32_t kHintMagic = 0x48494e54u;
constexpr int kStagePairs = 1024;
constexpr uint32_t kNoKey = 0xffffffffu;            // larger than every 31-bit key
// pass 1 workgroups per CU (measured: 3 beats 2 and 4 at 25.6e6 and 110e6)
constexpr int kPass1WorkgroupsPerCU = 3;
constexpr uint32_t kCandChunkMax = 4096;           // bracket candidates per step-3 work unit, at most
constexpr uint32_t kStep3Chunks = 512;             // step-3 work units aimed for

// Fields are written by workgroup 0 of one launch and read by later
// launches only, never by other workgroups of the launch that writes them.
struct TopkCtl {
    uint32_t p1, n1;      // radix path: top digit and the rank left under it (step 3)
    uint32_t pad0[2];
    uint32_t T;           // threshold key
    uint32_t m;           // tied elements (key == T) to keep
    uint32_t ties;        // elements with key == T
    uint32_t tie_mode;    // 1 when 0 < m < ties
    uint32_t fast;        // 1: bracket path
    uint32_t lo, hi;      // bracket of keys
    uint32_t bracket_on;  // pass 1 collected the bracket
    uint32_t above;       // bracket path: pairs pass 1 sent (key > hi)
    uint32_t ncand;       // bracket path: candidates collected
    uint32_t wide;        // 1: the bracket is kBracketWide keys wide
    uint32_t pad;
    unsigned long long emit;   // pass 1: pairs above the bracket (count in the low bits)
    unsigned long long cand;   // pass 1: bracket candidates
    unsigned long long emit2;  // pairs appended after pass 1 (steps 3 and emit)
    uint32_t last;             // threshold of the previous call (kNoKey if none)
    uint32_t tie_list;         // bracket path: keys equal to T listed by step 4
    // Kept across calls (not cleared by reset): the thresholds of the last
    // three calls, each valid when its magic word is set.
    uint32_t hint_key, hint_magic;
    uint32_t prev_key, prev_magic;
    uint32_t prev2_key, prev2_magic;
    // calls left with the wide bracket (valid when wide_magic is set)
    uint32_t wide_left, wide_magic;
};
static_assert(sizeof(TopkCtl) <= 256, "control block must fit its slot");
constexpr int kCtlClearWords = offsetof(TopkCtl, hint_key) / 4;
static_assert(offsetof(TopkCtl, hint_key) % 4 == 0, "control words are 32-bit");
static_assert(kCtlClearWords <= kBlock, "reset clears the control block with one workgroup");

constexpr size_t kCtlBytes = 256;
// radix path: 1024 coarse + 2^20 fine bins for bits 19..0; bracket path:
// 1024 coarse + up to 2^21 fine bins for key - lo (the fine bins last)
constexpr size_t kHistWords = kBins1 + 2 * size_t(kCoarse) + size_t(kFine) + size_t(kBracketWide);
constexpr size_t kHistBytes = sizeof(uint32_t) * kHistWords;
static_assert(kHistWords % 4 == 0, "histograms are cleared with 16-byte stores");

size_t round256(size_t b) { return (b + 255) & ~size_t(255); }

struct Workspace {
    TopkCtl *ctl;
    uint32_t *hist1, *rcoarse, *rfine, *coarse, *fine, *tile_ties;
    int32_t *cand_idx;
    float *cand_val;
    int32_t *ties;  // bracket path: indices of the keys equal to T
    uint32_t ccap;
};

// Bracket path with some keys equal to T dropped: the tied keys are all
// candidates, so up to this many are ranked from a list instead of a pass
// over the whole vector.
constexpr uint32_t kTieList = 16384;

// Candidate buffer size: the bracket around the k-th magnitude of an
// error-feedback vector holds several times k keys (about 8k measured on the
// segmented 25.6e6-element workload), so room for 16k.
int64_t candidate_capacity(int64_t d, int64_t k) {
    int64_t c = 16 * k;
    if (c < 262144) c = 262144;
    if (c > d) c = d;
    if (c < 1) c = 1;
    return c;
}

Workspace carve(void *ws, int64_t d, int64_t k) {
    char *b = static_cast<char *>(ws);
    const int64_t tiles = d > 0 ? (d + kTile - 1) / kTile : 1;
    Workspace w;
    w.ctl = reinterpret_cast<TopkCtl *>(b);
    w.hist1 = reinterpret_cast<uint32_t *>(b + kCtlBytes);
    w.rcoarse = w.hist1 + kBins1;
    w.rfine = w.rcoarse + kCoarse;
    w.coarse = w.rfine + kFine;
    w.fine = w.coarse + kCoarse;
    size_t off = kCtlBytes + round256(kHistBytes);
    w.tile_ties = reinterpret_cast<uint32_t *>(b + off);
    off += round256(sizeof(uint32_t) * size_t(tiles));
    w.ccap = uint32_t(candidate_capacity(d, k));
    w.cand_idx = reinterpret_cast<int32_t *>(b + off);
    off += round256(sizeof(int32_t) * size_t(w.ccap));
    w.cand_val = reinterpret_cast<float *>(b + off);
    off += round256(sizeof(float) * size_t(w.ccap));
    w.ties = reinterpret_cast<int32_t *>(b + off);
    return w;
}

// Loads the 16 values of a tile for this thread (index = tile0 + (j * kBlock
// + tid) * 4 + c, the hard-threshold kernel's map).  Elements past d read as
// zero and are cleared in `valid`.
template <bool kVector>
__device__ __forceinline__ void load_tile(const float *__restrict__ src, int64_t tile0,
                                          int64_t d, float (&v)[kVecPerThread][4],
                                          uint32_t &valid) {
    const int tid = threadIdx.x;
    if (kVector && tile0 + kTile <= d) {
        const f32x4 *s4 = reinterpret_cast<const f32x4 *>(src + tile0);
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
            const f32x4 x = s4[j * kBlock + tid];
#pragma unroll
            for (int c = 0; c < 4; ++c) v[j][c] = x[c];
        }
        valid = 0xffffu;
    } else {
        valid = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t i = tile0 + int64_t(j * kBlock + tid) * 4 + c;
                v[j][c] = 0.0f;
                if (i < d) {
                    v[j][c] = src[i];
                    valid |= 1u << (4 * j + c);
                }
            }
        }
    }
}

__device__ __forceinline__ int64_t elem_index(int64_t tile0, int j, int c) {
    return tile0 + int64_t(j * kBlock + int(threadIdx.x)) * 4 + c;
}

// Inclusive sum of v over the lanes of the wave up to this one.
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t o = __shfl_up(v, off);
        if (lane >= off) v += o;
    }
    return v;
}

// Called by every thread of one workgroup.  Bins are ranked from the top
// (highest bin first); finds the bin where the running count first reaches
// `need` (1 <= need <= sum of bins) and writes {bin, count above the bin,
// count in the bin} to s_out ({0, 0, 0} if no bin qualifies).  A wave scan
// of per-thread sums, then one exchange of wave totals: two barriers.
template <int kBins>
__device__ void select_bin(const uint32_t *hist, uint32_t need, uint32_t *s_scan,
                           uint32_t *s_out) {
    constexpr int kPer = kBins / kBlock;
    static_assert(kPer >= 1 && kBins % kBlock == 0, "whole bins per thread");
    const int t = threadIdx.x;
    const int lane = t & (kWave - 1);
    const int wave = t / kWave;
    if (t == 0) {
        s_out[0] = 0u;
        s_out[1] = 0u;
        s_out[2] = 0u;
    }
    uint32_t c[kPer];
    uint32_t tot = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        c[i] = hist[kBins - 1 - (t * kPer + i)];
        tot += c[i];
    }
    const uint32_t incl_w = wave_inclusive_sum(tot);
    if (lane == kWave - 1) s_scan[wave] = incl_w;
    __syncthreads();
    uint32_t off = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) off += q < wave ? s_scan[q] : 0u;
    const uint32_t incl = off + incl_w;
    const uint32_t excl = incl - tot;
    if (excl < need && incl >= need) {
        uint32_t run = excl;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            if (run + c[i] >= need) {
                s_out[0] = uint32_t(kBins - 1 - (t * kPer + i));
                s_out[1] = run;
                s_out[2] = c[i];
                break;
            }
            run += c[i];
        }
    }
    __syncthreads();
}

// Zeroes the control block (except the hints) and every histogram, and
// forms the bracket: 2^20 or 2^21 keys centred on the threshold predicted from the
// last calls (the last threshold plus the last step in key space, the step
// capped at 2^18 keys, or at 2^21 during a steady drift; the last threshold
// alone when only one is known).  Grid-stride over the histogram words.
__global__ __launch_bounds__(kBlock) void topk_reset_kernel(Workspace ws) {
    // read by every workgroup (kept across calls; this launch writes none
    // of them)
    const bool hinted = ws.ctl->hint_magic == kHintMagic;
    const bool wide = hinted && ws.ctl->wide_magic == kHintMagic && ws.ctl->wide_left > 0u;
    const uint32_t width = wide ? kBracketWide : kBracketNarrow;
    if (blockIdx.x == 0) {
        uint32_t *w = reinterpret_cast<uint32_t *>(ws.ctl);
        if (int(threadIdx.x) < kCtlClearWords) w[threadIdx.x] = 0u;
        __syncthreads();
        if (threadIdx.x == 0) {
            TopkCtl *c = ws.ctl;
            c->last = kNoKey;
            if (c->hint_magic == kHintMagic) {
                // the step since the previous call, capped at an eighth of
                // the bracket (so the last threshold stays inside it), or
                // at the bracket's width when the step before went the same
                // way and at least half as far: a steady drift of up to
                // ~18 % in |p| per call is then followed
                const int64_t h1 = int64_t(c->hint_key & 0x7fffffffu);
                int64_t pred = h1;
                if (c->prev_magic == kHintMagic) {
                    const int64_t h0 = int64_t(c->prev_key & 0x7fffffffu);
                    int64_t step = h1 - h0;
                    int64_t cap = kStepCap;
                    if (c->prev2_magic == kHintMagic) {
                        const int64_t before = h0 - int64_t(c->prev2_key & 0x7fffffffu);
                        const bool same_way = (step > 0 && before > 0) || (step < 0 && before < 0);
                        const int64_t as = step < 0 ? -step : step;
                        const int64_t ab = before < 0 ? -before : before;
                        if (same_way && 2 * ab >= as) cap = kStepCapSteady;
                    }
                    step = step > cap ? cap : (step < -cap ? -cap : step);
                    pred = h1 + step;
                    if (pred < 0) pred = 0;
                    if (pred > 0x7fffffff) pred = 0x7fffffff;
                }
                const uint32_t p = uint32_t(pred);
                const uint32_t lo = p > width / 2 ? p - width / 2 : 0u;
                c->last = uint32_t(h1);
                c->lo = lo;
                c->hi = lo + (width - 1);
                c->wide = wide ? 1u : 0u;
                c->bracket_on = 1u;
            }
        }
    }
    // the histograms up to the bracket's fine bins, and as many of those as
    // the bracket has keys
    f32x4 *h4 = reinterpret_cast<f32x4 *>(ws.hist1);
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    const size_t n4 = (kHistWords - kBracketWide + (hinted ? width : 0u)) / 4;
    for (size_t i = size_t(blockIdx.x) * kBlock + threadIdx.x; i < n4;
         i += size_t(gridDim.x) * kBlock)
        h4[i] = z;
}

// Adds 1 to hist[bin] for every active lane of the wave; the lanes that share
// the first active lane's bin add together with one atomic (a vector of equal
// magnitudes costs one atomic per wave, not 64).  Called by all lanes.
__device__ __forceinline__ void wave_aggregated_add(uint32_t *hist, uint32_t bin, bool active) {
    const uint64_t act = __ballot(active);
    if (act == 0) return;
    const int leader = __ffsll(static_cast<unsigned long long>(act)) - 1;
    const uint32_t lbin = __shfl(bin, leader);
    const bool same = active && bin == lbin;
    const uint64_t mates = __ballot(same);
    if (same) {
        if (int(threadIdx.x & (kWave - 1)) == leader) atomicAdd(hist + lbin, uint32_t(__popcll(mates)));
    } else if (active) {
        atomicAdd(hist + bin, 1u);
    }
}

// Adds 1 to fine[(key - sub) mod kBins] for every element (j, c) of this
// thread selected by bit 4*j + c of `mask`.  Each round takes the lowest
// remaining selected element of every lane, so a wave runs as many rounds as
// its fullest lane has selected elements (usually none or a few) instead of
// one per element slot.  Called by all lanes.
template <uint32_t kBins>
__device__ __forceinline__ void fine_add_masked(uint32_t *fine, uint32_t mask,
                                                const float (&p)[kVecPerThread][4],
                                                uint32_t sub) {
    while (__ballot(mask != 0u) != 0ull) {
        const bool act = mask != 0u;
        uint32_t key = 0u;
        if (act) {
            const int b = __ffs(mask) - 1;
            mask &= mask - 1u;
            float x = 0.0f;
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    if (b == 4 * j + c) x = p[j][c];
            key = magnitude_key(x);
        }
        wave_aggregated_add(fine, (key - sub) & (kBins - 1), act);
    }
}

struct Pass1Shared {
    uint32_t h[kBins1];
    uint32_t coarse[kCoarse];
    PairStageN<kStagePairs> above;   // keys above the bracket -> payload
    PairStageN<kStagePairs> inside;  // keys in the bracket -> candidates
};

template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_pass1_kernel(const float *__restrict__ g,
                                                            float *__restrict__ e, int64_t d,
                                                            float lr, uint32_t ntiles, uint32_t k,
                                                            int32_t *__restrict__ idx,
                                                            float *__restrict__ val,
                                                            Workspace ws) {
    __shared__ Pass1Shared sh;
    const int tid = threadIdx.x;
    const bool bracket = ws.ctl->bracket_on != 0u;
    const uint32_t lo = ws.ctl->lo, hi = ws.ctl->hi;
    // coarse bins of 1024 or 2048 keys (kCoarse of them span the bracket)
    const uint32_t coarse_shift = ws.ctl->wide != 0u ? 11u : 10u;
    for (int b = tid; b < kBins1; b += kBlock) sh.h[b] = 0u;
    for (int b = tid; b < kCoarse; b += kBlock) sh.coarse[b] = 0u;
    __syncthreads();
    uint32_t fill_above = 0, fill_inside = 0;

    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float p[kVecPerThread][4];
        uint32_t valid;
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
                f32x4 o;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    o[c] = ef_accumulate(ev[j][c], lr, gv[j][c]);
                    p[j][c] = o[c];
                }
                __builtin_nontemporal_store(o, e4 + j * kBlock + tid);
            }
            valid = 0xffffu;
        } else {
            valid = 0;
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int64_t i = elem_index(tile0, j, c);
                    p[j][c] = 0.0f;
                    if (i < d) {
                        p[j][c] = ef_accumulate(e[i], lr, g[i]);
                        e[i] = p[j][c];
                        valid |= 1u << (4 * j + c);
                    }
                }
            }
        }
        uint32_t m_above = 0, m_inside = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int b = 4 * j + c;
                if ((valid >> b) & 1u) {
                    const uint32_t key = magnitude_key(p[j][c]);
                    atomicAdd(&sh.h[key >> 20], 1u);
                    if (bracket) {
                        const bool in = key >= lo && key <= hi;
                        m_above |= uint32_t(key > hi) << b;
                        m_inside |= uint32_t(in) << b;
                        if (in) atomicAdd(&sh.coarse[(key - lo) >> coarse_shift], 1u);
                    }
                }
            }
        }
        // fine bins in global memory: lanes with equal keys add together
        if (bracket) fine_add_masked<kBracketWide>(ws.fine, m_inside, p, lo);
        if (bracket) {
            stage_mask(sh.above, fill_above, m_above, p, tile0, &ws.ctl->emit, k, idx, val);
            stage_mask(sh.inside, fill_inside, m_inside, p, tile0, &ws.ctl->cand, ws.ccap,
                       ws.cand_idx, ws.cand_val);
        }
    }
    if (bracket) {
        stage_flush(sh.above, fill_above, false, &ws.ctl->emit, nullptr, k, idx, val);
        stage_flush(sh.inside, fill_inside, false, &ws.ctl->cand, nullptr, ws.ccap, ws.cand_idx,
                    ws.cand_val);
    }
    __syncthreads();
    for (int b = tid; b < kBins1; b += kBlock)
        if (sh.h[b]) atomicAdd(ws.hist1 + b, sh.h[b]);
    if (bracket)
        for (int b = tid; b < kCoarse; b += kBlock)
            if (sh.coarse[b]) atomicAdd(ws.coarse + b, sh.coarse[b]);
}

// Radix path: histograms of bits 19..0 of the keys whose bits 30..20 equal
// `prefix`: bits 19..10 in 1024 coarse bins (LDS, then merged), all twenty
// bits in 2^20 fine bins (global).
template <bool kVector>
__device__ void radix_refine20(const float *__restrict__ e, int64_t d, uint32_t ntiles,
                               uint32_t prefix, uint32_t *coarse, uint32_t *fine, uint32_t *h) {
    const int tid = threadIdx.x;
    for (int b = tid; b < kCoarse; b += kBlock) h[b] = 0u;
    __syncthreads();
    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float v[kVecPerThread][4];
        uint32_t valid;
        load_tile<kVector>(e, tile0, d, v, valid);
        uint32_t under = 0;  // elements whose key lies under the top digit
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t key = magnitude_key(v[j][c]);
                const bool in = ((valid >> (4 * j + c)) & 1u) && (key >> 20) == prefix;
                if (in) atomicAdd(&h[(key >> 10) & (kCoarse - 1)], 1u);
                under |= uint32_t(in) << (4 * j + c);
            }
        }
        fine_add_masked<kFine>(fine, under, v, 0u);
    }
    __syncthreads();
    for (int b = tid; b < kCoarse; b += kBlock)
        if (h[b]) atomicAdd(coarse + b, h[b]);
}

// Threshold and tie bookkeeping, written by workgroup 0 once T is exact; T
// and the previous call's threshold are kept for the next call's bracket.
__device__ __forceinline__ void set_threshold(TopkCtl *c, uint32_t T, uint32_t m, uint32_t ties) {
    c->T = T;
    c->m = m;
    c->ties = ties;
    c->tie_mode = m < ties ? 1u : 0u;
    c->prev2_key = c->prev_key;
    c->prev2_magic = c->last != kNoKey ? c->prev_magic : 0u;
    c->prev_key = c->last;
    c->prev_magic = c->last != kNoKey ? kHintMagic : 0u;
    c->hint_key = T;
    c->hint_magic = kHintMagic;
}

struct SelectShared {
    uint32_t scan[kBlock];
    uint32_t sel[4];
};

// Step 3: path decision, then the bracket path's selection and emission or
// the radix path's second digit histogram.
template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_step3_kernel(float *__restrict__ e, int64_t d,
                                                            uint32_t ntiles, uint32_t k,
                                                            int32_t *__restrict__ idx,
                                                            float *__restrict__ val,
                                                            Workspace ws) {
    __shared__ SelectShared ss;
    __shared__ uint32_t h[1024];
    __shared__ uint32_t s_wave[kWaves];
    __shared__ unsigned long long s_base;
    TopkCtl *c = ws.ctl;
    const int tid = threadIdx.x;
    const bool lead = blockIdx.x == 0 && tid == 0;
    const uint64_t above = c->emit & kCountMask;
    const uint64_t inside = c->cand & kCountMask;
    bool fast = c->bracket_on != 0u && above <= k && above + inside >= k && inside <= ws.ccap;
    if (lead) {
        // the next calls' bracket width: wide for kWideCalls calls after the
        // threshold fell outside this call's bracket, narrow at once after a
        // bracket that held more keys than the candidate buffer
        const bool outside = c->bracket_on != 0u && (above > k || above + inside < k);
        const bool overfull = c->bracket_on != 0u && inside > ws.ccap;
        const uint32_t left = c->wide_magic == kHintMagic ? c->wide_left : 0u;
        c->wide_left = outside ? kWideCalls : (overfull || left == 0u ? 0u : left - 1u);
        c->wide_magic = kHintMagic;
    }

    // Bracket path: rank `need` among the candidates, coarse then fine.
    const uint32_t need = fast ? k - uint32_t(above) : 0u;
    uint32_t T = kNoKey, m = 0u, ties = 0u;
    if (need > 0u) {
        select_bin<kCoarse>(ws.coarse, need, ss.scan, ss.sel);
        const uint32_t cb = ss.sel[0], above_c = ss.sel[1];
        __syncthreads();
        if (c->wide != 0u) {
            constexpr int kPer = int(kBracketWide) / kCoarse;
            select_bin<kPer>(ws.fine + size_t(cb) * kPer, need - above_c, ss.scan, ss.sel);
            T = c->lo + cb * uint32_t(kPer) + ss.sel[0];
        } else {
            constexpr int kPer = int(kBracketNarrow) / kCoarse;
            select_bin<kPer>(ws.fine + size_t(cb) * kPer, need - above_c, ss.scan, ss.sel);
            T = c->lo + cb * uint32_t(kPer) + ss.sel[0];
        }
        m = need - above_c - ss.sel[1];
        ties = ss.sel[2];
        __syncthreads();  // ss.sel is rewritten below
        // Ties beyond the list are ranked by a scan of e after this kernel,
        // and this kernel sets e to +0 at every pair it keeps; when T is the
        // key of zero those cleared coordinates would read as ties.  The
        // radix path ranks the ties before anything is cleared.
        if (T == 0u && m < ties && ties > kTieList) fast = false;
    }
    if (!fast) {
        // the pairs pass 1 sent are ignored: the radix path writes the whole
        // payload from slot 0 in the emit launch
        select_bin<kBins1>(ws.hist1, k, ss.scan, ss.sel);
        const uint32_t prefix = ss.sel[0];
        if (lead) {
            c->fast = 0u;
            c->p1 = prefix;
            c->n1 = k - ss.sel[1];
        }
        radix_refine20<kVector>(e, d, ntiles, prefix, ws.rcoarse, ws.rfine, h);
        return;
    }

    const bool all_ties = m >= ties;
    if (lead) {
        c->fast = 1u;
        c->above = uint32_t(above);
        c->ncand = uint32_t(inside);
        if (need > 0u) {
            set_threshold(c, T, m, ties);
        } else {  // pass 1 already sent exactly k pairs
            c->T = kNoKey;
            c->m = 0u;
            c->ties = 0u;
            c->tie_mode = 0u;
        }
    }
    // pairs pass 1 sent: zero their residuals (above <= k, so all were written)
    for (uint32_t j = blockIdx.x * kBlock + tid; j < uint32_t(above); j += gridDim.x * kBlock)
        e[idx[j]] = 0.0f;
    // candidates: chunks of `per` candidates per thread, one block-wide prefix
    // and one atomic on the shared payload counter per chunk; `per` grows
    // with the candidate count so that about kStep3Chunks chunks take it (an
    // atomic per workgroup per kBlock candidates serialises on that one
    // address at millions of candidates, while too few chunks leave most
    // workgroups idle)
    constexpr int kPer = kCandChunkMax / kBlock;
    const uint32_t n = uint32_t(inside);
    const uint32_t per = min(uint32_t(kPer), max(1u, (n + kStep3Chunks * kBlock - 1) /
                                                         (kStep3Chunks * kBlock)));
    const uint32_t chunk = per * kBlock;
    for (uint32_t base = blockIdx.x * chunk; base < n; base += gridDim.x * chunk) {
        int32_t ci[kPer];
        float cv[kPer];
        uint32_t keep = 0;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const uint32_t j = base + uint32_t(u * kBlock + tid);
            ci[u] = 0;
            cv[u] = 0.0f;
            if (uint32_t(u) < per && j < n) {
                ci[u] = ws.cand_idx[j];
                cv[u] = ws.cand_val[j];
                const uint32_t key = magnitude_key(cv[u]);
                keep |= uint32_t(key > T || (all_ties && key == T)) << u;
            }
        }
        uint32_t total;
        const uint32_t pos = block_prefix_small(uint32_t(__popc(keep)), s_wave, total);
        if (total == 0) continue;
        if (tid == 0) s_base = atomicAdd(&c->emit2, (unsigned long long)total) & kCountMask;
        __syncthreads();
        uint64_t o = above + s_base + pos;
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            if ((keep >> u) & 1u) {
                if (o < k) {
                    idx[o] = ci[u];
                    val[o] = cv[u];
                }
                e[ci[u]] = 0.0f;
                ++o;
            }
        }
        __syncthreads();  // s_base is reused by the next chunk
    }
}

// Step 4.  Radix path: coarse then fine selection of bits 19..0 (T exact),
// then one sweep of p that appends every key > T to the payload (and the
// keys equal to T when all of them are kept) and, when ties at T must be
// split, lists the tied indices (at most kTieList of them) or counts them
// per tile (more).  Bracket path, ties to split: the tied candidates listed
// (at most kTieList), else per-tile tie counts.
template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_step4_kernel(float *__restrict__ e, int64_t d,
                                                            uint32_t ntiles,
                                                            int32_t *__restrict__ idx,
                                                            float *__restrict__ val, uint64_t cap,
                                                            Workspace ws) {
    __shared__ PairStage st;
    __shared__ SelectShared ss;
    TopkCtl *c = ws.ctl;
    const uint32_t lane = threadIdx.x & (kWave - 1);
    uint32_t T, tie_mode, ties;
    const bool radix = c->fast == 0u;
    if (radix) {
        const uint32_t need = c->n1;
        select_bin<kCoarse>(ws.rcoarse, need, ss.scan, ss.sel);
        const uint32_t cb = ss.sel[0], above_c = ss.sel[1];
        __syncthreads();
        select_bin<kFinePerCoarse>(ws.rfine + size_t(cb) * kFinePerCoarse, need - above_c,
                                   ss.scan, ss.sel);
        T = (c->p1 << 20) | (cb << 10) | ss.sel[0];
        const uint32_t m = need - above_c - ss.sel[1];
        ties = ss.sel[2];
        tie_mode = m < ties ? 1u : 0u;
        if (blockIdx.x == 0 && threadIdx.x == 0) set_threshold(c, T, m, ties);
    } else {
        T = c->T;
        tie_mode = c->tie_mode;
        ties = c->ties;
    }
    const bool list = tie_mode != 0u && ties <= kTieList;
    if (!radix) {
        if (tie_mode == 0u) return;
        if (list) {
            // every key equal to T is a candidate; list them
            const uint32_t n = c->ncand;
            const uint32_t stride = gridDim.x * kBlock;
            for (uint32_t base = blockIdx.x * kBlock; base < n; base += stride) {
                const uint32_t j = base + threadIdx.x;
                const bool tie = j < n && magnitude_key(ws.cand_val[j]) == T;
                const uint64_t mask = __ballot(tie);
                if (mask == 0) continue;
                uint32_t slot = 0;
                if (lane == 0) slot = atomicAdd(&c->tie_list, uint32_t(__popcll(mask)));
                slot = __shfl(slot, 0) + lanes_below(mask);
                if (tie && slot < kTieList) ws.ties[slot] = ws.cand_idx[j];
            }
            return;
        }
    }
    // A sweep of p: radix path, the payload's keys > T (all of it when no
    // tie is dropped) from slot 0; either path with many ties to split, the
    // per-tile tie counts.  e is cleared at the sent keys at once, except
    // with per-tile counts at T = 0: the emission ranks ties by scanning e
    // for T, where cleared coordinates would read as ties, so it clears
    // them itself.
    const bool counts = tie_mode != 0u && !list;
    const bool clear_now = !counts || T != 0u;
    uint32_t fill = 0;
    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float v[kVecPerThread][4];
        uint32_t valid;
        load_tile<kVector>(e, tile0, d, v, valid);
        uint32_t keep = 0, tie = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
                const int b = 4 * j + cc;
                const uint32_t key = magnitude_key(v[j][cc]);
                const bool ok = (valid >> b) & 1u;
                keep |= uint32_t(ok && (key > T || (tie_mode == 0u && key == T))) << b;
                tie |= uint32_t(ok && key == T) << b;
            }
        if (counts) {
            uint32_t total;
            block_prefix_small(uint32_t(__popc(tie)), st.wave, total);
            if (threadIdx.x == 0) ws.tile_ties[tile] = total;
        } else if (tie_mode != 0u && __ballot(tie != 0u) != 0ull) {
            // list the tied indices of this wave, slot by slot
#pragma unroll
            for (int b = 0; b < 16; ++b) {
                const bool t = (tie >> b) & 1u;
                const uint64_t mask = __ballot(t);
                if (mask == 0) continue;
                uint32_t slot = 0;
                if (lane == 0) slot = atomicAdd(&c->tie_list, uint32_t(__popcll(mask)));
                slot = __shfl(slot, 0) + lanes_below(mask);
                if (t && slot < kTieList) ws.ties[slot] = int32_t(elem_index(tile0, b / 4, b % 4));
            }
        }
        if (!radix) continue;
        stage_mask(st, fill, keep, v, tile0, &c->emit2, cap, idx, val);
        if (clear_now) {
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
                for (int cc = 0; cc < 4; ++cc)
                    if ((keep >> (4 * j + cc)) & 1u) e[elem_index(tile0, j, cc)] = 0.0f;
        }
    }
    if (radix) stage_flush(st, fill, false, &c->emit2, nullptr, cap, idx, val);
}

// Sum of tile_ties[lo, hi) over the workgroup.
__device__ __forceinline__ uint32_t tie_count_range(const uint32_t *tile_ties, uint32_t lo,
                                                    uint32_t hi, uint32_t *s_wave) {
    uint32_t v = 0;
    for (uint32_t i = lo + threadIdx.x; i < hi; i += kBlock) v += tile_ties[i];
    return block_sum(v, s_wave);
}

// Bracket path, some ties dropped: the m lowest of the n listed tie
// indices by a radix select on the index (bits 30..20, 19..10, 9..0; bins
// stored reversed so the top-down select_bin picks from the bottom), then
// emitted after the pairs already sent.  One workgroup.
__device__ void emit_listed_ties(const Workspace &ws, uint32_t m, float *e, int32_t *idx,
                                 float *val, uint64_t cap, PairStage &st, SelectShared &ss) {
    const int tid = threadIdx.x;
    const uint32_t n = min(ws.ctl->tie_list, kTieList);
    uint32_t *h = reinterpret_cast<uint32_t *>(st.idx);  // 2048 words of the unused stage
    uint32_t prefix = 0, rem = m;
#pragma unroll 1
    for (int level = 0; level < 3; ++level) {
        const int shift = 20 - 10 * level;
        const uint32_t bins = level == 0 ? 2048u : 1024u;
        for (uint32_t b = tid; b < 2048u; b += kBlock) h[b] = 0u;
        __syncthreads();
        for (uint32_t j = tid; j < n; j += kBlock) {
            const uint32_t i = uint32_t(ws.ties[j]);
            if (level > 0 && (i >> (shift + 10)) != prefix) continue;
            atomicAdd(&h[bins - 1u - ((i >> shift) & (bins - 1u))], 1u);
        }
        __syncthreads();
        if (level == 0) select_bin<2048>(h, rem, ss.scan, ss.sel);
        else select_bin<1024>(h, rem, ss.scan, ss.sel);
        prefix = (prefix << (level == 0 ? 11 : 10)) | (bins - 1u - ss.sel[0]);
        rem -= ss.sel[1];
        __syncthreads();
    }
    const uint32_t imax = prefix;
    for (uint32_t j = tid; j < n; j += kBlock) {
        const int32_t i = ws.ties[j];
        if (uint32_t(i) > imax) continue;
        const uint64_t o = atomicAdd(&ws.ctl->emit2, 1ull) & kCountMask;
        if (o < cap) {
            idx[o] = i;
            val[o] = e[i];
        }
        e[i] = 0.0f;
    }
}

// Final emission: the ties of rank < m when some are dropped (every other
// kept pair is already sent, by step 3 on the bracket path and by step 4 on
// the radix path); returns at once otherwise.  Listed ties: one workgroup
// keeps the m lowest indices.  Counted ties: a sweep ranks them in index
// order, reading only the tiles that hold ties, except at T = 0 on the
// radix path, where it also clears e at the keys > T (step 4 left them as p)
// and so reads every tile.
template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_emit_kernel(float *__restrict__ e, int64_t d,
                                                           int32_t *__restrict__ idx,
                                                           float *__restrict__ val,
                                                           uint64_t cap, uint32_t ntiles,
                                                           Workspace ws) {
    __shared__ PairStage st;
    __shared__ SelectShared ss;
    const bool fast = ws.ctl->fast != 0u;
    const bool tie_mode = ws.ctl->tie_mode != 0u;
    if (!tie_mode) return;
    const uint32_t T = ws.ctl->T;
    const uint32_t m = ws.ctl->m;
    // Radix path: the whole payload from slot 0.  Bracket path: after the
    // pairs of pass 1 (above) and step 3 (counted in emit2).
    const uint64_t base = fast ? ws.ctl->above : 0u;
    idx += base;
    val += base;
    cap -= base;
    if (ws.ctl->ties <= kTieList) {
        // the ties step 4 listed: workgroup 0 keeps the m lowest indices
        if (blockIdx.x == 0) emit_listed_ties(ws, m, e, idx, val, cap, st, ss);
        return;
    }
    uint32_t fill = 0;
    // ties in the tiles before this workgroup's current tile
    uint32_t ties_before = 0, counted_to = 0;

    const bool every_tile = !fast && T == 0u;
    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        if (!every_tile && ws.tile_ties[tile] == 0u) continue;  // the same in every thread
        const int64_t tile0 = int64_t(tile) * kTile;
        float v[kVecPerThread][4];
        uint32_t valid;
        load_tile<kVector>(e, tile0, d, v, valid);
        uint32_t keep = 0, tie = 0, above = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int b = 4 * j + c;
                const uint32_t key = magnitude_key(v[j][c]);
                const bool ok = (valid >> b) & 1u;
                above |= uint32_t(ok && every_tile && key > T) << b;
                tie |= uint32_t(ok && key == T) << b;
            }
        }
        // Rank of each tied element in index order: earlier tiles, then
        // earlier vector slots j (all lower indices), then lower threads in
        // slot j, then lower c within the thread.
        ties_before += tie_count_range(ws.tile_ties, counted_to, tile, st.wave);
        counted_to = tile;
        uint32_t rank = ties_before;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
            const uint32_t tj = (tie >> (4 * j)) & 0xfu;
            uint32_t slot_total;
            uint32_t r = rank + block_prefix_small(__popc(tj), st.wave, slot_total);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((tj >> c) & 1u) {
                    keep |= uint32_t(r < m) << (4 * j + c);
                    ++r;
                }
            }
            rank += slot_total;
        }
        stage_mask(st, fill, keep, v, tile0, &ws.ctl->emit2, cap, idx, val);
        const uint32_t clear = keep | above;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if ((clear >> (4 * j + c)) & 1u) e[elem_index(tile0, j, c)] = 0.0f;
    }
    stage_flush(st, fill, false, &ws.ctl->emit2, nullptr, cap, idx, val);
}

}  // namespace

size_t topk_path_flag_offset() { return offsetof(TopkCtl, fast); }

size_t topk_workspace_size(int64_t d, int64_t k) {
    const int64_t tiles = d > 0 ? (d + kTile - 1) / kTile : 1;
    const int64_t ccap = candidate_capacity(d, k);
    return kCtlBytes + round256(kHistBytes) + round256(sizeof(uint32_t) * size_t(tiles)) +
           round256(sizeof(int32_t) * kTieList) +
           round256(sizeof(int32_t) * size_t(ccap)) + round256(sizeof(float) * size_t(ccap));
}

hipError_t launch_topk(const float *g, float *e, int64_t d, float lr, int64_t k,
                       int32_t *idx, float *val, void *workspace, hipStream_t stream) {
    if (d == 0) return hipSuccess;
    const uint32_t ntiles = uint32_t((d + kTile - 1) / kTile);
    const uint32_t grid = balanced_grid(ntiles, kScanWorkgroupsPerCU);
    const uint32_t sgrid = balanced_grid(ntiles, kStageWorkgroupsPerCU);
    const uint32_t pgrid = balanced_grid(ntiles, kPass1WorkgroupsPerCU);
    const Workspace ws = carve(workspace, d, k);
    const uint32_t kk = uint32_t(k);
    const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(e)) & 15u) == 0;

    // 8.4 MB of histograms to zero (12.6 MB with the wide bracket): enough
    // workgroups to stream it (64 took 1 us longer per call)
    topk_reset_kernel<<<persistent_grid(1024), kBlock, 0, stream>>>(ws);
    if (vec)
        topk_pass1_kernel<true><<<pgrid, kBlock, 0, stream>>>(g, e, d, lr, ntiles, kk, idx, val, ws);
    else
        topk_pass1_kernel<false><<<pgrid, kBlock, 0, stream>>>(g, e, d, lr, ntiles, kk, idx, val, ws);
    if (k == 0) return hipGetLastError();
    if (vec) {
        topk_step3_kernel<true><<<grid, kBlock, 0, stream>>>(e, d, ntiles, kk, idx, val, ws);
        topk_step4_kernel<true><<<sgrid, kBlock, 0, stream>>>(e, d, ntiles, idx, val, uint64_t(k), ws);
        topk_emit_kernel<true><<<sgrid, kBlock, 0, stream>>>(e, d, idx, val, uint64_t(k), ntiles, ws);
    } else {
        topk_step3_kernel<false><<<grid, kBlock, 0, stream>>>(e, d, ntiles, kk, idx, val, ws);
        topk_step4_kernel<false><<<sgrid, kBlock, 0, stream>>>(e, d, ntiles, idx, val, uint64_t(k), ws);
        topk_emit_kernel<false><<<sgrid, kBlock, 0, stream>>>(e, d, idx, val, uint64_t(k), ntiles, ws);
    }
    return hipGetLastError();
}

}  // namespace efs
