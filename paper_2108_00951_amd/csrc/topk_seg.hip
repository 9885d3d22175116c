// Layer-wise Top-k with error feedback (Appendix C.5: the Top-k sparsifier
// applied to each layer's tensor on its own; Algorithm 1 for the error).
// Segment s is coordinates [off[s], off[s+1]) and keeps min(k[s], size)
// of them: the largest keys (31-bit patterns of |p|), equal keys to the
// lower index, exactly as the flat Top-k ranks them.
//
// Work is cut into tiles: the 4096-element blocks of the vector, clipped to
// each segment, so every tile belongs to one segment and every whole tile is
// 16-byte aligned.  The two sweeps take short slices of consecutive tiles in
// turn across the vector (longer ones with many segments).  Five launches
// (six above 2048 segments, where the reset takes two):
//
//   reset    one workgroup checks the layout and forms the per-segment
//            tables (tile ranges, payload offsets, candidate regions, the
//            bracket); the others zero the per-segment histograms (a light
//            segment, below, only its bracket histogram).
//   pass1    p = e + lr*g written into e (12 B/element, streamed with the
//            non-temporal hint); LDS histogram of key
//            bits 30..18 (8192 bins) per segment, flushed (non-zero bins) to
//            the segment's global histogram, except for a light segment (a
//            bracket and at most kLightTiles tiles).  A segment within one
//            tile is selected right there.  With a bracket [lo, hi] around the
//            segment's threshold predicted from its last three calls on this
//            workspace (error feedback moves it little and smoothly; the
//            bracket reaches 2^wl keys below the prediction and 2^wh above,
//            each 2^12..2^19, adapted per segment), keys above hi go straight
//            to the payload, keys inside it to the candidates and to a
//            1024-bin histogram of the bracket.
//   select1  one workgroup per segment: when pass1 had a bracket and its
//            counts prove the k-th key inside it, the bracket bin da holding
//            it, and pass2's work items for the segment.  Otherwise the digit
//            D1 holding the k-th key (for a light segment from a histogram
//            select1 forms from its elements) and the mode: none (k = 0), all
//            (k = size), candidates (the keys in D1 fit the segment's
//            candidate region) or scan (they do not: a large set of equal or
//            nearly equal magnitudes).
//   pass2    radix path, a read of p (4 B/element): keys above D1 go to the
//            payload and their e to +0 (mode all: every key); keys in D1 are
//            appended to the candidate region and histogrammed by bits 17..8.
//            Bracket path, spread over the whole grid, one work item per
//            wave: e cleared at the pairs above the bracket; candidates in
//            bins above da to the payload, those in bin da listed after the
//            candidates.
//   final    per segment with work, by one of a grid of workgroups: among
//            its candidates (radix path) bits 17..8, then 7..0 give the exact
//            threshold T; among the keys of bin da (bracket path) the low
//            bits of key - lo give it.  Then,
//            when only some keys equal to T are kept, the lowest indices among
//            them by a radix select on the index; emits, clears e, and keeps
//            T as the next hint.  Scan mode does the same over the segment's
//            elements.  Results never depend on the hint.
//
// Payload: segment s's pairs at [kout[s], kout[s] + min(k[s], size)), kout the
// exclusive prefix of those counts; order within a segment unspecified.
#include <stddef.h>

#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

constexpr int kShift1 = 18;     // digit 1: key bits 30..18
constexpr int kShift2 = 8;      // digit 2: key bits 17..8; digit 3: bits 7..0
constexpr int kDigit1 = 1 << (31 - kShift1);
constexpr int kDigit2 = 1 << (kShift1 - kShift2);
constexpr int kDigit3 = 1 << kShift2;
constexpr int kIdxBins = 2048;  // index radix for ties: 11 + 10 + 10 bits
constexpr int kCandLds = 18432;  // candidates the final pass holds in LDS (144 KiB)
// ... with more than kFinalWideMin segments: a smaller buffer (30 KiB), so
// that four workgroups share a CU
constexpr int kCandLdsSmall = 3840;
constexpr int kFinalWideMin = 256;
constexpr int64_t kCandPerK = 16;
constexpr int64_t kCandExtra = 4096;

enum : uint32_t {
    kModeNone = 0, kModeAll = 1, kModeCand = 2, kModeScan = 3, kModeFast = 4,
    kModeDone = 5  // a segment within one tile, selected entirely in pass1
};

// SegState::bracket: 0 none, kBracketFull a bracket with the digit-1
// histogram kept as well, kBracketLight a bracket alone.  A segment of at
// most kLightTiles tiles with a bracket is light: pass1 keeps no digit-1
// histogram for it and the reset zeroes only its 4 KiB bracket histogram
// (32 KiB less per layer to clear each call, the larger part of the reset
// with thousands of layers, and no histogram flush in pass1).  When its
// bracket misses, select1 forms the digit-1 histogram from the segment's
// elements (at most kLightTiles * kTile of them, one sweep by the
// segment's workgroup) and the radix path follows as for any other miss.
constexpr uint32_t kBracketFull = 1u, kBracketLight = 2u;
constexpr uint32_t kLightTiles = 4;

// log2 of how far the bracket reaches below and above the predicted
// threshold, each adapted per segment between these (2^19 keys are 3-6 % of
// |p|, 2^12 keys 0.02-0.05 %)
constexpr uint32_t kWidthMax = 19, kWidthMin = 12, kWidthStart = 17;
// cap on the extrapolated step, in keys: wide when the last two steps agree
// (a steady drift), narrow otherwise (a jump is not repeated)
constexpr int64_t kMaxStep = 1 << 22, kMaxStepUnsure = 1 << 18;
constexpr int kFineBins = 1024;                // bracket histogram: the bracket in 1024 bins
// pass2 work item: payload slots or candidates, one wave's worth (kWorkPerLane
// a lane); a workgroup's four waves take four items at once
constexpr int kWorkPerLane = 8;
constexpr uint32_t kChunk = kWorkPerLane * kWave;
// The sweeps take slices of `slice` consecutive tiles (at most
// kSliceTilesMax), slice b + i * grid for workgroup b: the resident
// workgroups stream one compact window of the vector at a time (measured
// faster than one long range per workgroup), and a slice is long enough to
// amortise its flushes.
constexpr int64_t kSliceTilesMax = 4;
// With more segments than a two-round search covers, a slice starts with a
// third round of dependent reads: the slices are then made as long as the
// grid allows (up to kSliceTilesMaxMany), so that each workgroup searches
// once or a few times.
constexpr int32_t kSearchTwoRounds = kWave * kWave;
constexpr int64_t kSliceTilesMaxMany = 64;
// A one-tile segment with k at most kSmallK takes k block-wide maxima
// instead of the three-level radix select (k barriers instead of about 17).
constexpr int64_t kSmallK = 8;
// Flags of groups of consecutive tiles (2^sweep_shift tiles a group, at most
// kSweepGroups groups): select1 marks the groups of the segments that need
// pass2's tile sweep, and pass2 skips every slice whose groups are unmarked.
constexpr int kSweepGroups = 8192;
constexpr int kSliceWorkgroupsPerCU = 8;
constexpr uint32_t kNoBin = 0xffffffffu;
constexpr uint32_t kNoWork = 0xffffffffu;      // work-list slot not in use this call
static_assert(kFineBins == kDigit2, "the bracket histogram lives in a segment's second histogram");
static_assert(kWidthMax <= 19, "a bracket spans under 2^20 keys, so a bin at most 1024");
constexpr uint32_t kHintMagic = 0x53454748u;

struct SegCtl {
    uint32_t status;   // 0: layout accepted; 1: rejected (the call changed nothing)
    uint32_t tiles;    // tiles of all segments
    uint32_t bracket;  // segments that selected from the bracket (a diagnostic)
    uint32_t pass2;    // nonzero when some segment needs pass2's tile sweep
    uint32_t wtotal;   // work-list slots of all segments (bracket path, for pass2)
    uint32_t pad[59];
};
static_assert(sizeof(SegCtl) == 256, "control block is 256 bytes");

struct SegInfo {
    int64_t off, size, kout, k, coff, ccap;
    uint32_t tile0, ntiles;
    uint32_t wbase, wmax;  // the segment's work-list slots (bracket path)
};
static_assert(sizeof(SegInfo) == 64, "segment info is 64 bytes");

struct SegState {
    uint32_t mode, d1, need1, c1;
    uint32_t emit;     // pairs written to the payload (pass1 with a bracket, or pass2)
    uint32_t ccur;     // candidates appended (pass1 with a bracket, or pass2)
    uint32_t bracket;  // 1: pass1 collects keys in [lo, hi], emits keys above hi
    uint32_t lo, hi;
    uint32_t shift;    // bracket bin of a key: (key - lo) >> shift, 1024 bins
    uint32_t da;       // bracket path: the bin holding the k-th key (kNoBin: none needed)
    uint32_t needa;    // keys of bin da to keep
    uint32_t ca;       // keys in bin da
    uint32_t ecut;     // pairs above the bracket (payload slots 0 .. ecut-1)
    uint32_t tcur;     // keys of bin da listed by pass2 after the candidates
    uint32_t miss;     // bracket not used: 1 threshold below it, 2 above it, 3 too many keys in it
};
static_assert(sizeof(SegState) == 64, "segment state is 64 bytes");

// Thresholds of the last calls on this workspace and the bracket widths,
// kept across calls (the reset only reads them); they decide the bracket,
// never a result.
struct SegHint {
    uint32_t key, prev, prev2;  // the last three thresholds
    uint32_t magic, width;      // validity; bracket widths (packed, see below)
    uint32_t pad[3];
};

// A bracket reaches 2^wl keys below the predicted threshold and 2^wh above
// it; the two are adapted separately, since under error feedback the keys
// crowd just below the threshold and are sparse above it.  Packed as
// wl | wh << 8.
__device__ __forceinline__ uint32_t width_lo(uint32_t w) { return w & 0xffu; }
__device__ __forceinline__ uint32_t width_hi(uint32_t w) { return (w >> 8) & 0xffu; }
__device__ __forceinline__ uint32_t make_widths(uint32_t wl, uint32_t wh) { return wl | (wh << 8); }
__device__ __forceinline__ bool widths_ok(uint32_t w) {
    return (w >> 16) == 0u && width_lo(w) >= kWidthMin && width_lo(w) <= kWidthMax &&
           width_hi(w) >= kWidthMin && width_hi(w) <= kWidthMax;
}
static_assert(sizeof(SegHint) == 32, "hint is 32 bytes");

// The hint after a call whose threshold was T.
__device__ __forceinline__ SegHint next_hint(const SegHint &old, uint32_t T, uint32_t width) {
    const bool ok = old.magic == kHintMagic;
    SegHint h = {};
    h.key = T;
    h.prev = ok ? old.key : T;
    h.prev2 = ok ? old.prev : T;
    h.magic = kHintMagic;
    h.width = width;
    return h;
}

// The reset forms a bracket for a segment from its hint when the segment
// spans several tiles, keeps some but not all of its elements, and the
// hint is well formed.
__device__ __forceinline__ bool hint_usable(const SegHint &h) {
    return h.magic == kHintMagic && h.key <= 0x7fffffffu && h.prev <= 0x7fffffffu &&
           h.prev2 <= 0x7fffffffu && widths_ok(h.width);
}
__device__ __forceinline__ uint32_t bracket_kind(uint32_t ntiles, int64_t keff, int64_t size,
                                                 const SegHint &h) {
    if (!(ntiles > 1u && keff > 0 && keff < size && hint_usable(h))) return 0u;
    return ntiles <= kLightTiles ? kBracketLight : kBracketFull;
}

struct SegWs {
    SegCtl *ctl;
    SegHint *hint;          // [nseg]
    SegInfo *info;
    uint32_t *tile_prefix;  // [nseg + 1]
    SegState *st;
    uint32_t *hist1;        // [nseg][kDigit1]
    uint32_t *hist2;        // [nseg][kDigit2]; on the bracket path, the bracket histogram
    uint2 *cand;            // (bits of p, index)
    uint2 *work;            // pass2 work list: (segment | kind << 31, first slot)
    struct ResetChunk *chunks;  // the reset's per-chunk sums (many layers)
    uint32_t *sweep;        // [kSweepGroups] tile-group flags for pass2's sweep
    int64_t ccap_total;
    uint32_t work_cap;
    uint32_t sweep_shift;   // tile t is in group t >> sweep_shift
};

struct SegLayout {
    size_t info, tile_prefix, st, hint, hist1, hist2, cand, work, chunks, sweep, bytes;
    int64_t ccap_total, work_cap;
};

size_t round256(size_t b) { return (b + 255) & ~size_t(255); }

SegLayout seg_layout(int32_t nseg, int64_t k_total) {
    SegLayout L;
    L.ccap_total = kCandPerK * k_total + kCandExtra * nseg;
    size_t o = sizeof(SegCtl);
    L.info = o;
    o += round256(sizeof(SegInfo) * size_t(nseg));
    L.tile_prefix = o;
    o += round256(4 * (size_t(nseg) + 1));
    L.st = o;
    o += round256(sizeof(SegState) * size_t(nseg));
    L.hint = o;
    o += round256(sizeof(SegHint) * size_t(nseg));
    L.hist1 = o;
    o += round256(4 * size_t(kDigit1) * size_t(nseg));
    L.hist2 = o;
    o += round256(4 * size_t(kDigit2) * size_t(nseg));
    L.cand = o;
    o += round256(8 * size_t(L.ccap_total));
    // one entry per kChunk payload slots or candidates of a segment
    L.work_cap = (k_total + L.ccap_total) / kChunk + 2 * int64_t(nseg) + 1;
    L.work = o;
    o += round256(8 * size_t(L.work_cap));
    // the reset's per-chunk sums (layouts of more than kResetSingleMax layers)
    L.chunks = o;
    o += round256(32 * ((size_t(nseg) + 511) / 512));
    L.sweep = o;
    o += round256(4 * size_t(kSweepGroups));
    L.bytes = o;
    return L;
}

// ---------------------------------------------------------------------------
// Block-wide helpers (every thread of the workgroup calls them)
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t wave_incl_u32(uint32_t v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t o = __shfl_up(v, off);
        if (lane >= off) v += o;
    }
    return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const uint64_t o = __shfl_xor(v, off);
        v = o > v ? o : v;
    }
    return v;
}

__device__ __forceinline__ int64_t wave_incl_i64(int64_t v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int64_t o = __shfl_up(v, off);
        if (lane >= off) v += o;
    }
    return v;
}

// In a histogram of kBins bins (LDS or global), ranked from the top
// (kFromTop) or from the bottom, the bin where the running count first
// reaches `need` (1 <= need <= sum).  s_out gets {bin, count before the bin,
// count in the bin}; {0, 0, 0} when no bin qualifies.  Two barriers.
template <int kBins, bool kFromTop>
__device__ void pick_bin(const uint32_t *hist, uint32_t need, uint32_t *s_wave, uint32_t *s_out) {
    constexpr int kPer = kBins / kBlock;
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
        const int r = t * kPer + i;  // rank position
        c[i] = hist[kFromTop ? kBins - 1 - r : r];
        tot += c[i];
    }
    const uint32_t incl_w = wave_incl_u32(tot);
    if (lane == kWave - 1) s_wave[wave] = incl_w;
    __syncthreads();
    uint32_t off = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) off += q < wave ? s_wave[q] : 0u;
    const uint32_t incl = off + incl_w;
    const uint32_t excl = incl - tot;
    if (excl < need && incl >= need) {
        uint32_t run = excl;
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            if (run + c[i] >= need) {
                const int r = t * kPer + i;
                s_out[0] = uint32_t(kFromTop ? kBins - 1 - r : r);
                s_out[1] = run;
                s_out[2] = c[i];
                break;
            }
            run += c[i];
        }
    }
    __syncthreads();
}

// Segment holding tile t: the largest s with tile_prefix[s] <= t, which
// then has t < tile_prefix[s+1] (empty segments own no tiles and are never
// returned).  A 64-way search: each round every lane of the wave probes one
// position, so nseg <= 4096 takes two rounds of loads instead of twelve
// dependent ones.  Every wave computes the same result.
__device__ __forceinline__ int32_t segment_of_tile(const uint32_t *tp, int32_t nseg, uint32_t t) {
    const int lane = threadIdx.x & (kWave - 1);
    int32_t lo = 0, hi = nseg;  // tp[lo] <= t, and the answer is below hi
    while (hi - lo > 1) {
        const int32_t step = (hi - lo + kWave - 1) / kWave;
        const int32_t probe = lo + lane * step;
        const bool ok = probe < hi && tp[probe] <= t;
        const uint64_t m = __ballot(ok);  // lanes 0..L, lane 0 always set
        const int32_t L = 63 - __clzll(m);
        lo += L * step;
        hi = min(hi, lo + step);
    }
    return lo;
}

// The segment holding tile t when the segment s before it ended at t
// (t == tp[s + 1]): usually the next one, else a search past empty ones.
__device__ __forceinline__ int32_t segment_after(const uint32_t *tp, int32_t nseg, int32_t s,
                                                 uint32_t t) {
    return tp[s + 2] > t ? s + 1 : segment_of_tile(tp, nseg, t);
}

// Word i of a table held one dword a lane (lane i), as a wave-uniform value.
__device__ __forceinline__ uint32_t tab_word(uint32_t v, int i) {
    return __builtin_amdgcn_readlane(v, i);
}

__device__ __forceinline__ int64_t tab_i64(uint32_t v, int i) {
    return int64_t(uint64_t(tab_word(v, i)) | (uint64_t(tab_word(v, i + 1)) << 32));
}
static_assert(offsetof(SegInfo, size) == 8 && offsetof(SegInfo, kout) == 16 &&
                  offsetof(SegInfo, k) == 24 && offsetof(SegInfo, coff) == 32 &&
                  offsetof(SegInfo, ccap) == 40 && offsetof(SegInfo, tile0) == 48 &&
                  offsetof(SegInfo, ntiles) == 52 && offsetof(SegInfo, wmax) == 60,
              "SegInfo words read from a lane-spread table");

// The tables of segment s spread over the lanes of a wave, so that a sweep
// loads the next segment's while it works on the current one (one register,
// no LDS): lanes 0..15 its SegInfo, lane 16 tile_prefix[s + 1] (where it
// ends), lanes 17..20 the bracket, lo, hi and shift of its state (which
// pass1 does not change).  Nothing is loaded for s >= nseg; every wave loads
// its own copy.
constexpr int kTabNext = 16, kTabState = 17, kTabLanes = 21;
static_assert(offsetof(SegState, lo) == offsetof(SegState, bracket) + 4 &&
                  offsetof(SegState, hi) == offsetof(SegState, bracket) + 8 &&
                  offsetof(SegState, shift) == offsetof(SegState, bracket) + 12,
              "bracket, lo, hi, shift are consecutive words");

__device__ __forceinline__ uint32_t load_seg_table(const SegWs &ws, int32_t nseg, int32_t s) {
    const int lane = threadIdx.x & (kWave - 1);
    if (s >= nseg || lane >= kTabLanes) return 0u;
    const uint32_t *src =
        lane < kTabNext ? reinterpret_cast<const uint32_t *>(ws.info + s) + lane
        : lane == kTabNext ? ws.tile_prefix + s + 1
                           : reinterpret_cast<const uint32_t *>(ws.st + s) +
                                 offsetof(SegState, bracket) / 4 + (lane - kTabState);
    return *src;
}

__device__ __forceinline__ SegInfo tab_info(uint32_t v, int b) {
    SegInfo r;
    r.off = tab_i64(v, b + 0);
    r.size = tab_i64(v, b + 2);
    r.kout = tab_i64(v, b + 4);
    r.k = tab_i64(v, b + 6);
    r.coff = tab_i64(v, b + 8);
    r.ccap = tab_i64(v, b + 10);
    r.tile0 = tab_word(v, b + 12);
    r.ntiles = tab_word(v, b + 13);
    r.wbase = tab_word(v, b + 14);
    r.wmax = tab_word(v, b + 15);
    return r;
}

// Element (j, c) of this thread in the 4096-element block starting at
// `block0` (index block0 + (j * kBlock + tid) * 4 + c, the hard threshold's
// map).
__device__ __forceinline__ int64_t tile_elem(int64_t block0, int j, int c) {
    return block0 + int64_t(j * kBlock + int(threadIdx.x)) * 4 + c;
}

// The same element's offset from `block0` (below kTile).
__device__ __forceinline__ uint32_t tile_off(int j, int c) {
    return uint32_t(j * kBlock + int(threadIdx.x)) * 4u + uint32_t(c);
}

// Slice j of every thread's elements covers offsets [j * 1024, (j + 1) * 1024)
// of the block: whether it meets [lo, hi) (the same for the whole workgroup).
__device__ __forceinline__ bool slice_meets(int j, uint32_t lo, uint32_t hi) {
    return uint32_t(j) * (4u * kBlock) < hi && uint32_t(j + 1) * (4u * kBlock) > lo;
}

// Tiles of a segment: the 4096-element blocks it overlaps.
__host__ __device__ __forceinline__ int64_t segment_tiles(int64_t off, int64_t size) {
    return size == 0 ? 0 : ((off + size - 1) / kTile) - (off / kTile) + 1;
}

// Tile t of segment `inf`: the block start and the element range [lo, hi).
struct TileRange {
    int64_t block0, lo, hi;
};

__device__ __forceinline__ TileRange tile_range(const SegInfo &inf, uint32_t t) {
    TileRange r;
    r.block0 = (inf.off / kTile + int64_t(t - inf.tile0)) * kTile;
    r.lo = max(inf.off, r.block0);
    r.hi = min(inf.off + inf.size, r.block0 + kTile);
    return r;
}

// ---------------------------------------------------------------------------
// reset
// ---------------------------------------------------------------------------

// The reset runs 512-thread workgroups: workgroup 0 forms the tables in
// chunks of 512 segments (one block-wide scan per chunk, the next chunk's
// loads in flight meanwhile), the others zero histograms.
constexpr int kResetBlock = 512;
constexpr int kResetWaves = kResetBlock / kWave;

// Tiles and work-list slots stay far below 2^32 for any accepted layout
// (sizes >= 0 summing to d < 2^31); a layout breaking that is rejected by
// its per-segment checks, whatever its sums.
struct Sums {
    int64_t k, c;   // pairs, candidate slots
    uint32_t t, w;  // tiles, work-list slots
};

// Exclusive prefix of v over the workgroup's threads in order; `total` gets
// the sum.  Two barriers.
__device__ __forceinline__ Sums reset_scan(Sums v, Sums *s_wave, Sums &total) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const Sums incl = {wave_incl_i64(v.k), wave_incl_i64(v.c), wave_incl_u32(v.t),
                       wave_incl_u32(v.w)};
    if (lane == kWave - 1) s_wave[wave] = incl;
    __syncthreads();
    Sums off = {0, 0, 0u, 0u}, tot = {0, 0, 0u, 0u};
#pragma unroll
    for (int q = 0; q < kResetWaves; ++q) {
        const Sums x = s_wave[q];
        if (q < wave) {
            off.k += x.k;
            off.c += x.c;
            off.t += x.t;
            off.w += x.w;
        }
        tot.k += x.k;
        tot.c += x.c;
        tot.t += x.t;
        tot.w += x.w;
    }
    __syncthreads();
    total = tot;
    return Sums{off.k + incl.k - v.k, off.c + incl.c - v.c, off.t + incl.t - v.t,
                off.w + incl.w - v.w};
}

// What the reset reads of one segment's layout.
struct SegIn {
    int64_t lo, hi, k;
};

__device__ __forceinline__ SegIn load_seg(const int64_t *off, const int64_t *kin, int32_t s,
                                          int32_t nseg) {
    SegIn in = {};
    if (s < nseg) {
        in.lo = off[s];
        in.hi = off[s + 1];
        in.k = kin[s];
    }
    return in;
}

// The per-layer quantities the tables are built from: pairs kept, candidate
// slots, tiles and work-list slots; `bad` is set for a layer outside the
// rules (negative size or k, outside [0, d)).
__device__ __forceinline__ Sums seg_sums(const SegIn &in, int32_t s, int32_t nseg, int64_t d,
                                         bool &bad) {
    Sums v = {0, 0, 0u, 0u};
    if (s >= nseg) return v;
    const int64_t size = in.hi - in.lo;
    if (size < 0 || in.k < 0 || in.lo < 0 || in.hi > d) bad = true;
    if (size >= 0 && in.k >= 0) {
        const int64_t keff = in.k < size ? in.k : size;
        const uint32_t nt = uint32_t(segment_tiles(in.lo, size));
        const int64_t ccap = (nt > 1u && keff > 0 && keff < size) ? kCandPerK * keff + kCandExtra : 0;
        // bracket path: the pairs above the bracket (at most k) and the
        // candidates (at most ccap), kChunk per work item
        const int64_t wmax = ccap > 0 ? (keff + kChunk - 1) / kChunk + (ccap + kChunk - 1) / kChunk : 0;
        v = Sums{keff, ccap, nt, uint32_t(wmax)};
    }
    return v;
}

// One chunk of kResetBlock layers, s = c0 + thread: their tables after
// `carry` (the sums of all layers before the chunk) and their bracket from
// the hints.  Returns the chunk's sums.  Called by every thread of the
// workgroup.
__device__ __forceinline__ Sums reset_chunk(const SegWs &ws, const SegIn &in, int32_t s,
                                            int32_t nseg, int64_t d, Sums carry, Sums *s_wave,
                                            bool &bad) {
    SegHint h = {};
    if (s < nseg) h = ws.hint[s];  // used after the scan
    const Sums v = seg_sums(in, s, nseg, d, bad);
    Sums tot;
    const Sums ex = reset_scan(v, s_wave, tot);
    if (s < nseg) {
        const int64_t size = in.hi - in.lo;
        const int64_t keff = v.k, ccap = v.c;
        const uint32_t nt = v.t;
        SegInfo inf;
        inf.off = in.lo;
        inf.size = size;
        inf.kout = carry.k + ex.k;
        inf.k = keff;
        inf.coff = carry.c + ex.c;
        inf.ccap = ccap;
        inf.tile0 = uint32_t(carry.t + ex.t);
        inf.ntiles = nt;
        inf.wbase = uint32_t(carry.w + ex.w);
        inf.wmax = v.w;
        ws.info[s] = inf;
        ws.tile_prefix[s] = uint32_t(carry.t + ex.t);
        SegState z = {};
        const uint32_t kind = bracket_kind(nt, keff, size, h);
        if (kind != 0u) {
            // last threshold plus the last step (capped): error feedback
            // makes thresholds drift smoothly from call to call
            const int64_t last = int64_t(h.key) - int64_t(h.prev);
            const int64_t before = int64_t(h.prev) - int64_t(h.prev2);
            const int64_t al = last < 0 ? -last : last, ab = before < 0 ? -before : before;
            const bool steady = (last >= 0) == (before >= 0) && 2 * ab >= al && 2 * al >= ab;
            const int64_t cap = steady ? kMaxStep : kMaxStepUnsure;
            const int64_t step = max(-cap, min(cap, last));
            const int64_t pred = max(int64_t(0), min(int64_t(0x7fffffff), int64_t(h.key) + step));
            z.bracket = kind;
            z.lo = uint32_t(max(int64_t(0), pred - (int64_t(1) << width_lo(h.width))));
            z.hi = uint32_t(min(pred + (int64_t(1) << width_hi(h.width)) - 1, int64_t(0x7fffffff)));
            // hi - lo + 1 <= 2^20 keys in kFineBins bins
            const uint32_t span_bits = 32u - uint32_t(__clz(int(z.hi - z.lo) | 1));
            z.shift = span_bits > 10u ? span_bits - 10u : 0u;
        }
        ws.st[s] = z;
    }
    return tot;
}

// Zeroes the sweep flags and the histograms of the layers that span more
// than one tile (a one-tile layer is selected inside pass1), workgroup w of
// nw: the digit-1 histogram unless the layer is light this call (the table
// workgroup decides that from the same hint), and the bracket or digit-2
// histogram.  An invalid layout is rejected, so what is zeroed for it does
// not matter.
__device__ __forceinline__ void reset_zero(const SegWs &ws, const int64_t *off,
                                           const int64_t *kin, int32_t nseg, int32_t w,
                                           int32_t nw) {
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 *fl = reinterpret_cast<f32x4 *>(ws.sweep);
    for (int q = w * kResetBlock + threadIdx.x; q < kSweepGroups / 4; q += nw * kResetBlock)
        fl[q] = z;
    for (int32_t sg = w; sg < nseg; sg += nw) {
        const int64_t lo = off[sg], size = off[sg + 1] - lo;
        if (size < 0) continue;
        const uint32_t nt = uint32_t(segment_tiles(lo, size));
        if (nt <= 1u) continue;
        const int64_t kk = kin[sg];
        const int64_t keff = kk < size ? kk : size;
        const bool light = bracket_kind(nt, keff, size, ws.hint[sg]) == kBracketLight;
        f32x4 *h2 = reinterpret_cast<f32x4 *>(ws.hist2 + int64_t(sg) * kDigit2);
        if (!light) {
            f32x4 *h1 = reinterpret_cast<f32x4 *>(ws.hist1 + int64_t(sg) * kDigit1);
            for (int q = threadIdx.x; q < kDigit1 / 4; q += kResetBlock) h1[q] = z;
        }
        for (int q = threadIdx.x; q < kDigit2 / 4; q += kResetBlock) h2[q] = z;
    }
}

// The control block once every layer's tables are formed: the layout is
// rejected when a layer broke the rules, the offsets do not run from 0 to d,
// or the sums exceed what the workspace was sized for.  One thread.
__device__ __forceinline__ void reset_publish(const SegWs &ws, const int64_t *off, int32_t nseg,
                                              int64_t d, int64_t k_total, Sums total, bool bad) {
    if (off[0] != 0 || off[nseg] != d) bad = true;
    const bool reject = bad || total.k > k_total || total.c > ws.ccap_total ||
                        total.w > ws.work_cap;
    ws.ctl->bracket = 0u;
    ws.ctl->pass2 = 0u;
    ws.ctl->wtotal = reject ? 0u : total.w;
    ws.ctl->status = reject ? 1u : 0u;
    ws.ctl->tiles = reject ? 0u : total.t;
    if (!reject) ws.tile_prefix[nseg] = total.t;
}

// Up to kResetSingleMax layers: workgroup 0 forms the tables in chunks of
// kResetBlock layers, the next chunk's loads in flight meanwhile; the other
// workgroups zero histograms.
constexpr int32_t kResetSingleMax = 4 * kResetBlock;

__global__ __launch_bounds__(kResetBlock) void seg_reset_kernel(SegWs ws,
                                                                const int64_t *__restrict__ off,
                                                                const int64_t *__restrict__ kin,
                                                                int32_t nseg, int64_t d,
                                                                int64_t k_total) {
    if (blockIdx.x > 0) {
        reset_zero(ws, off, kin, nseg, int32_t(blockIdx.x) - 1, int32_t(gridDim.x) - 1);
        return;
    }
    __shared__ Sums s_wave[kResetWaves];
    __shared__ uint32_t s_bad;
    const int t = threadIdx.x;
    if (t == 0) s_bad = 0u;
    __syncthreads();
    bool bad = false;
    Sums carry = {0, 0, 0u, 0u};
    // the tables are written as the chunks go; a rejected layout leaves them
    // meaningless, and every later kernel then returns at once
    SegIn nxt = load_seg(off, kin, t, nseg);
    for (int32_t c0 = 0; c0 < nseg; c0 += kResetBlock) {
        const int32_t s = c0 + t;
        const SegIn in = nxt;
        nxt = load_seg(off, kin, s + kResetBlock, nseg);  // next chunk, in flight
        const Sums tot = reset_chunk(ws, in, s, nseg, d, carry, s_wave, bad);
        carry.k += tot.k;
        carry.c += tot.c;
        carry.t += tot.t;
        carry.w += tot.w;
    }
    if (bad) atomicOr(&s_bad, 1u);
    __syncthreads();
    if (t == 0) reset_publish(ws, off, nseg, d, k_total, carry, s_bad != 0u);
}

// More layers: the tables in two launches of one workgroup per chunk of
// kResetBlock layers.  The first sums each chunk (and the workgroups after
// the chunks zero histograms); the second adds up the sums of the chunks
// before its own and forms that chunk's tables, and its last workgroup
// publishes the control block.
struct ResetChunk {
    Sums sums;
    uint32_t bad, pad;
};
static_assert(sizeof(ResetChunk) == 32, "a chunk's sums take 32 bytes");

__global__ __launch_bounds__(kResetBlock) void seg_reset_sums_kernel(SegWs ws,
                                                                     const int64_t *__restrict__ off,
                                                                     const int64_t *__restrict__ kin,
                                                                     int32_t nseg, int64_t d,
                                                                     int32_t nchunks) {
    if (int32_t(blockIdx.x) >= nchunks) {
        reset_zero(ws, off, kin, nseg, int32_t(blockIdx.x) - nchunks,
                   int32_t(gridDim.x) - nchunks);
        return;
    }
    __shared__ Sums s_wave[kResetWaves];
    __shared__ uint32_t s_bad;
    if (threadIdx.x == 0) s_bad = 0u;
    __syncthreads();
    const int32_t s = int32_t(blockIdx.x) * kResetBlock + int32_t(threadIdx.x);
    bool bad = false;
    const Sums v = seg_sums(load_seg(off, kin, s, nseg), s, nseg, d, bad);
    if (bad) atomicOr(&s_bad, 1u);
    Sums tot;
    reset_scan(v, s_wave, tot);   // its barriers also order s_bad
    if (threadIdx.x == 0) {
        ResetChunk r = {};
        r.sums = tot;
        r.bad = s_bad;
        ws.chunks[blockIdx.x] = r;
    }
}

__global__ __launch_bounds__(kResetBlock) void seg_reset_tables_kernel(SegWs ws,
                                                                       const int64_t *__restrict__ off,
                                                                       const int64_t *__restrict__ kin,
                                                                       int32_t nseg, int64_t d,
                                                                       int64_t k_total,
                                                                       int32_t nchunks) {
    __shared__ Sums s_wave[kResetWaves];
    const int32_t c = int32_t(blockIdx.x);
    const bool last = c == nchunks - 1;
    const int32_t s = c * kResetBlock + int32_t(threadIdx.x);
    const SegIn in = load_seg(off, kin, s, nseg);
    // the sums of the chunks before this one (all of them, and their flags,
    // for the last)
    Sums before = {0, 0, 0u, 0u};
    uint32_t flags = 0u;
    for (int32_t q = int32_t(threadIdx.x); q < (last ? nchunks : c); q += kResetBlock) {
        const ResetChunk r = ws.chunks[q];
        if (q < c) {
            before.k += r.sums.k;
            before.c += r.sums.c;
            before.t += r.sums.t;
            before.w += r.sums.w;
        }
        flags |= r.bad;
    }
    Sums carry;
    reset_scan(before, s_wave, carry);
    __shared__ uint32_t s_flags;
    if (threadIdx.x == 0) s_flags = 0u;
    __syncthreads();
    if (flags) atomicOr(&s_flags, 1u);
    bool unused = false;   // this chunk's flag is in ws.chunks already
    const Sums tot = reset_chunk(ws, in, s, nseg, d, carry, s_wave, unused);
    if (last && threadIdx.x == 0) {
        const Sums all = {carry.k + tot.k, carry.c + tot.c, carry.t + tot.t, carry.w + tot.w};
        reset_publish(ws, off, nseg, d, k_total, all, s_flags != 0u);
    }
}

// ---------------------------------------------------------------------------
// pass1: p = e + lr*g into e, histogram of key bits 30..18 per segment
// ---------------------------------------------------------------------------

__device__ __forceinline__ void flush_hist(uint32_t *lds, int bins, uint32_t *global) {
    __syncthreads();
    for (int b = threadIdx.x; b < bins; b += kBlock) {
        const uint32_t v = lds[b];
        if (v != 0u) {
            atomicAdd(&global[b], v);
            lds[b] = 0u;
        }
    }
    __syncthreads();
}

// Selections of a workgroup are staged in LDS and written out in coalesced
// runs behind one atomic per run (a global atomic per tile would stall every
// wave for a round trip): payload pairs (index, bits of p) and candidates
// (bits of p, index) of the current segment.
constexpr int kStageCap = 496;  // keeps pass1 (with its 32 KiB histogram) at 4 workgroups per CU

struct Stage {
    uint32_t e_idx[kStageCap];
    uint32_t e_val[kStageCap];
    uint2 cand[kStageCap];
    uint32_t wave[kWaves];
    uint32_t base;
};

__device__ __forceinline__ void flush_emit(Stage &sg, uint32_t &fill, SegState *st,
                                           const SegInfo &inf, int32_t *idx, float *val) {
    __syncthreads();
    if (fill == 0u) return;
    if (threadIdx.x == 0) sg.base = atomicAdd(&st->emit, fill);
    __syncthreads();
    const uint32_t base = sg.base;
    for (uint32_t q = threadIdx.x; q < fill; q += kBlock) {
        const int64_t slot = int64_t(base) + q;
        if (slot < inf.k) {
            idx[inf.kout + slot] = int32_t(sg.e_idx[q]);
            val[inf.kout + slot] = __uint_as_float(sg.e_val[q]);
        }
    }
    fill = 0u;
    __syncthreads();
}

// Bracket histogram of a segment: a candidate key (in [lo, hi]) counted in
// its bin (global memory: pass1 keeps the digit-1 histogram in LDS).
struct Fine {
    uint32_t *hist;  // nullptr: not counted
    uint32_t lo, shift;
};

__device__ __forceinline__ void count_fine(const Fine &f, uint32_t bits) {
    if (f.hist) atomicAdd(&f.hist[(((bits & 0x7fffffffu) - f.lo) >> f.shift) & (kFineBins - 1)], 1u);
}

__device__ __forceinline__ void flush_cand(Stage &sg, uint32_t &fill, SegState *st,
                                           const SegInfo &inf, uint2 *cand, const Fine &fine) {
    __syncthreads();
    if (fill == 0u) return;
    if (threadIdx.x == 0) sg.base = atomicAdd(&st->ccur, fill);
    __syncthreads();
    const uint32_t base = sg.base;
    for (uint32_t q = threadIdx.x; q < fill; q += kBlock) {
        const int64_t slot = int64_t(base) + q;
        const uint2 v = sg.cand[q];
        if (slot < inf.ccap) cand[inf.coff + slot] = v;
        count_fine(fine, v.x);
    }
    fill = 0u;
    __syncthreads();
}

// Both stages flushed at once, as at the end of a segment: the two slot
// reservations (one atomic each, from two waves) are in flight together, one
// round trip instead of two.
__device__ __forceinline__ void flush_both(Stage &sg, uint32_t &efill, uint32_t &cfill,
                                           SegState *st, const SegInfo &inf, int32_t *idx,
                                           float *val, uint2 *cand, const Fine &fine) {
    __syncthreads();
    if (efill == 0u && cfill == 0u) return;
    if (threadIdx.x == 0 && efill != 0u) sg.wave[0] = atomicAdd(&st->emit, efill);
    if (threadIdx.x == kWave && cfill != 0u) sg.wave[1] = atomicAdd(&st->ccur, cfill);
    __syncthreads();
    const uint32_t ebase = sg.wave[0], cbase = sg.wave[1];
    for (uint32_t q = threadIdx.x; q < efill; q += kBlock) {
        const int64_t slot = int64_t(ebase) + q;
        if (slot < inf.k) {
            idx[inf.kout + slot] = int32_t(sg.e_idx[q]);
            val[inf.kout + slot] = __uint_as_float(sg.e_val[q]);
        }
    }
    for (uint32_t q = threadIdx.x; q < cfill; q += kBlock) {
        const int64_t slot = int64_t(cbase) + q;
        const uint2 v = sg.cand[q];
        if (slot < inf.ccap) cand[inf.coff + slot] = v;
        count_fine(fine, v.x);
    }
    efill = 0u;
    cfill = 0u;
    __syncthreads();
}

// Stages this tile's selections (called by every thread of the workgroup):
// elements of `emit_mask` for the payload (e cleared there when zero_e), of
// `cand_mask` for the candidates (counted in `fine` when it has a
// histogram).  When a tile selects more of either than a stage holds (mode
// all, or many equal keys), its slots are reserved directly with one atomic
// and written without staging.
__device__ __forceinline__ void stage_tile(Stage &sg, uint32_t &efill, uint32_t &cfill,
                                           const float (&p)[kVecPerThread][4], int64_t block0,
                                           uint32_t emit_mask, uint32_t cand_mask,
                                           const SegInfo &inf, SegState *st, uint2 *cand,
                                           int32_t *idx, float *val, float *e, bool zero_e,
                                           const Fine &fine) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const uint32_t mine = uint32_t(__popc(emit_mask)) | (uint32_t(__popc(cand_mask)) << 16);
    const uint32_t incl = wave_incl_u32(mine);
    if (lane == kWave - 1) sg.wave[wave] = incl;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
        off += q < wave ? sg.wave[q] : 0u;
        tot += sg.wave[q];
    }
    const uint32_t pre = off + incl - mine;
    const uint32_t te = tot & 0xffffu, tc = tot >> 16;
    __syncthreads();  // sg.wave is reused below and by the next tile
    if (te == 0u && tc == 0u) return;
    const bool edirect = te > uint32_t(kStageCap);
    const bool cdirect = tc > uint32_t(kStageCap);
    if (!edirect && efill + te > uint32_t(kStageCap)) flush_emit(sg, efill, st, inf, idx, val);
    if (!cdirect && cfill + tc > uint32_t(kStageCap)) flush_cand(sg, cfill, st, inf, cand, fine);
    uint32_t ebase = 0, cbase = 0;
    if (edirect || cdirect) {
        if (threadIdx.x == 0) {
            if (edirect) sg.wave[0] = atomicAdd(&st->emit, te);
            if (cdirect) sg.wave[1] = atomicAdd(&st->ccur, tc);
        }
        __syncthreads();
        ebase = sg.wave[0];
        cbase = sg.wave[1];
        __syncthreads();
    }
    uint32_t ep = pre & 0xffffu, cp = pre >> 16;
#pragma unroll
    for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint32_t bit = 1u << (4 * j + c);
            const int64_t i = tile_elem(block0, j, c);
            if (emit_mask & bit) {
                if (edirect) {
                    const int64_t slot = int64_t(ebase) + ep;
                    if (slot < inf.k) {
                        idx[inf.kout + slot] = int32_t(i);
                        val[inf.kout + slot] = p[j][c];
                    }
                } else {
                    sg.e_idx[efill + ep] = uint32_t(i);
                    sg.e_val[efill + ep] = __float_as_uint(p[j][c]);
                }
                if (zero_e) e[i] = 0.0f;
                ++ep;
            }
            if (cand_mask & bit) {
                const uint2 v = make_uint2(__float_as_uint(p[j][c]), uint32_t(i));
                if (cdirect) {
                    const int64_t slot = int64_t(cbase) + cp;
                    if (slot < inf.ccap) cand[inf.coff + slot] = v;
                    count_fine(fine, v.x);
                } else {
                    sg.cand[cfill + cp] = v;
                }
                ++cp;
            }
        }
    }
    if (!edirect) efill += te;
    if (!cdirect) cfill += tc;
    __syncthreads();
}

// A segment that lies within one tile is selected here, by the workgroup
// holding it: for a small k, k rounds of a block-wide maximum of (key, lower
// index first); otherwise a radix select on the keys of its elements (bits
// 30..20, 19..10, 9..0, histograms in LDS), the keys equal to the threshold
// kept in index order.  The pairs are written to the segment's payload
// region and e cleared at them (e already holds p).  Element (j, c) of a
// thread is index block0 + tile_off(j, c), block0 being the segment's first
// element.  `hist` is 2048 words of zeroed LDS, zeroed again on return.
// Called by every thread of the workgroup.
__device__ void select_in_tile(const float (&p)[kVecPerThread][4], uint32_t valid,
                               int64_t block0, const SegInfo &inf, uint32_t *hist,
                               uint32_t *s_wave, uint32_t *s_out, int32_t *idx, float *val,
                               float *e) {
    const int tid = threadIdx.x;
    // slices j >= jn hold none of the segment (its elements start at block0)
    const int jn = int((uint32_t(inf.size) + 4u * kBlock - 1u) / (4u * kBlock));
    uint32_t key[kVecPerThread][4];
#pragma unroll
    for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) key[j][c] = magnitude_key(p[j][c]);
    uint32_t keep = 0;
    if (inf.k >= inf.size) {
        keep = valid;
    } else if (inf.k <= kSmallK) {
        // k rounds of a block-wide maximum over the elements not yet kept,
        // of (key, then the lower index): one barrier a round
        __shared__ uint64_t s_best[2][kWaves];
        const int lane = tid & (kWave - 1);
        const int wave = tid / kWave;
#pragma unroll 1
        for (int r = 0; r < int(inf.k); ++r) {
            // this thread's elements in (j, c) order are in index order, so
            // the first strictly larger key is its best
            const uint32_t open = valid & ~keep;
            uint64_t best = 0;
            if (__any(open != 0u)) {  // waves past the segment's end skip this
                uint32_t bk = 0, bs = 32;
#pragma unroll
                for (int j = 0; j < kVecPerThread; ++j)
                    if (j < jn)
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            if (((open >> (4 * j + c)) & 1u) && (bs == 32 || key[j][c] > bk)) {
                                bk = key[j][c];
                                bs = uint32_t(4 * j + c);
                            }
                if (bs != 32) {
                    const uint32_t pos =
                        ((bs >> 2) * uint32_t(kBlock) + uint32_t(tid)) * 4u + (bs & 3u);
                    best = (uint64_t(bk) << 32) | (0xffffffffu - pos);
                }
                best = wave_max_u64(best);
            }
            if (lane == 0) s_best[r & 1][wave] = best;
            __syncthreads();
            uint64_t all = s_best[r & 1][0];
#pragma unroll
            for (int q = 1; q < kWaves; ++q) all = s_best[r & 1][q] > all ? s_best[r & 1][q] : all;
            // every valid element scores above 0, and k < size of them exist
            const uint32_t pos = 0xffffffffu - uint32_t(all);
            const uint32_t quad = pos >> 2;
            if (int(quad % uint32_t(kBlock)) == tid)
                keep |= 1u << (4 * (quad / uint32_t(kBlock)) + (pos & 3u));
        }
    } else if (inf.k > 0) {
        uint32_t need = uint32_t(inf.k), prefix = 0;
#pragma unroll 1
        for (int level = 0; level < 3; ++level) {
            const int shift = 20 - 10 * level;
            const uint32_t mask = level == 0 ? 2047u : 1023u;
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    if (((valid >> (4 * j + c)) & 1u) &&
                        (level == 0 || (key[j][c] >> (shift + 10)) == prefix))
                        atomicAdd(&hist[(key[j][c] >> shift) & mask], 1u);
            __syncthreads();
            if (level == 0) pick_bin<2048, true>(hist, need, s_wave, s_out);
            else pick_bin<1024, true>(hist, need, s_wave, s_out);
            prefix = (prefix << (level == 0 ? 11 : 10)) | s_out[0];
            need -= s_out[1];
            for (int b = tid; b < 2048; b += kBlock) hist[b] = 0u;
            __syncthreads();
        }
        const uint32_t T = prefix;  // need = keys equal to T to keep
        uint32_t tie = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t bit = 1u << (4 * j + c);
                if (!(valid & bit)) continue;
                if (key[j][c] > T) keep |= bit;
                else if (key[j][c] == T) tie |= bit;
            }
        // tie ranks in index order: vector slot j, then thread, then c
        uint32_t rank = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
            const uint32_t tj = (tie >> (4 * j)) & 0xfu;
            uint32_t slot_total;
            uint32_t r = rank + block_prefix_small(uint32_t(__popc(tj)), s_wave, slot_total);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if ((tj >> c) & 1u) {
                    keep |= uint32_t(r < need) << (4 * j + c);
                    ++r;
                }
            rank += slot_total;
        }
    }
    uint32_t total;
    int64_t slot = inf.kout + block_prefix_small(uint32_t(__popc(keep)), s_wave, total);
#pragma unroll
    for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if ((keep >> (4 * j + c)) & 1u) {
                const int64_t i = tile_elem(block0, j, c);
                idx[slot] = int32_t(i);
                val[slot] = p[j][c];
                e[i] = 0.0f;
                ++slot;
            }
}

// Small one-tile segments (at most kWaveLayerMax elements, k <= kSmallK or
// every element kept) are selected by one wave each, so that a workgroup
// takes up to kWaves of them at once with no barrier: models with thousands
// of tensors have mostly such layers, and one at a time each cost the
// workgroup a memory round trip and a few barriers.
constexpr int kWaveLayerMax = 16 * kWave;  // 16 elements a lane

__device__ __forceinline__ bool wave_layer(int64_t size, int64_t k) {
    return size <= kWaveLayerMax && (k <= kSmallK || k >= size);
}

// One wave: the error-feedback step and the selection of segment `inf`
// (one tile, 1 <= size <= kWaveLayerMax): element q * 64 + lane of the
// segment in slot q of the lane, k rounds of a wave-wide maximum of (key,
// lower index first) as in select_in_tile, the kept pairs written to the
// segment's payload region in index order, e' = p elsewhere and +0 at them.
__device__ __forceinline__ void select_in_wave(const float *__restrict__ g, float *__restrict__ e,
                                               float lr, int32_t *__restrict__ idx,
                                               float *__restrict__ val, const SegInfo &inf) {
    constexpr int kSlots = kWaveLayerMax / kWave;
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const uint32_t size = uint32_t(inf.size);
    const float *gs = g + inf.off;
    float *es = e + inf.off;
    float p[kSlots];
    uint32_t valid = 0;
    // loads first (a slot past the end reads the last element, which the
    // segment owns), then p
    float gv[kSlots], ev[kSlots];
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
        if (uint32_t(q) * kWave >= size) break;  // the same for the whole wave
        const uint32_t o = min(uint32_t(q) * kWave + lane, size - 1u);
        gv[q] = gs[o];
        ev[q] = es[o];
    }
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
        p[q] = 0.0f;
        if (uint32_t(q) * kWave >= size) break;
        p[q] = ef_accumulate(ev[q], lr, gv[q]);
        if (uint32_t(q) * kWave + lane < size) valid |= 1u << q;
    }
    uint32_t keep = 0;
    if (inf.k >= inf.size) {
        keep = valid;
    } else {
#pragma unroll 1
        for (int r = 0; r < int(inf.k); ++r) {
            // slots in q order are in index order: the first strictly larger
            // key is this lane's best
            const uint32_t open = valid & ~keep;
            uint32_t bk = 0, bq = 32;
#pragma unroll
            for (int q = 0; q < kSlots; ++q)
                if (((open >> q) & 1u) && (bq == 32 || magnitude_key(p[q]) > bk)) {
                    bk = magnitude_key(p[q]);
                    bq = uint32_t(q);
                }
            uint64_t best = 0;  // every valid element scores above 0
            if (bq != 32) best = (uint64_t(bk) << 32) | (0xffffffffu - (bq * kWave + lane));
            const uint32_t o = 0xffffffffu - uint32_t(wave_max_u64(best));
            if ((o & (kWave - 1)) == lane) keep |= 1u << (o / kWave);
        }
    }
    // e' and the kept pairs, ranked in index order (slot, then lane)
    uint32_t rank = 0;
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
        if (uint32_t(q) * kWave >= size) break;
        const bool kq = (keep >> q) & 1u;
        const uint64_t m = __ballot(kq);
        const uint32_t o = uint32_t(q) * kWave + lane;
        if (kq) {
            const int64_t slot = inf.kout + rank + lanes_below(m);
            idx[slot] = int32_t(inf.off + o);
            val[slot] = p[q];
        }
        if ((valid >> q) & 1u) es[o] = kq ? 0.0f : p[q];
        rank += uint32_t(__popcll(m));
    }
}

// Segment s (holding tile t, one tile, small) and the segments after it
// that hold tiles t + 1, t + 2, ... (below t1) and are small one-tile
// segments as well, up to kWaves of them: wave w selects segment s + w.
// Returns how many were taken (at least 1; the same in every thread).  No
// barrier: each wave reads the tables of s + 1 .. s + 3 itself, one dword a
// lane (lanes 16 (w - 1) .. 16 w - 1 hold segment s + w's SegInfo).
__device__ __forceinline__ uint32_t wave_layers(const float *__restrict__ g,
                                                float *__restrict__ e, float lr,
                                                int32_t *__restrict__ idx,
                                                float *__restrict__ val, int32_t nseg,
                                                const SegWs &ws, int32_t s, const SegInfo &inf,
                                                uint32_t t, uint32_t t1) {
    constexpr int kInfoWords = sizeof(SegInfo) / 4;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
    uint32_t tab = 0u;  // a segment not loaded reads as 0 tiles
    {
        const int w = 1 + lane / kInfoWords;
        if (w < kWaves && s + w < nseg && t + uint32_t(w) < t1)
            tab = reinterpret_cast<const uint32_t *>(ws.info + s + w)[lane % kInfoWords];
    }
    uint32_t run = 1;
#pragma unroll
    for (int w = 1; w < kWaves; ++w) {
        const int b = kInfoWords * (w - 1);
        // segments s .. s + w - 1 hold one tile each, so s + w (when it
        // holds any tile) holds tile t + w
        if (run == uint32_t(w) && tab_word(tab, b + 13) == 1u &&
            wave_layer(tab_i64(tab, b + 2), tab_i64(tab, b + 6)))
            run = uint32_t(w + 1);
    }
    if (uint32_t(wave) < run) {
        if (wave == 0) {
            select_in_wave(g, e, lr, idx, val, inf);
        } else {
            const int b = kInfoWords * (wave - 1);
            SegInfo mi;
            mi.off = tab_i64(tab, b + 0);
            mi.size = tab_i64(tab, b + 2);
            mi.kout = tab_i64(tab, b + 4);
            mi.k = tab_i64(tab, b + 6);
            select_in_wave(g, e, lr, idx, val, mi);
        }
    }
    return run;
}

// Tiles [t0, t1) of pass1; every selection, count and histogram is flushed
// before it returns (the LDS histogram is left zero).
template <bool kAligned>
__device__ void pass1_slice(const float *__restrict__ g, float *__restrict__ e, float lr,
                            int32_t *__restrict__ idx, float *__restrict__ val, int32_t nseg,
                            const SegWs &ws, uint32_t t0, uint32_t t1, uint32_t *hist, Stage &sg,
                            uint32_t *s_wave, uint32_t *s_out) {
    int32_t s = segment_of_tile(ws.tile_prefix, nseg, t0);
    uint32_t next = ws.tile_prefix[s + 1];
    SegInfo inf = ws.info[s];
    SegState *st = ws.st + s;
    uint32_t bracket = st->bracket, lo = st->lo, hi = st->hi;
    Fine fine = {ws.hist2 + int64_t(s) * kDigit2, lo, st->shift};
    // the following segment's tables, in flight while this one is swept
    uint32_t tab = load_seg_table(ws, nseg, s + 1);
    uint32_t efill = 0, cfill = 0;
    __syncthreads();
    for (uint32_t t = t0; t < t1; ++t) {
        if (t >= next) {
            if (bracket) {
                flush_both(sg, efill, cfill, st, inf, idx, val, ws.cand, fine);
            }
            // a one-tile or a light segment leaves the LDS histogram zero
            if (inf.ntiles > 1 && bracket != kBracketLight)
                flush_hist(hist, kDigit1, ws.hist1 + int64_t(s) * kDigit1);
            if (s + 1 < nseg && tab_word(tab, kTabNext) > t) {
                // tile t (== tile_prefix[s + 1]) opens segment s + 1: the
                // prefetched tables
                ++s;
                inf = tab_info(tab, 0);
                next = tab_word(tab, kTabNext);
                bracket = tab_word(tab, kTabState);
                lo = tab_word(tab, kTabState + 1);
                hi = tab_word(tab, kTabState + 2);
                fine = Fine{ws.hist2 + int64_t(s) * kDigit2, lo, tab_word(tab, kTabState + 3)};
            } else {
                // past empty segments
                s = segment_of_tile(ws.tile_prefix, nseg, t);
                next = ws.tile_prefix[s + 1];
                inf = ws.info[s];
                bracket = ws.st[s].bracket;
                lo = ws.st[s].lo;
                hi = ws.st[s].hi;
                fine = Fine{ws.hist2 + int64_t(s) * kDigit2, lo, ws.st[s].shift};
            }
            st = ws.st + s;
            tab = load_seg_table(ws, nseg, s + 1);
        }
        if (inf.ntiles == 1 && wave_layer(inf.size, inf.k)) {
            // this and the following small one-tile segments, a wave each;
            // the last of them becomes the current segment (no bracket, no
            // histogram: nothing to flush when the next tile leaves it)
            const uint32_t run = wave_layers(g, e, lr, idx, val, nseg, ws, s, inf, t, t1);
            s += int32_t(run) - 1;
            t += run - 1;
            next = t + 1;
            st = ws.st + s;
            if (run > 1) tab = load_seg_table(ws, nseg, s + 1);
            continue;
        }
        const TileRange r = tile_range(inf, t);
        float p[kVecPerThread][4];
        uint32_t valid = 0;
        if (kAligned && r.lo == r.block0 && r.hi == r.block0 + kTile) {
            const f32x4 *g4 = reinterpret_cast<const f32x4 *>(g + r.block0);
            f32x4 *e4 = reinterpret_cast<f32x4 *>(e + r.block0);
            f32x4 gv[kVecPerThread], ev[kVecPerThread];
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
                gv[j] = __builtin_nontemporal_load(g4 + j * kBlock + threadIdx.x);
                ev[j] = __builtin_nontemporal_load(e4 + j * kBlock + threadIdx.x);
            }
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
                f32x4 pv;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    pv[c] = ef_accumulate(ev[j][c], lr, gv[j][c]);
                    p[j][c] = pv[c];
                }
                __builtin_nontemporal_store(pv, e4 + j * kBlock + threadIdx.x);
            }
            valid = 0xffffu;
        } else {
            // a segment's first or last block: only its own elements are
            // read and written (the rest of the block belongs to neighbours).
            // A segment within one block is laid over the threads from its
            // first element on, so that a small one fills few slices and
            // waves; slices outside the elements are skipped.
            const int64_t base = inf.ntiles == 1 ? inf.off : r.block0;
            const uint32_t lo = uint32_t(r.lo - base), hi = uint32_t(r.hi - base);
            const float *gb = g + base;
            float *eb = e + base;
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
                for (int c = 0; c < 4; ++c) p[j][c] = 0.0f;
                if (!slice_meets(j, lo, hi)) continue;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t o = tile_off(j, c);
                    if (o >= lo && o < hi) {
                        p[j][c] = ef_accumulate(eb[o], lr, gb[o]);
                        eb[o] = p[j][c];
                        valid |= 1u << (4 * j + c);
                    }
                }
            }
            if (inf.ntiles == 1) {
                select_in_tile(p, valid, base, inf, hist, s_wave, s_out, idx, val, e);
                continue;
            }
        }
        uint32_t emit_mask = 0, cand_mask = 0;
        const bool digits = bracket != kBracketLight;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
            if (!__any(((valid >> (4 * j)) & 0xfu) != 0u)) continue;  // none in this wave
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t bit = 1u << (4 * j + c);
                if (!(valid & bit)) continue;
                const uint32_t key = magnitude_key(p[j][c]);
                if (digits) atomicAdd(&hist[key >> kShift1], 1u);
                if (key > hi) emit_mask |= bit;
                else if (key >= lo) cand_mask |= bit;
            }
        }
        // keys above the bracket go to the payload (e is cleared only once
        // the bracket is confirmed), keys inside it to the candidates and
        // the bracket histogram
        if (bracket)
            stage_tile(sg, efill, cfill, p, r.block0, emit_mask, cand_mask, inf, st, ws.cand, idx,
                       val, e, false, fine);
    }
    if (bracket) {
        flush_both(sg, efill, cfill, st, inf, idx, val, ws.cand, fine);
    }
    if (inf.ntiles > 1 && bracket != kBracketLight)
        flush_hist(hist, kDigit1, ws.hist1 + int64_t(s) * kDigit1);
    __syncthreads();  // the next slice starts with another segment's state
}

template <bool kAligned>
__global__ __launch_bounds__(kBlock, 4) void seg_pass1_kernel(const float *__restrict__ g,
                                                           float *__restrict__ e, float lr,
                                                           int32_t *__restrict__ idx,
                                                           float *__restrict__ val, int32_t nseg,
                                                           SegWs ws, uint32_t slice) {
    __shared__ uint32_t hist[kDigit1];
    __shared__ Stage sg;
    __shared__ uint32_t s_wave[kWaves];
    __shared__ uint32_t s_out[3];
    if (ws.ctl->status != 0u) return;
    const uint32_t T = ws.ctl->tiles;
    for (int b = threadIdx.x; b < kDigit1; b += kBlock) hist[b] = 0u;
    for (uint32_t t0 = blockIdx.x * slice; t0 < T; t0 += gridDim.x * slice)
        pass1_slice<kAligned>(g, e, lr, idx, val, nseg, ws, t0, min(T, t0 + slice), hist, sg,
                              s_wave, s_out);
}

// ---------------------------------------------------------------------------
// select1: per segment, the bracket bin or the digit of the k-th key, and the mode
// ---------------------------------------------------------------------------

// Marks the tile groups of segment `inf` for pass2's sweep.  Called by
// every thread of the workgroup.
__device__ __forceinline__ void mark_sweep(const SegWs &ws, const SegInfo &inf) {
    const uint32_t g0 = inf.tile0 >> ws.sweep_shift;
    const uint32_t g1 = min((inf.tile0 + inf.ntiles - 1u) >> ws.sweep_shift,
                            uint32_t(kSweepGroups - 1));
    for (uint32_t q = g0 + threadIdx.x; q <= g1; q += kBlock) ws.sweep[q] = 1u;
}

// Radix path of segment s (0 < k < size): from its digit-1 histogram, the
// digit D1 holding the k-th key, the keys still needed inside it, and the
// mode (none, candidates, or scan when the keys in D1 overflow the segment's
// candidate region).  Called by every thread of the workgroup.
__device__ void choose_digit1(const SegWs &ws, int32_t s, const SegInfo &inf, SegState *st,
                              uint32_t *s_wave, uint32_t *s_out) {
    pick_bin<kDigit1, true>(ws.hist1 + int64_t(s) * kDigit1, uint32_t(inf.k), s_wave, s_out);
    if (threadIdx.x == 0) {
        // the radix path emits and collects from scratch in pass2
        st->emit = 0u;
        st->ccur = 0u;
        const uint32_t c1 = s_out[2];
        st->d1 = s_out[0];
        st->need1 = uint32_t(inf.k) - s_out[1];
        st->c1 = c1;
        st->mode = c1 == 0u ? kModeNone : (int64_t(c1) <= inf.ccap ? kModeCand : kModeScan);
        // a flag, stored (an atomic per segment on one word serialises when
        // thousands of segments take this path)
        if (c1 != 0u) ws.ctl->pass2 = 1u;
    }
    const bool sweep = s_out[2] != 0u;
    __syncthreads();  // s_out is reused by the caller
    if (sweep) mark_sweep(ws, inf);
}

// The digit-1 histogram of a light segment whose bracket missed (pass1 kept
// none for it), formed from its elements: e holds p everywhere in the
// segment, since pass1 clears e only once the bracket is confirmed.  The
// counts are at most kLightTiles * kTile, so two 16-bit counts share an LDS
// word (16 KiB); the 8192 bins are then stored whole into the segment's
// global histogram, which choose_digit1 reads.  One sweep of e in 16-byte
// vectors (the few elements before the first 16-byte boundary and after the
// last one at a time).  Called by every thread of the workgroup.
__device__ void light_digit1(const SegWs &ws, const float *__restrict__ e, const SegInfo &inf,
                             int32_t s, uint32_t *pack) {
    const uint32_t tid = threadIdx.x;
    for (uint32_t b = tid; b < uint32_t(kDigit1 / 2); b += kBlock) pack[b] = 0u;
    __syncthreads();
    const float *seg = e + inf.off;
    const uint32_t n = uint32_t(inf.size);
    // seg + h is the first 16-byte boundary at or after seg (e is 4-byte aligned)
    const uint32_t h = min(n, uint32_t(((16u - (reinterpret_cast<uintptr_t>(seg) & 15u)) & 15u) / 4u));
    const uint32_t nv = (n - h) / 4u;
    const uint32_t t0 = h + 4u * nv;
    for (uint32_t i = tid; i < h + (n - t0); i += kBlock) {
        const uint32_t d1 = magnitude_key(seg[i < h ? i : t0 + (i - h)]) >> kShift1;
        atomicAdd(&pack[d1 >> 1], 1u << (16u * (d1 & 1u)));
    }
    const f32x4 *v4 = reinterpret_cast<const f32x4 *>(seg + h);
    constexpr uint32_t kV = 4;  // 16-byte loads per thread in flight
    for (uint32_t base = 0; base < nv; base += kV * kBlock) {
        f32x4 x[kV];
#pragma unroll
        for (uint32_t u = 0; u < kV; ++u) {
            const uint32_t q = base + u * kBlock + tid;
            if (q < nv) x[u] = v4[q];
        }
#pragma unroll
        for (uint32_t u = 0; u < kV; ++u) {
            if (base + u * kBlock + tid < nv) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t d1 = magnitude_key(x[u][c]) >> kShift1;
                    atomicAdd(&pack[d1 >> 1], 1u << (16u * (d1 & 1u)));
                }
            }
        }
    }
    __syncthreads();
    uint2 *h1 = reinterpret_cast<uint2 *>(ws.hist1 + int64_t(s) * kDigit1);
    for (uint32_t b = tid; b < uint32_t(kDigit1 / 2); b += kBlock) {
        const uint32_t v = pack[b];
        h1[b] = make_uint2(v & 0xffffu, v >> 16);
    }
    __syncthreads();  // the workgroup reads the histogram back
}

__device__ void select1_segment(const SegWs &ws, const float *__restrict__ e, int32_t s,
                                uint32_t *s_wave, uint32_t *s_out, uint32_t *s_pack) {
    const SegInfo inf = ws.info[s];
    SegState *st = ws.st + s;
    if (inf.ntiles <= 1) {  // selected in pass1 (or empty)
        if (threadIdx.x == 0) st->mode = kModeDone;
        return;
    }
    if (inf.k == 0 || inf.k == inf.size) {
        if (threadIdx.x == 0) {
            st->mode = inf.k == 0 ? kModeNone : kModeAll;
            if (inf.k != 0) ws.ctl->pass2 = 1u;
        }
        if (inf.k != 0) mark_sweep(ws, inf);
        return;
    }
    // bracket confirmed when #(key > hi) <= k <= #(key >= lo) and every key in
    // the bracket was collected: the bracket histogram then names the bin da
    // holding the k-th key; keys in higher bins are kept, keys in lower bins
    // dropped, and only bin da is ranked (by the final pass, from a list that
    // pass2 writes after the candidates, so it must fit there)
    const SegState cur = *st;
    uint32_t *fine = ws.hist2 + int64_t(s) * kDigit2;
    __syncthreads();  // every thread has read the state before it changes
    if (cur.bracket && int64_t(cur.emit) <= inf.k && int64_t(cur.emit) + cur.ccur >= inf.k &&
        int64_t(cur.ccur) <= inf.ccap) {
        const uint32_t need = uint32_t(inf.k) - cur.emit;
        uint32_t da = kNoBin, needa = 0u, ca = 0u;
        if (need > 0u) {
            pick_bin<kFineBins, true>(fine, need, s_wave, s_out);
            da = s_out[0];
            needa = need - s_out[1];
            ca = s_out[2];
        }
        if (int64_t(cur.ccur) + ca <= inf.ccap) {
            // pass2's work: clear e at the pairs above the bracket, and sort
            // the candidates into kept, dropped and bin da
            const uint32_t na = (cur.emit + kChunk - 1) / kChunk;
            const uint32_t nc = need > 0u ? (cur.ccur + kChunk - 1) / kChunk : 0u;
            __syncthreads();  // s_out is read above by every thread
            if (threadIdx.x == 0) {
                st->mode = kModeFast;
                st->need1 = need;
                st->da = da;
                st->needa = needa;
                st->ca = ca;
                st->ecut = cur.emit;
                st->tcur = 0u;
            }
            // the items go to the segment's own slots, the rest of them marked
            // unused: every slot of the list is written every call
            for (uint32_t q = threadIdx.x; q < inf.wmax; q += kBlock) {
                const uint32_t w = inf.wbase + q;
                if (w < ws.work_cap)
                    ws.work[w] = q < na ? make_uint2(uint32_t(s), q * kChunk)
                                 : q < na + nc ? make_uint2(uint32_t(s) | 0x80000000u, (q - na) * kChunk)
                                               : make_uint2(kNoWork, 0u);
            }
            return;
        }
    }
    for (uint32_t q = threadIdx.x; q < inf.wmax; q += kBlock)
        if (inf.wbase + q < ws.work_cap) ws.work[inf.wbase + q] = make_uint2(kNoWork, 0u);
    if (cur.bracket) {
        // missed: the radix path follows; the bracket histogram shares the
        // memory pass2 counts in
        f32x4 *h = reinterpret_cast<f32x4 *>(fine);
        const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int q = threadIdx.x; q < kDigit2 / 4; q += kBlock) h[q] = z;
        if (threadIdx.x == 0)
            st->miss = int64_t(cur.emit) > inf.k ? 2u
                       : (int64_t(cur.emit) + cur.ccur < inf.k ? 1u : 3u);
    }
    if (cur.bracket == kBracketLight) light_digit1(ws, e, inf, s, s_pack);
    choose_digit1(ws, s, inf, st, s_wave, s_out);
}

// One workgroup per segment (a loop over segments per workgroup serialises
// their latencies: measured slower with thousands of segments).
__global__ __launch_bounds__(kBlock) void seg_select1_kernel(SegWs ws, const float *__restrict__ e) {
    __shared__ uint32_t s_wave[kWaves];
    __shared__ uint32_t s_out[3];
    __shared__ uint32_t s_pack[kDigit1 / 2];
    if (ws.ctl->status != 0u) return;
    select1_segment(ws, e, int32_t(blockIdx.x), s_wave, s_out, s_pack);
}

// ---------------------------------------------------------------------------
// pass2: keys above D1 to the payload, keys in D1 to the candidates; the
// bracket path's work items
// ---------------------------------------------------------------------------

// The radix path's sweep over tiles [t0, t1).
template <bool kAligned>
__device__ void pass2_tiles(float *__restrict__ e, int32_t *__restrict__ idx,
                            float *__restrict__ val, int32_t nseg, const SegWs &ws, uint32_t t0,
                            uint32_t t1, uint32_t *hist, Stage &sg) {
    const Fine nofine = {nullptr, 0u, 0u};
    for (int b = threadIdx.x; b < kDigit2; b += kBlock) hist[b] = 0u;
    int32_t s = segment_of_tile(ws.tile_prefix, nseg, t0);
    uint32_t next = ws.tile_prefix[s + 1];
    SegInfo inf = ws.info[s];
    SegState *st = ws.st + s;
    uint32_t mode = st->mode, D1 = st->d1;
    bool dirty = false;
    uint32_t efill = 0, cfill = 0;
    __syncthreads();
    for (uint32_t t = t0; t < t1; ++t) {
        if (t >= next) {
            flush_both(sg, efill, cfill, st, inf, idx, val, ws.cand, nofine);
            if (dirty) flush_hist(hist, kDigit2, ws.hist2 + int64_t(s) * kDigit2);
            dirty = false;
            s = segment_after(ws.tile_prefix, nseg, s, t);
            next = ws.tile_prefix[s + 1];
            inf = ws.info[s];
            st = ws.st + s;
            mode = st->mode;
            D1 = st->d1;
        }
        if (mode == kModeNone || mode == kModeFast || mode == kModeDone) {
            t = next - 1;  // nothing to do in this segment: skip its tiles
            continue;
        }
        const TileRange r = tile_range(inf, t);
        float p[kVecPerThread][4];
        uint32_t valid = 0;
        if (kAligned && r.lo == r.block0 && r.hi == r.block0 + kTile) {
            const f32x4 *e4 = reinterpret_cast<const f32x4 *>(e + r.block0);
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
                const f32x4 v = e4[j * kBlock + threadIdx.x];
#pragma unroll
                for (int c = 0; c < 4; ++c) p[j][c] = v[c];
            }
            valid = 0xffffu;
        } else {
            const float *eb = e + r.block0;
            const uint32_t lo = uint32_t(r.lo - r.block0), hi = uint32_t(r.hi - r.block0);
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
                for (int c = 0; c < 4; ++c) p[j][c] = 0.0f;
                if (!slice_meets(j, lo, hi)) continue;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t o = tile_off(j, c);
                    if (o >= lo && o < hi) {
                        p[j][c] = eb[o];
                        valid |= 1u << (4 * j + c);
                    }
                }
            }
        }
        uint32_t emit_mask = 0, cand_mask = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t bit = 1u << (4 * j + c);
                if (!(valid & bit)) continue;
                const uint32_t key = magnitude_key(p[j][c]);
                const uint32_t dg = key >> kShift1;
                if (mode == kModeAll || (mode == kModeCand && dg > D1)) emit_mask |= bit;
                if (dg == D1 && mode != kModeAll) {
                    atomicAdd(&hist[(key >> kShift2) & (kDigit2 - 1)], 1u);
                    if (mode == kModeCand) cand_mask |= bit;
                }
            }
        }
        dirty = dirty || mode != kModeAll;
        if (mode != kModeScan)
            stage_tile(sg, efill, cfill, p, r.block0, emit_mask, cand_mask, inf, st, ws.cand, idx,
                       val, e, true, nofine);
    }
    flush_both(sg, efill, cfill, st, inf, idx, val, ws.cand, nofine);
    if (dirty) flush_hist(hist, kDigit2, ws.hist2 + int64_t(s) * kDigit2);
}

// One work item of a segment on the bracket path (select1 lists them), run
// by one wave (the four waves of a workgroup take four items at once, so a
// workgroup's items cost a quarter of the dependent round trips in turn):
//   kind 0: payload slots [first, first + kChunk) of the pairs above the
//           bracket: their e is cleared (pass1 left it for a fallback);
//   kind 1: candidates [first, first + kChunk): bins above da to the payload
//           (e cleared), bin da appended to the list after the candidates,
//           kWorkPerLane per lane behind one pair of atomics.

__device__ void bracket_work(uint2 item, float *__restrict__ e, int32_t *__restrict__ idx,
                             float *__restrict__ val, const SegWs &ws) {
    const int32_t s = int32_t(item.x & 0x7fffffffu);
    const uint32_t first = item.y;
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const SegInfo inf = ws.info[s];
    SegState *st = ws.st + s;
    if (!(item.x >> 31)) {
        const uint32_t end = min(first + kChunk, st->ecut);
        for (uint32_t q = first + lane; q < end; q += kWave) e[idx[inf.kout + q]] = 0.0f;
        return;
    }
    const uint32_t lo = st->lo, shift = st->shift, da = st->da, ccur = st->ccur;
    const uint32_t end = min(first + kChunk, ccur);
    const uint2 *cand = ws.cand + inf.coff;
    uint2 v[kWorkPerLane];
    uint32_t keep = 0u, tie = 0u;
#pragma unroll
    for (int u = 0; u < kWorkPerLane; ++u) {
        const uint32_t q = first + uint32_t(u * kWave) + lane;
        v[u] = make_uint2(0u, 0u);
        if (q < end) {
            v[u] = cand[q];
            const uint32_t bin = ((v[u].x & 0x7fffffffu) - lo) >> shift;
            keep |= uint32_t(bin > da) << u;
            tie |= uint32_t(bin == da) << u;
        }
    }
    uint32_t tk, tt;
    uint32_t pk = wave_prefix_small(uint32_t(__popc(keep)), tk);
    uint32_t pt = wave_prefix_small(uint32_t(__popc(tie)), tt);
    uint32_t bk = 0u, bt = 0u;
    if (lane == 0u) {
        bk = tk ? atomicAdd(&st->emit, tk) : 0u;
        bt = tt ? atomicAdd(&st->tcur, tt) : 0u;
    }
    pk += uint32_t(__shfl(int(bk), 0));
    pt += uint32_t(__shfl(int(bt), 0));
#pragma unroll
    for (int u = 0; u < kWorkPerLane; ++u) {
        if ((keep >> u) & 1u) {
            if (int64_t(pk) < inf.k) {
                idx[inf.kout + pk] = int32_t(v[u].y);
                val[inf.kout + pk] = __uint_as_float(v[u].x);
                e[v[u].y] = 0.0f;
            }
            ++pk;
        }
        if ((tie >> u) & 1u) {
            if (int64_t(ccur) + pt < inf.ccap) ws.cand[inf.coff + ccur + pt] = v[u];
            ++pt;
        }
    }
}

template <bool kAligned>
__global__ __launch_bounds__(kBlock) void seg_pass2_kernel(float *__restrict__ e,
                                                           int32_t *__restrict__ idx,
                                                           float *__restrict__ val, int32_t nseg,
                                                           SegWs ws, uint32_t slice) {
    __shared__ uint32_t hist[kDigit2];
    __shared__ Stage sg;
    if (ws.ctl->status != 0u) return;
    const uint32_t T = ws.ctl->tiles;
    if (ws.ctl->pass2 != 0u)
        for (uint32_t t0 = blockIdx.x * slice; t0 < T; t0 += gridDim.x * slice) {
            const uint32_t t1 = min(T, t0 + slice);
            const uint32_t g1 = min((t1 - 1u) >> ws.sweep_shift, uint32_t(kSweepGroups - 1));
            uint32_t marked = 0u;
            for (uint32_t q = t0 >> ws.sweep_shift; q <= g1; ++q) marked |= ws.sweep[q];
            if (marked) pass2_tiles<kAligned>(e, idx, val, nseg, ws, t0, t1, hist, sg);
        }
    // work list: workgroup b owns slots b, b + grid, b + 2 grid, ... (a
    // segment's items are consecutive slots, so they spread over workgroups);
    // its threads read those slots together, then the workgroup runs the
    // items in use (select1 writes every slot each call).
    const uint32_t W = min(ws.ctl->wtotal, ws.work_cap);
    const uint32_t per = (W + gridDim.x - 1) / gridDim.x;
    uint2 *list = sg.cand;  // staging is flushed: its candidate area holds the slots in use
    for (uint32_t r0 = 0; r0 < per; r0 += kBlock) {
        const uint32_t r = r0 + threadIdx.x;
        const uint32_t w = blockIdx.x + r * gridDim.x;
        uint2 item = make_uint2(0u, 0u);
        bool use = false;
        if (r < per && w < W) {
            item = ws.work[w];
            use = item.x != kNoWork && (item.x & 0x7fffffffu) < uint32_t(nseg);
        }
        uint32_t n_use;
        const uint32_t pos = block_prefix_small(use ? 1u : 0u, sg.wave, n_use);
        if (use) list[pos] = item;
        __syncthreads();
        for (uint32_t q = threadIdx.x / kWave; q < n_use; q += kWaves)
            bracket_work(list[q], e, idx, val, ws);
        __syncthreads();  // the list is rewritten by the next round
    }
}

// ---------------------------------------------------------------------------
// final: each segment's exact threshold, its ties, the last pairs
// ---------------------------------------------------------------------------

template <int kCap>
struct FinalShared {
    static constexpr int cap = kCap;
    uint32_t hist[kIdxBins];
    uint2 cand[kCap];
    uint32_t wave[kWaves];
    uint32_t out[3];
    uint32_t cursor;
};

constexpr uint32_t kNone = 0xffffffffu;  // no item (larger than every index)
constexpr int kUnroll = 8;               // items loaded per thread at a time

// Calls f(key, index, bits of p) for every item of the segment's selection
// set: the candidate list (LDS or global), or, in scan mode, every element
// of the segment.  kUnroll loads per thread are in flight together.
template <int kMode, bool kLds, typename Sh, typename F>
__device__ __forceinline__ void for_items(const Sh &sh, const uint2 *cand,
                                          const float *e, const SegInfo &inf, int64_t n, F f) {
    for (int64_t base = 0; base < n; base += int64_t(kUnroll) * kBlock) {
        uint2 it[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t q = base + u * kBlock + threadIdx.x;
            it[u] = make_uint2(0u, kNone);
            if (q < n) {
                if (kMode == kModeCand) {
                    it[u] = kLds ? sh.cand[q] : cand[q];
                } else {
                    const int64_t i = inf.off + q;
                    it[u] = make_uint2(__float_as_uint(e[i]), uint32_t(i));
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (it[u].y != kNone) f(it[u].x & 0x7fffffffu, it[u].y, it[u].x);
    }
}

// With the threshold key T known and `need3` of the `ties` keys equal to T
// to keep: choose the ties (the lowest indices, by a radix select on the
// index: bits 30..20, 19..10, 9..0, unless all are kept), emit every item
// above T and the chosen ties from payload slot `cursor0` on, clear their e,
// and record T as the next call's hint.
template <int kMode, bool kLds, typename Sh>
__device__ void finish(Sh &sh, const SegInfo &inf, const uint2 *cand, int64_t n,
                       float *e, int32_t *idx, float *val, uint32_t T, uint32_t need3,
                       uint32_t ties, uint32_t cursor0, SegHint *hint, uint32_t width) {
    const int tid = threadIdx.x;
    uint32_t imax = 0xffffffffu;
    if (need3 < ties) {
        uint32_t prefix = 0, rem = need3;
#pragma unroll 1
        for (int level = 0; level < 3; ++level) {
            const int shift = 20 - 10 * level;
            for (int b = tid; b < kIdxBins; b += kBlock) sh.hist[b] = 0u;
            __syncthreads();
            for_items<kMode, kLds>(sh, cand, e, inf, n, [&](uint32_t key, uint32_t i, uint32_t) {
                if (key != T) return;
                if (level > 0 && (i >> (shift + 10)) != prefix) return;
                atomicAdd(&sh.hist[(i >> shift) & (level == 0 ? kIdxBins - 1 : 1023)], 1u);
            });
            __syncthreads();
            if (level == 0) pick_bin<kIdxBins, false>(sh.hist, rem, sh.wave, sh.out);
            else pick_bin<1024, false>(sh.hist, rem, sh.wave, sh.out);
            prefix = (prefix << (level == 0 ? 11 : 10)) | sh.out[0];
            rem -= sh.out[1];
            __syncthreads();
        }
        imax = prefix;
    }
    if (tid == 0) sh.cursor = cursor0;
    __syncthreads();
    const int64_t kend = inf.k;
    for_items<kMode, kLds>(sh, cand, e, inf, n, [&](uint32_t key, uint32_t i, uint32_t bits) {
        if (!(key > T || (key == T && i <= imax))) return;
        const uint32_t slot = atomicAdd(&sh.cursor, 1u);
        if (int64_t(slot) < kend) {
            idx[inf.kout + slot] = int32_t(i);
            val[inf.kout + slot] = __uint_as_float(bits);
            e[i] = 0.0f;
        }
    });
    if (tid == 0) {
        *hint = next_hint(*hint, T, width);
    }
}

// Radix path: D1 from pass1, digit 2 from pass2's histogram of the keys in
// D1, digit 3 from a pass over the items.  Scan mode also emits every key
// above D1 (pass2 left them in place).
template <int kMode, bool kLds, typename Sh>
__device__ void final_select(Sh &sh, const SegInfo &inf, const SegState &st,
                             const uint2 *cand, int64_t n, float *e, int32_t *idx, float *val,
                             const uint32_t *hist2, SegHint *hint, uint32_t width) {
    const int tid = threadIdx.x;
    const uint32_t D1 = st.d1;
    for (int b = tid; b < kDigit2; b += kBlock) sh.hist[b] = hist2[b];
    __syncthreads();
    pick_bin<kDigit2, true>(sh.hist, st.need1, sh.wave, sh.out);
    const uint32_t D2 = sh.out[0];
    const uint32_t need2 = st.need1 - sh.out[1];
    const uint32_t P2 = (D1 << (kShift1 - kShift2)) | D2;  // key >> kShift2 of (D1, D2)
    __syncthreads();
    for (int b = tid; b < kDigit3; b += kBlock) sh.hist[b] = 0u;
    __syncthreads();
    for_items<kMode, kLds>(sh, cand, e, inf, n, [&](uint32_t key, uint32_t, uint32_t) {
        if ((key >> kShift2) == P2) atomicAdd(&sh.hist[key & (kDigit3 - 1)], 1u);
    });
    __syncthreads();
    pick_bin<kDigit3, true>(sh.hist, need2, sh.wave, sh.out);
    const uint32_t T = (P2 << kShift2) | sh.out[0];
    const uint32_t need3 = need2 - sh.out[1];
    const uint32_t ties = sh.out[2];
    __syncthreads();
    finish<kMode, kLds>(sh, inf, cand, n, e, idx, val, T, need3, ties,
                        kMode == kModeCand ? st.emit : 0u, hint, width);
}

// Bracket path: pass1 put the keys above the bracket in the payload,
// pass2 cleared their e, emitted the candidates of the bracket bins above
// da and listed the `ca` candidates of bin da; rank those by the low
// `shift` bits of key - lo (the exact threshold T), then by index among
// keys equal to T, and emit the `needa` kept ones into the last slots.
template <bool kLds, typename Sh>
__device__ void final_fast(Sh &sh, const SegInfo &inf, const SegState &st,
                           const uint2 *list, int64_t n, float *e, int32_t *idx, float *val,
                           SegHint *hint, uint32_t width) {
    const int tid = threadIdx.x;
    if (st.needa == 0u) {  // the pairs above the bracket were exactly k
        if (tid == 0) {
            *hint = next_hint(*hint, min(st.hi, 0x7ffffffeu) + 1u, width);
        }
        return;
    }
    const uint32_t lo = st.lo, shift = st.shift;
    const uint32_t sub_mask = (1u << shift) - 1u;
    for (int b = tid; b < kIdxBins; b += kBlock) sh.hist[b] = 0u;
    __syncthreads();
    for_items<kModeCand, kLds>(sh, list, e, inf, n, [&](uint32_t key, uint32_t, uint32_t) {
        atomicAdd(&sh.hist[(key - lo) & sub_mask], 1u);
    });
    __syncthreads();
    pick_bin<kIdxBins, true>(sh.hist, st.needa, sh.wave, sh.out);
    const uint32_t T = lo + ((st.da << shift) | sh.out[0]);
    const uint32_t need3 = st.needa - sh.out[1];
    const uint32_t ties = sh.out[2];
    __syncthreads();
    finish<kModeCand, kLds>(sh, inf, list, n, e, idx, val, T, need3, ties,
                            uint32_t(inf.k) - st.needa, hint, width);
}

// The next bracket widths: the lower side narrower after a bracket that
// held many more keys below the threshold than the segment keeps, or more
// than it can hold; both sides wider after the threshold fell outside it.
__device__ __forceinline__ uint32_t next_width(const SegHint &oh, const SegState &st,
                                               const SegInfo &inf) {
    const uint32_t w0 = oh.magic == kHintMagic && widths_ok(oh.width)
                            ? oh.width : make_widths(kWidthStart, kWidthStart);
    uint32_t wl = width_lo(w0), wh = width_hi(w0);
    if (st.mode == kModeFast) {
        if (int64_t(st.ccur) - int64_t(st.need1) > inf.k + 1024 && wl > kWidthMin) --wl;
    } else if (st.bracket && st.miss == 3u) {
        if (wl > kWidthMin) --wl;
    } else if (st.bracket) {
        wl = min(wl + 1u, kWidthMax);
        wh = min(wh + 1u, kWidthMax);
    }
    return make_widths(wl, wh);
}

// The bracket path's final step for a segment whose bin da lists at most
// kWave keys, by one wave and without barriers: each lane ranks one listed
// key against the others (larger key first, then the lower index), the
// `needa` best are emitted into the segment's last slots with e cleared at
// them, and the key ranked needa-th is the threshold T kept as the next
// hint: the same result as final_fast.
__device__ __forceinline__ void final_fast_wave(float *__restrict__ e, int32_t *__restrict__ idx,
                                                float *__restrict__ val, const SegWs &ws,
                                                int32_t s) {
    const uint32_t lane = threadIdx.x & (kWave - 1);
    const SegState st = ws.st[s];
    const SegInfo inf = ws.info[s];
    SegHint *hint = ws.hint + s;
    const SegHint oh = *hint;
    const uint32_t width = next_width(oh, st, inf);
    if (st.needa == 0u) {  // the pairs above the bracket were exactly k
        if (lane == 0u) *hint = next_hint(oh, min(st.hi, 0x7ffffffeu) + 1u, width);
        return;
    }
    const uint32_t n = min(st.ca, st.tcur);  // at most kWave, at least needa
    const uint2 *list = ws.cand + inf.coff + st.ccur;
    const bool mine = lane < n;
    uint2 it = make_uint2(0u, 0u);
    if (mine) it = list[lane];
    const uint32_t key = it.x & 0x7fffffffu;
    uint32_t rank = 0;
#pragma unroll 1
    for (uint32_t j = 0; j < n; ++j) {
        const uint32_t kj = __builtin_amdgcn_readlane(key, j);
        const uint32_t ij = __builtin_amdgcn_readlane(it.y, j);
        rank += (kj > key || (kj == key && ij < it.y)) ? 1u : 0u;
    }
    const uint64_t at = __ballot(mine && rank == st.needa - 1u);
    const uint32_t T = __builtin_amdgcn_readlane(key, at != 0ull ? __builtin_ctzll(at) : 0);
    if (mine && rank < st.needa) {
        const int64_t slot = inf.k - int64_t(st.needa) + rank;
        idx[inf.kout + slot] = int32_t(it.y);
        val[inf.kout + slot] = __uint_as_float(it.x);
        e[it.y] = 0.0f;
    }
    if (lane == 0u) *hint = next_hint(oh, T, width);
}

template <typename Sh>
__device__ void final_segment(float *__restrict__ e, int32_t *__restrict__ idx,
                              float *__restrict__ val, const SegWs &ws, int32_t s, Sh &sh) {
    const SegState st = ws.st[s];
    if (st.mode != kModeCand && st.mode != kModeScan && st.mode != kModeFast) return;
    const SegInfo inf = ws.info[s];
    SegHint *hint = ws.hint + s;
    const uint32_t width = next_width(*hint, st, inf);
    const uint32_t *h2 = ws.hist2 + int64_t(s) * kDigit2;
    if (st.mode == kModeScan) {
        final_select<kModeScan, false>(sh, inf, st, nullptr, inf.size, e, idx, val, h2, hint, width);
        return;
    }
    // the candidates, or on the bracket path the list of bin da after them
    const bool fast = st.mode == kModeFast;
    const int64_t n = fast ? int64_t(st.needa ? min(st.ca, st.tcur) : 0u)
                           : min(int64_t(st.ccur), inf.ccap);
    const uint2 *cand = ws.cand + inf.coff + (fast ? st.ccur : 0u);
    const bool lds = n <= Sh::cap;
    if (lds) {
        for (int64_t base = 0; base < n; base += int64_t(kUnroll) * kBlock) {
            uint2 v[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int64_t q = base + u * kBlock + threadIdx.x;
                if (q < n) v[u] = cand[q];
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int64_t q = base + u * kBlock + threadIdx.x;
                if (q < n) sh.cand[q] = v[u];
            }
        }
        __syncthreads();
    }
    if (fast) {
        if (lds) final_fast<true>(sh, inf, st, cand, n, e, idx, val, hint, width);
        else final_fast<false>(sh, inf, st, cand, n, e, idx, val, hint, width);
    } else {
        if (lds) final_select<kModeCand, true>(sh, inf, st, cand, n, e, idx, val, h2, hint, width);
        else final_select<kModeCand, false>(sh, inf, st, cand, n, e, idx, val, h2, hint, width);
    }
}

// One workgroup per CU at most with the large candidate buffer, four with
// the small one (a larger list is ranked from global memory), looping over
// the segments b, b + grid, ...  Most need nothing here (one tile, none,
// all), so the workgroup first reads the modes of up to kBlock of its
// segments at once and then runs only those with something to rank (one
// dependent read per segment in turn was the larger cost with thousands of
// segments).
template <int kCap>
__global__ __launch_bounds__(kBlock) void seg_final_kernel(float *__restrict__ e,
                                                           int32_t *__restrict__ idx,
                                                           float *__restrict__ val, SegWs ws,
                                                           int32_t nseg) {
    __shared__ FinalShared<kCap> sh;
    __shared__ int32_t s_list[kBlock];
    __shared__ uint32_t s_wave[kWaves];
    if (ws.ctl->status != 0u) return;
    uint32_t fast = 0;  // segments resolved from the bracket, counted per thread
    const int32_t per = (nseg - int32_t(blockIdx.x) + int32_t(gridDim.x) - 1) / int32_t(gridDim.x);
    const uint32_t wave = threadIdx.x / kWave;
    for (int32_t g0 = 0; g0 < per; g0 += kBlock) {
        const int32_t q = g0 + int32_t(threadIdx.x);
        const int32_t s = int32_t(blockIdx.x) + q * int32_t(gridDim.x);
        uint32_t mode = kModeNone, listed = 0u;
        if (q < per) {
            const SegState *p = ws.st + s;
            mode = p->mode;
            if (mode == kModeFast) listed = p->needa != 0u ? min(p->ca, p->tcur) : 0u;
        }
        fast += mode == kModeFast ? 1u : 0u;
        // bracket-path segments with at most kWave keys to rank go to the
        // waves (listed from the end of s_list), the rest to the workgroup
        const bool small = mode == kModeFast && listed <= uint32_t(kWave);
        const bool work = !small && (mode == kModeCand || mode == kModeScan || mode == kModeFast);
        uint32_t n_work, n_small;
        const uint32_t pos = block_prefix_small(work ? 1u : 0u, s_wave, n_work);
        const uint32_t spos = block_prefix_small(small ? 1u : 0u, s_wave, n_small);
        if (work) s_list[pos] = s;
        if (small) s_list[kBlock - 1 - int(spos)] = s;
        __syncthreads();
        for (uint32_t i = wave; i < n_small; i += kWaves)
            final_fast_wave(e, idx, val, ws, s_list[kBlock - 1 - int(i)]);
        for (uint32_t i = 0; i < n_work; ++i) {
            final_segment(e, idx, val, ws, s_list[i], sh);
            __syncthreads();  // the LDS of this segment is free
        }
    }
    fast = block_sum(fast, s_wave);
    if (threadIdx.x == 0 && fast != 0u) atomicAdd(&ws.ctl->bracket, fast);
}

}  // namespace

size_t topk_segmented_workspace_size(int32_t nseg, int64_t k_total) {
    return seg_layout(nseg, k_total).bytes;
}

size_t topk_segmented_status_offset() { return offsetof(SegCtl, status); }
size_t topk_segmented_bracket_offset() { return offsetof(SegCtl, bracket); }

hipError_t launch_topk_segmented(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                                 const int64_t *offsets, const int64_t *k, int64_t k_total,
                                 int32_t *idx, float *val, void *workspace, hipStream_t stream) {
    const SegLayout L = seg_layout(nseg, k_total);
    char *base = static_cast<char *>(workspace);
    SegWs ws = {};
    ws.ctl = reinterpret_cast<SegCtl *>(base);
    ws.info = reinterpret_cast<SegInfo *>(base + L.info);
    ws.tile_prefix = reinterpret_cast<uint32_t *>(base + L.tile_prefix);
    ws.st = reinterpret_cast<SegState *>(base + L.st);
    ws.hint = reinterpret_cast<SegHint *>(base + L.hint);
    ws.hist1 = reinterpret_cast<uint32_t *>(base + L.hist1);
    ws.hist2 = reinterpret_cast<uint32_t *>(base + L.hist2);
    ws.cand = reinterpret_cast<uint2 *>(base + L.cand);
    ws.work = reinterpret_cast<uint2 *>(base + L.work);
    ws.chunks = reinterpret_cast<ResetChunk *>(base + L.chunks);
    ws.sweep = reinterpret_cast<uint32_t *>(base + L.sweep);
    ws.ccap_total = L.ccap_total;
    ws.work_cap = uint32_t(L.work_cap);
    // every tile index is below ceil(d / kTile) + nseg, so its group is below
    // kSweepGroups
    const int64_t max_tiles = (d + kTile - 1) / kTile + nseg;
    while (((max_tiles - 1) >> ws.sweep_shift) >= kSweepGroups) ++ws.sweep_shift;

    const uint32_t zero_grid = persistent_grid(nseg);  // one segment's histograms per pass
    if (nseg <= kResetSingleMax) {
        seg_reset_kernel<<<1 + zero_grid, kResetBlock, 0, stream>>>(ws, offsets, k, nseg, d, k_total);
    } else {
        const int32_t nchunks = (nseg + kResetBlock - 1) / kResetBlock;
        seg_reset_sums_kernel<<<uint32_t(nchunks) + zero_grid, kResetBlock, 0, stream>>>(
            ws, offsets, k, nseg, d, nchunks);
        seg_reset_tables_kernel<<<uint32_t(nchunks), kResetBlock, 0, stream>>>(ws, offsets, k, nseg,
                                                                               d, k_total, nchunks);
    }

    // slices: the tiles spread over kSliceWorkgroupsPerCU workgroups per CU
    // (4 resident), at most kSliceTilesMax tiles each (kSliceTilesMaxMany
    // with many segments)
    const int64_t wgs = int64_t(device_cu_count()) * kSliceWorkgroupsPerCU;
    const int64_t slice_max = nseg > kSearchTwoRounds ? kSliceTilesMaxMany : kSliceTilesMax;
    const int64_t slice = max(int64_t(1), min(slice_max, (max_tiles + wgs - 1) / wgs));
    const uint32_t grid = uint32_t(min(wgs, (max_tiles + slice - 1) / slice));
    const bool aligned = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(e)) & 15) == 0;
    if (aligned)
        seg_pass1_kernel<true><<<grid, kBlock, 0, stream>>>(g, e, lr, idx, val, nseg, ws, uint32_t(slice));
    else
        seg_pass1_kernel<false><<<grid, kBlock, 0, stream>>>(g, e, lr, idx, val, nseg, ws, uint32_t(slice));
    seg_select1_kernel<<<uint32_t(nseg), kBlock, 0, stream>>>(ws, e);
    if (aligned)
        seg_pass2_kernel<true><<<grid, kBlock, 0, stream>>>(e, idx, val, nseg, ws, uint32_t(slice));
    else
        seg_pass2_kernel<false><<<grid, kBlock, 0, stream>>>(e, idx, val, nseg, ws, uint32_t(slice));
    const int64_t cus = device_cu_count();
    if (nseg > kFinalWideMin)
        seg_final_kernel<kCandLdsSmall><<<uint32_t(min(int64_t(nseg), 4 * cus)), kBlock, 0, stream>>>(
            e, idx, val, ws, nseg);
    else
        seg_final_kernel<kCandLds><<<uint32_t(min(int64_t(nseg), cus)), kBlock, 0, stream>>>(
            e, idx, val, ws, nseg);
    return hipGetLastError();
}

}  // namespace efs
