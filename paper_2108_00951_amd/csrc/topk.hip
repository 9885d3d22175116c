// Exact Top-k sparsifier with error feedback (Algorithm 1 with Top-k; the
// per-iteration optimum of Lemma 2).
//
// Keys are the 31-bit patterns of |p| (monotone in |p| for non-NaN values),
// ranked larger first and, on equal keys, lower index first.  The k-th key T
// is found by radix select over three digits (bits 30..20, 19..10, 9..0); the
// paper notes radix select costs O(ceil(b/r) d) (section 1), here b = 31 and
// r = 11/10/10.  Launches, all on the caller's stream:
//
//   reset    zero the control block and histograms (one workgroup).
//   pass1    p = e + lr*g, written into e (12 B/element); workgroup-local LDS
//            histogram of the top digit, merged into global bins.
//   select   (one workgroup) the bin holding rank k, i.e. the next digit of T.
//   refine   (x2, each followed by select) read p (4 B/element); histogram
//            the next digit of the keys that match the known prefix.  After
//            the third select T is exact, with G = #(key > T) and m = k - G
//            of the `ties` keys equal to T to keep.
//   ties     only when 0 < m < ties: per-tile counts of key == T, then their
//            exclusive scan (one workgroup), so every tied element knows its
//            rank in index order (both return at once otherwise).
//   emit     read p (4 B/element); keep key > T and the tied elements whose
//            rank is below m; compact the k pairs (ballot prefix sums into an
//            LDS stage, one atomic per flush) and zero e at the kept
//            coordinates.
//
// Workgroups exchange data only through global atomics and kernel
// boundaries; no kernel waits on another workgroup.
//
// Workspace (all offsets 256-byte aligned):
//   [0, 256)                  TopkCtl
//   [256, 256 + 16 KiB)       histograms: 2048 + 1024 + 1024 uint32
//   [.., + 4*ntiles)          per-tile tie counts (exclusive prefix after scan)
#include "device_common.hpp"
#include "launch.hpp"

namespace efs {

namespace {

constexpr int kBins1 = 2048;  // bits 30..20
constexpr int kBins2 = 1024;  // bits 19..10
constexpr int kBins3 = 1024;  // bits 9..0

struct TopkCtl {
    uint32_t prefix;     // known high bits of T (11, then 21, then all 31)
    uint32_t need;       // elements still to take from the bucket `prefix`
    uint32_t T;          // threshold key
    uint32_t m;          // tied elements (key == T) to keep
    uint32_t ties;       // elements with key == T
    uint32_t tie_mode;   // 1 when 0 < m < ties (rank ties by index)
    uint32_t emitted;    // pairs emitted by the last call (equals k)
    uint32_t pad[9];
    unsigned long long emit;  // compaction word: workgroup tickets << 40 | pairs
};
static_assert(sizeof(TopkCtl) <= 256, "control block must fit its slot");

constexpr size_t kCtlBytes = 256;
constexpr size_t kHistBytes = sizeof(uint32_t) * (kBins1 + kBins2 + kBins3);

struct Workspace {
    TopkCtl *ctl;
    uint32_t *hist1, *hist2, *hist3, *tile_ties;
};

Workspace carve(void *ws) {
    char *b = static_cast<char *>(ws);
    Workspace w;
    w.ctl = reinterpret_cast<TopkCtl *>(b);
    w.hist1 = reinterpret_cast<uint32_t *>(b + kCtlBytes);
    w.hist2 = w.hist1 + kBins1;
    w.hist3 = w.hist2 + kBins2;
    w.tile_ties = reinterpret_cast<uint32_t *>(b + kCtlBytes + kHistBytes);
    return w;
}

// Loads the 16 values element (j, c) of a tile for this thread into v, with
// the same element map as the hard-threshold kernel:
//   index = tile0 + (j * kBlock + tid) * 4 + c.
// Elements past d read as NaN-free zeros and are flagged invalid in `valid`.
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

// Called by every thread of one workgroup.  Bins are ranked from the top
// (highest bin first); finds the bin where the running count first reaches
// `need` (1 <= need <= sum of bins).  Thread 0 of the owning chunk writes
// {bin, count above the bin, count in the bin} to s_out.
template <int kBins>
__device__ void select_bin(const uint32_t *hist, uint32_t need, uint32_t *s_scan,
                           uint32_t *s_out) {
    constexpr int kPer = kBins / kBlock;
    const int t = threadIdx.x;
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
    s_scan[t] = tot;
    __syncthreads();
    for (int off = 1; off < kBlock; off <<= 1) {
        const uint32_t add = t >= off ? s_scan[t - off] : 0u;
        __syncthreads();
        s_scan[t] += add;
        __syncthreads();
    }
    const uint32_t incl = s_scan[t];
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

__global__ __launch_bounds__(kBlock) void topk_reset_kernel(TopkCtl *ctl, uint32_t *hist,
                                                            uint32_t k) {
    uint32_t *w = reinterpret_cast<uint32_t *>(ctl);
    for (int i = threadIdx.x; i < int(kCtlBytes / 4); i += kBlock) w[i] = 0u;
    for (int i = threadIdx.x; i < kBins1 + kBins2 + kBins3; i += kBlock) hist[i] = 0u;
    if (threadIdx.x == 0) ctl->need = k;
}

template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_pass1_kernel(const float *__restrict__ g,
                                                            float *__restrict__ e, int64_t d,
                                                            float lr, uint32_t ntiles,
                                                            Workspace ws) {
    __shared__ uint32_t h[kBins1];
    const int tid = threadIdx.x;
    for (int b = tid; b < kBins1; b += kBlock) h[b] = 0u;
    __syncthreads();

    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
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
                f32x4 p;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    p[c] = ef_accumulate(ev[j][c], lr, gv[j][c]);
                    atomicAdd(&h[magnitude_key(p[c]) >> 20], 1u);
                }
                e4[j * kBlock + tid] = p;
            }
        } else {
#pragma unroll
            for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int64_t i = elem_index(tile0, j, c);
                    if (i < d) {
                        const float p = ef_accumulate(e[i], lr, g[i]);
                        e[i] = p;
                        atomicAdd(&h[magnitude_key(p) >> 20], 1u);
                    }
                }
            }
        }
    }
    __syncthreads();
    for (int b = tid; b < kBins1; b += kBlock)
        if (h[b]) atomicAdd(ws.hist1 + b, h[b]);
}

// Refinement pass: histogram of bits [kShift, kShift+10) over the keys whose
// bits above kShift+10 equal the prefix found so far.
template <bool kVector, int kShift>
__global__ __launch_bounds__(kBlock) void topk_refine_kernel(const float *__restrict__ e,
                                                             int64_t d, uint32_t ntiles,
                                                             Workspace ws) {
    constexpr int kBins = 1024;
    __shared__ uint32_t h[kBins];
    const int tid = threadIdx.x;
    uint32_t *hist = kShift == 10 ? ws.hist2 : ws.hist3;
    for (int b = tid; b < kBins; b += kBlock) h[b] = 0u;
    const uint32_t prefix = ws.ctl->prefix;
    __syncthreads();

    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float v[kVecPerThread][4];
        uint32_t valid;
        load_tile<kVector>(e, tile0, d, v, valid);
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t key = magnitude_key(v[j][c]);
                if (((valid >> (4 * j + c)) & 1u) && (key >> (kShift + 10)) == prefix)
                    atomicAdd(&h[(key >> kShift) & (kBins - 1)], 1u);
            }
        }
    }
    __syncthreads();
    for (int b = tid; b < kBins; b += kBlock)
        if (h[b]) atomicAdd(hist + b, h[b]);
}

// One workgroup: picks the bin of the histogram of pass kPass (1, 2, 3) that
// holds rank `need`, and narrows the threshold prefix.  After pass 3 the
// threshold key T, the tie count and the number m of ties to keep are known.
template <int kPass>
__global__ __launch_bounds__(kBlock) void topk_select_kernel(Workspace ws) {
    __shared__ uint32_t s_scan[kBlock];
    __shared__ uint32_t s_sel[4];
    const uint32_t need = ws.ctl->need;
    const uint32_t prefix = ws.ctl->prefix;
    if (kPass == 1)
        select_bin<kBins1>(ws.hist1, need, s_scan, s_sel);
    else
        select_bin<1024>(kPass == 2 ? ws.hist2 : ws.hist3, need, s_scan, s_sel);
    if (threadIdx.x != 0) return;
    const uint32_t np = kPass == 1 ? s_sel[0] : ((prefix << 10) | s_sel[0]);
    ws.ctl->prefix = np;
    if (kPass < 3) {
        ws.ctl->need = need - s_sel[1];
    } else {
        const uint32_t m = need - s_sel[1];
        ws.ctl->T = np;
        ws.ctl->m = m;
        ws.ctl->ties = s_sel[2];
        ws.ctl->tie_mode = m < s_sel[2] ? 1u : 0u;
    }
}

// Tie ranks (only when some but not all elements tied at T are kept): count
// key == T per tile, then an exclusive scan over tiles in index order.
template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_ties_kernel(const float *__restrict__ e,
                                                           int64_t d, uint32_t ntiles,
                                                           Workspace ws) {
    __shared__ uint32_t s_wave[kWaves];
    if (ws.ctl->tie_mode == 0u) return;
    const uint32_t T = ws.ctl->T;
    const int tid = threadIdx.x;
    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float v[kVecPerThread][4];
        uint32_t valid;
        load_tile<kVector>(e, tile0, d, v, valid);
        uint32_t cnt = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                cnt += (((valid >> (4 * j + c)) & 1u) && magnitude_key(v[j][c]) == T) ? 1u : 0u;
        uint32_t total;
        block_prefix_small(cnt, s_wave, total);
        if (tid == 0) ws.tile_ties[tile] = total;
    }
}

// Exclusive scan of tile_ties[0..ntiles) in place by one workgroup; each
// thread owns a contiguous chunk.
__global__ __launch_bounds__(kBlock) void topk_ties_scan_kernel(uint32_t ntiles, Workspace ws) {
    __shared__ uint32_t s_scan[kBlock];
    if (ws.ctl->tie_mode == 0u) return;
    const int tid = threadIdx.x;
    const uint32_t chunk = (ntiles + kBlock - 1) / kBlock;
    const uint32_t lo = min(ntiles, tid * chunk);
    const uint32_t hi = min(ntiles, lo + chunk);
    uint32_t sum = 0;
    for (uint32_t i = lo; i < hi; ++i) sum += ws.tile_ties[i];
    s_scan[tid] = sum;
    __syncthreads();
    for (int off = 1; off < kBlock; off <<= 1) {
        const uint32_t add = tid >= off ? s_scan[tid - off] : 0u;
        __syncthreads();
        s_scan[tid] += add;
        __syncthreads();
    }
    uint32_t run = s_scan[tid] - sum;
    for (uint32_t i = lo; i < hi; ++i) {
        const uint32_t c = ws.tile_ties[i];
        ws.tile_ties[i] = run;
        run += c;
    }
}

template <bool kVector>
__global__ __launch_bounds__(kBlock) void topk_emit_kernel(float *__restrict__ e, int64_t d,
                                                           int32_t *__restrict__ idx,
                                                           float *__restrict__ val,
                                                           uint64_t cap, uint32_t ntiles,
                                                           Workspace ws) {
    __shared__ PairStage st;
    const int tid = threadIdx.x;
    const uint32_t T = ws.ctl->T;
    const bool tie_mode = ws.ctl->tie_mode != 0u;
    const uint32_t m = ws.ctl->m;
    uint32_t fill = 0;

    for (uint32_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t tile0 = int64_t(tile) * kTile;
        float v[kVecPerThread][4];
        uint32_t valid;
        load_tile<kVector>(e, tile0, d, v, valid);
        uint32_t keep = 0, tie = 0;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int b = 4 * j + c;
                const uint32_t key = magnitude_key(v[j][c]);
                const bool ok = (valid >> b) & 1u;
                keep |= uint32_t(ok && key > T) << b;
                tie |= uint32_t(ok && key == T) << b;
            }
        }
        if (!tie_mode) {
            keep |= tie;
        } else {
            // Rank of each tied element in index order: earlier tiles, then
            // earlier vector slots j (all lower indices), then lower threads
            // in slot j, then lower c within the thread.
            uint32_t rank = ws.tile_ties[tile];
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
        }

        uint32_t total;
        const uint32_t pos = block_prefix_small(__popc(keep), st.wave, total);
        if (total == 0) continue;
        if (fill + total > uint32_t(kTile)) {
            stage_flush(st, fill, false, &ws.ctl->emit, nullptr, cap, idx, val);
            fill = 0;
        }
        uint32_t o = fill + pos;
#pragma unroll
        for (int j = 0; j < kVecPerThread; ++j) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if ((keep >> (4 * j + c)) & 1u) {
                    const int64_t i = elem_index(tile0, j, c);
                    st.idx[o] = int32_t(i);
                    st.val[o] = v[j][c];
                    e[i] = 0.0f;
                    ++o;
                }
            }
        }
        fill += total;
    }
    stage_flush(st, fill, true, &ws.ctl->emit, &ws.ctl->emitted, cap, idx, val);
}

}  // namespace

size_t topk_workspace_size(int64_t d) {
    const int64_t tiles = d > 0 ? (d + kTile - 1) / kTile : 1;
    const size_t bytes = kCtlBytes + kHistBytes + sizeof(uint32_t) * size_t(tiles);
    return (bytes + 255) & ~size_t(255);
}

hipError_t launch_topk(const float *g, float *e, int64_t d, float lr, int64_t k,
                       int32_t *idx, float *val, void *workspace, hipStream_t stream) {
    if (d == 0) return hipSuccess;
    const uint32_t ntiles = uint32_t((d + kTile - 1) / kTile);
    const uint32_t grid = balanced_grid(ntiles, kScanWorkgroupsPerCU);
    const uint32_t egrid = balanced_grid(ntiles, kStageWorkgroupsPerCU);
    const Workspace ws = carve(workspace);
    const bool vec = ((reinterpret_cast<uintptr_t>(g) | reinterpret_cast<uintptr_t>(e)) & 15u) == 0;

    topk_reset_kernel<<<1, kBlock, 0, stream>>>(ws.ctl, ws.hist1, uint32_t(k));
    if (vec)
        topk_pass1_kernel<true><<<grid, kBlock, 0, stream>>>(g, e, d, lr, ntiles, ws);
    else
        topk_pass1_kernel<false><<<grid, kBlock, 0, stream>>>(g, e, d, lr, ntiles, ws);
    if (k == 0) return hipGetLastError();
    topk_select_kernel<1><<<1, kBlock, 0, stream>>>(ws);
    if (vec) {
        topk_refine_kernel<true, 10><<<grid, kBlock, 0, stream>>>(e, d, ntiles, ws);
        topk_select_kernel<2><<<1, kBlock, 0, stream>>>(ws);
        topk_refine_kernel<true, 0><<<grid, kBlock, 0, stream>>>(e, d, ntiles, ws);
        topk_select_kernel<3><<<1, kBlock, 0, stream>>>(ws);
        topk_ties_kernel<true><<<grid, kBlock, 0, stream>>>(e, d, ntiles, ws);
        topk_ties_scan_kernel<<<1, kBlock, 0, stream>>>(ntiles, ws);
        topk_emit_kernel<true><<<egrid, kBlock, 0, stream>>>(e, d, idx, val, uint64_t(k), ntiles, ws);
    } else {
        topk_refine_kernel<false, 10><<<grid, kBlock, 0, stream>>>(e, d, ntiles, ws);
        topk_select_kernel<2><<<1, kBlock, 0, stream>>>(ws);
        topk_refine_kernel<false, 0><<<grid, kBlock, 0, stream>>>(e, d, ntiles, ws);
        topk_select_kernel<3><<<1, kBlock, 0, stream>>>(ws);
        topk_ties_kernel<false><<<grid, kBlock, 0, stream>>>(e, d, ntiles, ws);
        topk_ties_scan_kernel<<<1, kBlock, 0, stream>>>(ntiles, ws);
        topk_emit_kernel<false><<<egrid, kBlock, 0, stream>>>(e, d, idx, val, uint64_t(k), ntiles, ws);
    }
    return hipGetLastError();
}

}  // namespace efs
