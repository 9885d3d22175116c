// Host-side launchers of the efsparse kernels.  Arguments arrive here
// already validated by the C ABI layer (abi.cpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace efs {

hipError_t launch_ht(const float *g, float *e, int64_t d, float lr, float lambda,
                     int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                     void *telemetry, hipStream_t stream);

size_t topk_workspace_size(int64_t d, int64_t k);
size_t topk_path_flag_offset();
hipError_t launch_topk(const float *g, float *e, int64_t d, float lr, int64_t k,
                       int32_t *idx, float *val, void *workspace, hipStream_t stream);

// Layer-wise Top-k (topk_seg.hip).
constexpr int32_t kMaxSegments = 1 << 16;
size_t topk_segmented_workspace_size(int32_t nseg, int64_t k_total);
size_t topk_segmented_status_offset();
size_t topk_segmented_bracket_offset();
hipError_t launch_topk_segmented(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                                 const int64_t *offsets, const int64_t *k, int64_t k_total,
                                 int32_t *idx, float *val, void *workspace, hipStream_t stream);

// Exchange-and-average, alone (mode 0) or fused with the model update
// (apply.hip).  Status bits of the last call, at apply_status_offset() in the
// workspace.
constexpr int kMaxApplyWorkers = 64;
constexpr uint32_t kSparseTruncated = 1u;   // a count exceeded its payload's capacity
constexpr uint32_t kSparseBadIndex = 2u;    // an index outside [0, d) was ignored
// Workspace of the packed layout (four launches) and of the bucketed one
// (two launches, taken whenever the workspace holds it).
size_t apply_workspace_size(int32_t n, int64_t d, int64_t total_cap);
size_t apply_bucket_workspace_size(int32_t n, int64_t d);
size_t apply_status_offset();
hipError_t launch_apply(const int32_t *const *idx, const float *const *val,
                        const uint32_t *const *counts, const int64_t *caps, int32_t n,
                        int64_t d, int mode, float *x, float *m, float beta, float gamma,
                        void *workspace, size_t workspace_bytes, hipStream_t stream);

// Scratch held by the library per device for sparse_accumulate_static
// (scratch.hip): its device address on the current device.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch(void **ptr);

hipError_t launch_copy(const float *src, float *dst, int64_t n, bool per_tile, hipStream_t stream);
hipError_t launch_stream_probe(const float *x, float *y, int64_t n, int mode, bool per_tile,
                               hipStream_t stream);

// Workgroups for a grid-stride pass over `work_tiles` tiles: enough to fill
// every compute unit several times over, never more than there is work.
uint32_t persistent_grid(int64_t work_tiles);

// Compute units of the current device (queried once per device).
int device_cu_count();

// Grid for a grid-stride pass in which every workgroup stays resident: the
// fewest tiles per workgroup that the resident workgroups allow, and just
// enough workgroups to cover the tiles at that count (so no workgroup does
// more than one tile beyond any other).
uint32_t balanced_grid(int64_t work_tiles, int workgroups_per_cu);

}  // namespace efs
