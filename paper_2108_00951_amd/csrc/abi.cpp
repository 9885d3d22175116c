// C ABI of libefsparse.so: host-side argument validation, status codes and
// dispatch to the kernel launchers.  Nothing here touches the device until
// every argument has been checked; nothing here allocates or synchronises.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "../../include/efsparse.h"
#include "launch.hpp"
#include "device_common.hpp"

static_assert(efs::kMaxApplyWorkers == EFS_MAX_WORKERS, "worker limit differs from the header");
static_assert(efs::kSparseTruncated == EFS_SPARSE_TRUNCATED, "status bit differs from the header");
static_assert(efs::kSparseBadIndex == EFS_SPARSE_BAD_INDEX, "status bit differs from the header");
static_assert(efs::kMaxSegments == EFS_SEG_MAX, "segment limit differs from the header");
static_assert(efs::kStaticScratchBytes == EFS_STATIC_SCRATCH_BYTES, "scratch size differs from the header");
static_assert(sizeof(efs::Telemetry) == EFS_TELEMETRY_BYTES, "telemetry layout differs from the header");

namespace {

thread_local char g_message[256] = "";
thread_local efs_status g_sticky = EFS_OK;  // last non-OK status on this thread

efs_status fail(efs_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_message, sizeof g_message, fmt, ap);
    va_end(ap);
    g_sticky = s;
    return s;
}

efs_status check_launch(hipError_t err, const char *what) {
    if (err != hipSuccess)
        return fail(EFS_EHIP, "%s: kernel launch failed: %s", what, hipGetErrorString(err));
    return EFS_OK;
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

constexpr int64_t kMaxLen = INT32_MAX;

int g_cu_count[64];  // per device; 0 = not queried yet

}  // namespace

namespace efs {

int device_cu_count() {
    int dev = 0;
    int cus = 256;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64) {
        if (g_cu_count[dev] == 0) {
            int v = 0;
            if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                v > 0)
                g_cu_count[dev] = v;
            else
                g_cu_count[dev] = 256;
        }
        cus = g_cu_count[dev];
    }
    return cus;
}

uint32_t balanced_grid(int64_t work_tiles, int workgroups_per_cu) {
    if (work_tiles < 1) work_tiles = 1;
    const int64_t resident = int64_t(device_cu_count()) * workgroups_per_cu;
    const int64_t per_wg = (work_tiles + resident - 1) / resident;
    return uint32_t((work_tiles + per_wg - 1) / per_wg);
}

uint32_t persistent_grid(int64_t work_tiles) {
    const int64_t cap = int64_t(device_cu_count()) * 8;
    if (work_tiles < 1) work_tiles = 1;
    return uint32_t(work_tiles < cap ? work_tiles : cap);
}

}  // namespace efs

extern "C" {

const char *efs_status_string(efs_status s) {
    switch (s) {
        case EFS_OK: return "ok";
        case EFS_EINVAL: return "invalid argument";
        case EFS_ESPACE: return "workspace too small";
        case EFS_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char *efs_last_error_message(void) { return g_message; }

efs_status efs_last_error(void) {
    if (hipPeekAtLastError() != hipSuccess) return EFS_EHIP;
    const efs_status s = g_sticky;
    g_sticky = EFS_OK;
    return s;
}

static efs_status ht_common(const char *name, const float *g, float *e, int64_t d, float lr,
                            float lambda, int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                            void *telemetry, void *stream) {
    if (d < 0 || d > kMaxLen) return fail(EFS_EINVAL, "%s: d=%lld outside [0, 2^31-1]", name, (long long)d);
    if (d > 0 && (g == nullptr || e == nullptr)) return fail(EFS_EINVAL, "%s: g or e is NULL", name);
    if (!aligned(g, 4) || !aligned(e, 4)) return fail(EFS_EINVAL, "%s: g and e must be 4-byte aligned", name);
    if (!std::isfinite(lr)) return fail(EFS_EINVAL, "%s: lr must be finite", name);
    if (std::isnan(lambda) || lambda < 0.0f) return fail(EFS_EINVAL, "%s: lambda must be >= 0 and not NaN", name);
    if (cap < 0 || cap > kMaxLen) return fail(EFS_EINVAL, "%s: cap=%lld outside [0, 2^31-1]", name, (long long)cap);
    if (cap > 0 && (idx == nullptr || val == nullptr)) return fail(EFS_EINVAL, "%s: idx or val is NULL", name);
    if (!aligned(idx, 4) || !aligned(val, 4)) return fail(EFS_EINVAL, "%s: idx and val must be 4-byte aligned", name);
    if (counter == nullptr || !aligned(counter, 8)) return fail(EFS_EINVAL, "%s: counter must be non-NULL and 8-byte aligned", name);
    return check_launch(efs::launch_ht(g, e, d, lr, lambda, idx, val, cap, counter, telemetry,
                                       static_cast<hipStream_t>(stream)),
                        name);
}

efs_status ht_compress(const float *g, float *e, int64_t d, float lr, float lambda,
                       int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                       void *stream) {
    return ht_common("ht_compress", g, e, d, lr, lambda, idx, val, cap, counter, nullptr, stream);
}

efs_status ht_compress_telemetry(const float *g, float *e, int64_t d, float lr, float lambda,
                                 int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                                 void *telemetry, void *stream) {
    if (telemetry == nullptr || !aligned(telemetry, 8))
        return fail(EFS_EINVAL, "ht_compress_telemetry: telemetry must be non-NULL and 8-byte aligned");
    return ht_common("ht_compress_telemetry", g, e, d, lr, lambda, idx, val, cap, counter,
                     telemetry, stream);
}

size_t topk_workspace_bytes(int64_t d, int64_t k) {
    if (d < 0 || d > kMaxLen || k < 0 || k > d) return 0;
    return efs::topk_workspace_size(d, k);
}

size_t topk_path_flag_offset(void) { return efs::topk_path_flag_offset(); }

efs_status topk_compress(const float *g, float *e, int64_t d, float lr, int64_t k,
                         int32_t *idx, float *val, void *workspace, size_t workspace_bytes,
                         void *stream) {
    if (d < 0 || d > kMaxLen) return fail(EFS_EINVAL, "topk_compress: d=%lld outside [0, 2^31-1]", (long long)d);
    if (k < 0 || k > d) return fail(EFS_EINVAL, "topk_compress: k=%lld outside [0, d]", (long long)k);
    if (d > 0 && (g == nullptr || e == nullptr)) return fail(EFS_EINVAL, "topk_compress: g or e is NULL");
    if (!aligned(g, 4) || !aligned(e, 4)) return fail(EFS_EINVAL, "topk_compress: g and e must be 4-byte aligned");
    if (!std::isfinite(lr)) return fail(EFS_EINVAL, "topk_compress: lr must be finite");
    if (k > 0 && (idx == nullptr || val == nullptr)) return fail(EFS_EINVAL, "topk_compress: idx or val is NULL");
    if (!aligned(idx, 4) || !aligned(val, 4)) return fail(EFS_EINVAL, "topk_compress: idx and val must be 4-byte aligned");
    if (d > 0 && (workspace == nullptr || !aligned(workspace, 16)))
        return fail(EFS_EINVAL, "topk_compress: workspace must be non-NULL and 16-byte aligned");
    if (d > 0 && workspace_bytes < efs::topk_workspace_size(d, k))
        return fail(EFS_ESPACE, "topk_compress: workspace has %zu bytes, needs %zu", workspace_bytes,
                    efs::topk_workspace_size(d, k));
    return check_launch(efs::launch_topk(g, e, d, lr, k, idx, val, workspace,
                                         static_cast<hipStream_t>(stream)),
                        "topk_compress");
}

size_t topk_segmented_workspace_bytes(int32_t nseg, int64_t k_total) {
    if (nseg < 1 || nseg > efs::kMaxSegments || k_total < 0 || k_total > kMaxLen) return 0;
    return efs::topk_segmented_workspace_size(nseg, k_total);
}

size_t topk_segmented_status_offset(void) { return efs::topk_segmented_status_offset(); }

size_t topk_segmented_bracket_offset(void) { return efs::topk_segmented_bracket_offset(); }

efs_status topk_segmented_compress(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                                   const int64_t *offsets, const int64_t *k, int64_t k_total,
                                   int32_t *idx, float *val, void *workspace,
                                   size_t workspace_bytes, void *stream) {
    const char *name = "topk_segmented_compress";
    if (d < 0 || d > kMaxLen) return fail(EFS_EINVAL, "%s: d=%lld outside [0, 2^31-1]", name, (long long)d);
    if (nseg < 1 || nseg > efs::kMaxSegments)
        return fail(EFS_EINVAL, "%s: nseg=%d outside [1, %d]", name, nseg, efs::kMaxSegments);
    if (k_total < 0 || k_total > d) return fail(EFS_EINVAL, "%s: k_total=%lld outside [0, d]", name, (long long)k_total);
    if (d > 0 && (g == nullptr || e == nullptr)) return fail(EFS_EINVAL, "%s: g or e is NULL", name);
    if (!aligned(g, 4) || !aligned(e, 4)) return fail(EFS_EINVAL, "%s: g and e must be 4-byte aligned", name);
    if (!std::isfinite(lr)) return fail(EFS_EINVAL, "%s: lr must be finite", name);
    if (offsets == nullptr || k == nullptr || !aligned(offsets, 8) || !aligned(k, 8))
        return fail(EFS_EINVAL, "%s: offsets and k must be non-NULL and 8-byte aligned", name);
    if (k_total > 0 && (idx == nullptr || val == nullptr)) return fail(EFS_EINVAL, "%s: idx or val is NULL", name);
    if (!aligned(idx, 4) || !aligned(val, 4)) return fail(EFS_EINVAL, "%s: idx and val must be 4-byte aligned", name);
    if (d == 0) return EFS_OK;
    if (workspace == nullptr || !aligned(workspace, 16))
        return fail(EFS_EINVAL, "%s: workspace must be non-NULL and 16-byte aligned", name);
    const size_t need = efs::topk_segmented_workspace_size(nseg, k_total);
    if (workspace_bytes < need)
        return fail(EFS_ESPACE, "%s: workspace has %zu bytes, needs %zu", name, workspace_bytes, need);
    return check_launch(efs::launch_topk_segmented(g, e, d, lr, nseg, offsets, k, k_total, idx, val,
                                                   workspace, static_cast<hipStream_t>(stream)),
                        name);
}

size_t sparse_apply_workspace_bytes(int32_t n_workers, int64_t d, int64_t total_cap) {
    if (n_workers < 1 || n_workers > efs::kMaxApplyWorkers || d < 0 || d > kMaxLen ||
        total_cap < 0 || total_cap > int64_t(UINT32_MAX))
        return 0;
    return efs::apply_workspace_size(n_workers, d, total_cap);
}

size_t sparse_accumulate_workspace_bytes(int32_t n_workers, int64_t d, int64_t total_cap) {
    return sparse_apply_workspace_bytes(n_workers, d, total_cap);
}

size_t sparse_bucket_workspace_bytes(int32_t n_workers, int64_t d) {
    if (n_workers < 1 || n_workers > efs::kMaxApplyWorkers || d < 0 || d > kMaxLen) return 0;
    return efs::apply_bucket_workspace_size(n_workers, d);
}

size_t sparse_status_offset(void) { return efs::apply_status_offset(); }

// Checks shared by sparse_accumulate, sparse_accumulate_static and
// sparse_apply: the payload arrays and the output (x).  Returns EFS_OK when
// they are valid, with the sum of the capacities in *total.
static efs_status check_payload_args(const char *name, const int32_t *const *idx,
                                     const float *const *val, const uint32_t *const *counts,
                                     const int64_t *caps, int32_t n_workers, int64_t d,
                                     const float *x, int64_t *total_out) {
    if (n_workers < 1 || n_workers > efs::kMaxApplyWorkers)
        return fail(EFS_EINVAL, "%s: n_workers=%d outside [1, %d]", name, n_workers,
                    efs::kMaxApplyWorkers);
    if (d < 0 || d > kMaxLen) return fail(EFS_EINVAL, "%s: d=%lld outside [0, 2^31-1]", name, (long long)d);
    if (idx == nullptr || val == nullptr || caps == nullptr)
        return fail(EFS_EINVAL, "%s: idx, val and caps must be host arrays", name);
    if (d > 0 && (x == nullptr || !aligned(x, 16)))
        return fail(EFS_EINVAL, "%s: the output must be non-NULL and 16-byte aligned", name);
    int64_t total = 0;
    for (int32_t w = 0; w < n_workers; ++w) {
        if (caps[w] < 0 || caps[w] > kMaxLen)
            return fail(EFS_EINVAL, "%s: caps[%d]=%lld outside [0, 2^31-1]", name, w, (long long)caps[w]);
        if (caps[w] > 0 && (idx[w] == nullptr || val[w] == nullptr))
            return fail(EFS_EINVAL, "%s: payload %d has a NULL pointer", name, w);
        if (!aligned(idx[w], 4) || !aligned(val[w], 4))
            return fail(EFS_EINVAL, "%s: payload %d is not 4-byte aligned", name, w);
        if (counts != nullptr && counts[w] != nullptr && !aligned(counts[w], 4))
            return fail(EFS_EINVAL, "%s: count %d is not 4-byte aligned", name, w);
        total += caps[w];
    }
    if (total > int64_t(UINT32_MAX))
        return fail(EFS_EINVAL, "%s: total capacity %lld exceeds 2^32-1 pairs", name, (long long)total);
    *total_out = total;
    return EFS_OK;
}

// Bytes the call needs of a workspace of `have` bytes: 0 when it holds the
// bucketed layout or the packed one, else the packed layout's size.
static size_t workspace_shortfall(int32_t n_workers, int64_t d, int64_t total, size_t have) {
    if (have >= efs::apply_bucket_workspace_size(n_workers, d)) return 0;
    const size_t need = efs::apply_workspace_size(n_workers, d, total);
    return have >= need ? 0 : need;
}

// The payload checks plus the workspace (pointer, alignment, size).
static efs_status check_payloads(const char *name, const int32_t *const *idx,
                                 const float *const *val, const uint32_t *const *counts,
                                 const int64_t *caps, int32_t n_workers, int64_t d, const float *x,
                                 const void *workspace, size_t workspace_bytes) {
    int64_t total = 0;
    const efs_status s = check_payload_args(name, idx, val, counts, caps, n_workers, d, x, &total);
    if (s != EFS_OK || d == 0) return s;
    if (workspace == nullptr || !aligned(workspace, 16))
        return fail(EFS_EINVAL, "%s: workspace must be non-NULL and 16-byte aligned", name);
    // the bucketed layout whenever the workspace holds it, else the packed one
    const size_t need = workspace_shortfall(n_workers, d, total, workspace_bytes);
    if (need != 0)
        return fail(EFS_ESPACE, "%s: workspace has %zu bytes, needs %zu", name, workspace_bytes, need);
    return EFS_OK;
}

efs_status sparse_accumulate(const int32_t *const *idx, const float *const *val,
                             const uint32_t *const *counts, const int64_t *caps,
                             int32_t n_workers, int64_t d, float *out, void *workspace,
                             size_t workspace_bytes, void *stream) {
    const efs_status s = check_payloads("sparse_accumulate", idx, val, counts, caps, n_workers, d,
                                        out, workspace, workspace_bytes);
    if (s != EFS_OK || d == 0) return s;
    return check_launch(efs::launch_apply(idx, val, counts, caps, n_workers, d, EFS_APPLY_AVERAGE,
                                          out, nullptr, 0.0f, 0.0f, workspace, workspace_bytes,
                                          static_cast<hipStream_t>(stream)),
                        "sparse_accumulate");
}

efs_status sparse_accumulate_static(const int32_t *const *idx, const float *const *val,
                                    const uint32_t *const *counts, const int64_t *caps,
                                    int32_t n_workers, int64_t d, float *out, void *stream) {
    const char *name = "sparse_accumulate_static";
    int64_t total = 0;
    const efs_status s = check_payload_args(name, idx, val, counts, caps, n_workers, d, out, &total);
    if (s != EFS_OK || d == 0) return s;
    const size_t need = workspace_shortfall(n_workers, d, total, efs::kStaticScratchBytes);
    if (need != 0)
        return fail(EFS_ESPACE, "%s: the payloads need %zu bytes of scratch; the library holds %zu "
                    "per device (use sparse_accumulate with a workspace)", name, need,
                    efs::kStaticScratchBytes);
    void *scratch = nullptr;
    const hipError_t err = efs::static_scratch(&scratch);
    if (err != hipSuccess)
        return fail(EFS_EHIP, "%s: no scratch on the current device: %s", name, hipGetErrorString(err));
    return check_launch(efs::launch_apply(idx, val, counts, caps, n_workers, d, EFS_APPLY_AVERAGE,
                                          out, nullptr, 0.0f, 0.0f, scratch,
                                          efs::kStaticScratchBytes,
                                          static_cast<hipStream_t>(stream)),
                        name);
}

efs_status sparse_apply(const int32_t *const *idx, const float *const *val,
                        const uint32_t *const *counts, const int64_t *caps, int32_t n_workers,
                        int64_t d, int mode, float *x, float *m, float beta, float gamma,
                        void *workspace, size_t workspace_bytes, void *stream) {
    if (mode < EFS_APPLY_AVERAGE || mode > EFS_APPLY_MOMENTUM)
        return fail(EFS_EINVAL, "sparse_apply: mode %d is not one of EFS_APPLY_*", mode);
    if (mode == EFS_APPLY_MOMENTUM && d > 0) {
        if (m == nullptr || !aligned(m, 16))
            return fail(EFS_EINVAL, "sparse_apply: m must be non-NULL and 16-byte aligned");
        if (m == x) return fail(EFS_EINVAL, "sparse_apply: m and x must not alias");
    }
    if (mode == EFS_APPLY_MOMENTUM && (!std::isfinite(beta) || !std::isfinite(gamma)))
        return fail(EFS_EINVAL, "sparse_apply: beta and gamma must be finite");
    const efs_status s = check_payloads("sparse_apply", idx, val, counts, caps, n_workers, d, x,
                                        workspace, workspace_bytes);
    if (s != EFS_OK || d == 0) return s;
    return check_launch(efs::launch_apply(idx, val, counts, caps, n_workers, d, mode, x, m, beta,
                                          gamma, workspace, workspace_bytes,
                                          static_cast<hipStream_t>(stream)),
                        "sparse_apply");
}

// The probes address at most INT32_MAX tiles (one workgroup each in the
// one-tile-per-workgroup shape).
constexpr int64_t kProbeMaxElements = int64_t(INT32_MAX) * efs::kTile;

efs_status efs_copy_probe(const float *src, float *dst, int64_t n, void *stream) {
    if (n < 0 || n > kProbeMaxElements)
        return fail(EFS_EINVAL, "efs_copy_probe: n = %lld outside [0, %lld]", (long long)n,
                    (long long)kProbeMaxElements);
    if (n > 0 && (src == nullptr || dst == nullptr || !aligned(src, 16) || !aligned(dst, 16)))
        return fail(EFS_EINVAL, "efs_copy_probe: src and dst must be non-NULL and 16-byte aligned");
    return check_launch(efs::launch_copy(src, dst, n, false, static_cast<hipStream_t>(stream)),
                        "efs_copy_probe");
}

efs_status efs_stream_probe(const float *x, float *y, int64_t n, int mode, void *stream) {
    if (n < 0 || n > kProbeMaxElements)
        return fail(EFS_EINVAL, "efs_stream_probe: n = %lld outside [0, %lld]", (long long)n,
                    (long long)kProbeMaxElements);
    if (mode < 0 || mode > 7) return fail(EFS_EINVAL, "efs_stream_probe: mode %d outside 0..7", mode);
    const bool per_tile = (mode & 4) != 0;
    mode &= 3;
    if (n > 0 && (x == nullptr || y == nullptr || !aligned(x, 16) || !aligned(y, 16)))
        return fail(EFS_EINVAL, "efs_stream_probe: x and y must be non-NULL and 16-byte aligned");
    if (mode == 0)
        return check_launch(efs::launch_copy(x, y, n, per_tile, static_cast<hipStream_t>(stream)),
                            "efs_stream_probe");
    return check_launch(
        efs::launch_stream_probe(x, y, n, mode, per_tile, static_cast<hipStream_t>(stream)),
        "efs_stream_probe");
}

}  // extern "C"
