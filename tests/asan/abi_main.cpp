// Host-side argument validation of the C ABI, built with AddressSanitizer
// (host code only) and run without a GPU: every call below must be
// rejected, or, when valid, fail at most at the launch (no device), without
// any invalid memory access in the checks themselves.  Prints "ok" and
// exits 0 when every status is the expected one.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../include/efsparse.h"

static int failures = 0;

static void expect(const char *what, efs_status got, efs_status want) {
    if (got != want) {
        std::printf("FAIL %s: got %d want %d (%s)\n", what, int(got), int(want),
                    efs_last_error_message());
        ++failures;
    }
}

int main() {
    // fake device addresses: never dereferenced on the host
    float *f = reinterpret_cast<float *>(uintptr_t(0x100000));
    int32_t *i = reinterpret_cast<int32_t *>(uintptr_t(0x200000));
    uint32_t *c = reinterpret_cast<uint32_t *>(uintptr_t(0x300000));
    void *ws = reinterpret_cast<void *>(uintptr_t(0x400000));
    const efs_status inval = EFS_EINVAL, space = EFS_ESPACE, ok = EFS_OK;

    expect("ht d<0", ht_compress(f, f, -1, 0.1f, 1.0f, i, f, 10, c, nullptr), inval);
    expect("ht d>int32", ht_compress(f, f, int64_t(1) << 31, 0.1f, 1.0f, i, f, 10, c, nullptr), inval);
    expect("ht lambda nan", ht_compress(f, f, 10, 0.1f, NAN, i, f, 10, c, nullptr), inval);
    expect("ht lambda<0", ht_compress(f, f, 10, 0.1f, -1.0f, i, f, 10, c, nullptr), inval);
    expect("ht lr inf", ht_compress(f, f, 10, INFINITY, 1.0f, i, f, 10, c, nullptr), inval);
    expect("ht g null", ht_compress(nullptr, f, 10, 0.1f, 1.0f, i, f, 10, c, nullptr), inval);
    expect("ht misaligned", ht_compress(f, reinterpret_cast<float *>(uintptr_t(0x100002)), 10,
                                        0.1f, 1.0f, i, f, 10, c, nullptr), inval);
    expect("ht cap<0", ht_compress(f, f, 10, 0.1f, 1.0f, i, f, -1, c, nullptr), inval);
    expect("ht counter null", ht_compress(f, f, 10, 0.1f, 1.0f, i, f, 10, nullptr, nullptr), inval);
    expect("ht telemetry null", ht_compress_telemetry(f, f, 10, 0.1f, 1.0f, i, f, 10, c,
                                                      nullptr, nullptr), inval);

    const size_t tws = topk_workspace_bytes(1000, 10);
    if (tws == 0 || topk_workspace_bytes(10, 11) != 0 || topk_workspace_bytes(-1, 0) != 0) {
        std::printf("FAIL topk workspace sizes\n");
        ++failures;
    }
    expect("topk k>d", topk_compress(f, f, 10, 0.1f, 11, i, f, ws, tws, nullptr), inval);
    expect("topk ws small", topk_compress(f, f, 1000, 0.1f, 10, i, f, ws, tws - 1, nullptr), space);
    expect("topk ws null", topk_compress(f, f, 1000, 0.1f, 10, i, f, nullptr, tws, nullptr), inval);

    const int n = 3;
    std::vector<const int32_t *> idx(n, i);
    std::vector<const float *> val(n, f);
    std::vector<int64_t> caps(n, 5);
    const size_t aws = sparse_accumulate_workspace_bytes(n, 100, 15);
    expect("average n=0", sparse_accumulate(idx.data(), val.data(), nullptr, caps.data(), 0, 100,
                                            f, ws, aws, nullptr), inval);
    expect("average n>max", sparse_accumulate(idx.data(), val.data(), nullptr, caps.data(),
                                              EFS_MAX_WORKERS + 1, 100, f, ws, aws, nullptr), inval);
    caps[2] = -1;
    expect("average cap<0", sparse_accumulate(idx.data(), val.data(), nullptr, caps.data(), n, 100,
                                              f, ws, aws, nullptr), inval);
    caps[2] = 5;
    idx[1] = nullptr;
    expect("average null payload", sparse_accumulate(idx.data(), val.data(), nullptr, caps.data(),
                                                     n, 100, f, ws, aws, nullptr), inval);
    idx[1] = i;
    expect("average ws small", sparse_accumulate(idx.data(), val.data(), nullptr, caps.data(), n,
                                                 100, f, ws, aws - 1, nullptr), space);
    expect("average d=0", sparse_accumulate(idx.data(), val.data(), nullptr, caps.data(), n, 0,
                                            nullptr, nullptr, 0, nullptr), ok);
    expect("apply mode", sparse_apply(idx.data(), val.data(), nullptr, caps.data(), n, 100, 7, f,
                                      nullptr, 0.f, 0.f, ws, aws, nullptr), inval);
    expect("apply m aliases x", sparse_apply(idx.data(), val.data(), nullptr, caps.data(), n, 100,
                                             EFS_APPLY_MOMENTUM, f, f, 0.9f, 0.1f, ws, aws, nullptr),
           inval);

    std::vector<int64_t> off = {0, 5, 10};
    expect("layer-wise nseg=0", topk_segmented_compress(f, f, 10, 0.1f, 0, off.data(), off.data(),
                                                        1, i, f, ws, 1 << 20, nullptr), inval);
    expect("layer-wise k_total>d", topk_segmented_compress(f, f, 10, 0.1f, 2, off.data(),
                                                           off.data(), 11, i, f, ws, 1 << 20,
                                                           nullptr), inval);
    expect("probe mode", efs_stream_probe(f, f, 10, 9, nullptr), inval);
    // the last rejected call is sticky (EFS_EHIP instead where the runtime
    // holds an error of its own, e.g. no device)
    const efs_status sticky = efs_last_error();
    if (sticky != EFS_EINVAL && sticky != EFS_EHIP) {
        std::printf("FAIL sticky status %d\n", int(sticky));
        ++failures;
    }
    std::printf(failures ? "%d failures\n" : "ok\n", failures);
    return failures ? 1 : 0;
}
