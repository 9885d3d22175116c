/*
 * efsparse — error-feedback gradient sparsification on MI355X (gfx950).
 *
 * C ABI of libefsparse.so.  Implements the per-worker compression step of
 * "Rethinking gradient sparsification as total error minimization"
 * (arXiv 2108.00951), Algorithm 1 (distributed EF SGD):
 *
 *     p      = e + lr * g                 EF accumulate
 *     Delta  = C(p)                       compress (hard threshold or Top-k)
 *     e'     = p - Delta                  error update
 *     avg    = (1/n) sum_i Delta_i        exchange and average
 *
 * Conventions shared by every entry point
 *   - Every array argument is a DEVICE pointer owned by the caller; the
 *     library never allocates, frees or synchronises.  Work is enqueued on
 *     `stream` (a hipStream_t; NULL means the legacy default stream) and is
 *     complete only when that stream is.
 *   - Arguments are validated on the host before anything is enqueued.  On a
 *     non-OK status nothing was enqueued, except EFS_EHIP, which reports a
 *     launch failure (kernels launched before it stay enqueued).
 *     efs_last_error_message() then describes the failure (per thread).
 *   - Arithmetic is IEEE binary32 with round to nearest even; the accumulate
 *     is a multiply followed by a separately rounded add (never fused);
 *     subnormals are kept.
 *   - Indices are 0-based int32; d must not exceed INT32_MAX.
 *   - Payload pair order is unspecified (consumers must not rely on it).
 *     Payload values are the kept entries of p, unscaled.
 */
#ifndef EFSPARSE_H
#define EFSPARSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum efs_status {
    EFS_OK = 0,
    EFS_EINVAL = 1,   /* an argument failed validation; nothing enqueued      */
    EFS_ESPACE = 2,   /* workspace smaller than the query said; nothing enqueued */
    EFS_EHIP = 3      /* the HIP runtime rejected a launch                      */
} efs_status;

/* A counter object: EFS_COUNTER_WORDS uint32 words (16 bytes) of device
 * memory, 8-byte aligned, zero-filled once by the caller before first use.
 * Word 0 receives the payload count k_t of the last completed call; the
 * other words are the library's and are back at zero whenever no call that
 * uses the object is in flight.  One object must not be used by two calls
 * that may run concurrently. */
#define EFS_COUNTER_WORDS 4

/* Hard-threshold sparsifier with error feedback (Algorithm 1 with the
 * hard-threshold compressor C_lambda of section 4.2:
 * S_lambda(p) = { i : |p_i| >= lambda }).
 *
 *   g        [d] fp32, read only: the stochastic gradient g_t.
 *   e        [d] fp32, in place: e_t on entry, e_{t+1} on completion
 *            (+0.0f at kept coordinates, p_i elsewhere).  Must not overlap g
 *            or the payload.
 *   d        vector length, 0 <= d <= INT32_MAX.
 *   lr       step size gamma (finite).
 *   lambda   threshold in the units of p (lambda >= 0, not NaN; +inf keeps
 *            nothing).  Algorithm 1 writes the compressor as gamma*C(p/gamma);
 *            for the threshold of C in those units pass gamma*lambda here.
 *   idx,val  [cap] payload (int32 index, fp32 value p_i), unordered; only the
 *            first min(k_t, cap) slots are written.  May be NULL when cap == 0.
 *   cap      payload capacity, >= 0.
 *   counter  counter object (see above); word 0 receives k_t, the TRUE
 *            count even when it exceeds cap (then the payload is truncated
 *            and must be treated as invalid; e' is complete regardless).
 * Pointers g and e must be 4-byte aligned (16-byte alignment takes the
 * vector path).  NaN entries of p are never kept. */
efs_status ht_compress(const float *g, float *e, int64_t d, float lr, float lambda,
                       int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                       void *stream);

/* A telemetry object: EFS_TELEMETRY_BYTES of device memory, 8-byte aligned,
 * zero-filled by the caller before the first call; every call adds to it:
 *   double   err2_part[32] partial sums whose total is the sum over calls of
 *                          ||e_{t+1}||^2, the total error of Remark 4
 *                          (section 3) when the calls are the iterations
 *                          t = 0..T-1 (sum the 32 values to read it);
 *   double   sent_total    sum over calls of k_t (average density =
 *                          sent_total / (calls * d), the measure of data
 *                          volume used in section 6);
 *   uint32_t max_abs_bits  running max of |e_{t+1}| as the bit pattern of a
 *                          non-negative float (the hard threshold keeps it
 *                          below lambda: the absolute-compressor bound of
 *                          section 5);
 *   uint32_t calls         number of calls accumulated;
 *   16 bytes reserved.
 * The norm is summed in binary64, each workgroup adding its share into one
 * of the 32 parts with an atomic (one word for all of them serialises), so
 * its last bits can vary with the order of the additions. */
#define EFS_TELEMETRY_BYTES 288

/* ht_compress, and in the same pass the telemetry above added to
 * `telemetry` (device pointer, see EFS_TELEMETRY_BYTES). */
efs_status ht_compress_telemetry(const float *g, float *e, int64_t d, float lr, float lambda,
                                 int32_t *idx, float *val, int64_t cap, uint32_t *counter,
                                 void *telemetry, void *stream);

/* Bytes of device workspace topk_compress needs for (d, k). */
size_t topk_workspace_bytes(int64_t d, int64_t k);

/* Top-k sparsifier with error feedback (Algorithm 1 with Top-k, the
 * per-iteration optimum of Lemma 2): keeps the k coordinates of largest |p|.
 * Magnitudes are ranked by the bit pattern of |p| (so -0 and +0 tie, NaN
 * ranks above +inf); equal magnitudes go to the lower index.
 *
 *   g, e, d, lr   as for ht_compress.
 *   k             0 <= k <= d.
 *   idx, val      [k] payload of exactly k pairs (unordered).
 *   workspace     device memory of at least topk_workspace_bytes(d, k)
 *                 bytes, 16-byte aligned; contents need no initialisation.
 *                 The library keeps the last two thresholds in it: a
 *                 following call on the same workspace whose k-th magnitude
 *                 lies within about 6 to 12 % of their linear extrapolation
 *                 (the error-feedback case) selects from a small candidate
 *                 set instead of three more passes over p.
 *                 Results never depend on what the workspace held.  Not
 *                 shareable between concurrent calls.
 */
efs_status topk_compress(const float *g, float *e, int64_t d, float lr, int64_t k,
                         int32_t *idx, float *val, void *workspace,
                         size_t workspace_bytes, void *stream);

/* Byte offset, within a Top-k workspace, of a uint32 that is 1 after a call
 * that selected from the candidate set around the previous threshold and 0
 * after one that ran the full radix select (a diagnostic; read it after the
 * call has completed). */
size_t topk_path_flag_offset(void);

/* Layer-wise Top-k EF step (Appendix C.5: the sparsifier applied to each
 * layer's tensor on its own; Algorithm 1 for the error):
 *     p = e + lr*g ;  in every segment s = [offsets[s], offsets[s+1]) keep the
 *     min(k[s], size_s) entries of largest |p| (equal magnitudes: lower index
 *     first, as topk_compress ranks them) ;  e' = p with +0 at every kept entry.
 *
 *   g, e        as for topk_compress (e in/out, in place).
 *   nseg        number of segments, 1 <= nseg <= EFS_SEG_MAX.
 *   offsets     DEVICE int64[nseg + 1], 8-byte aligned: offsets[0] = 0,
 *               non-decreasing, offsets[nseg] = d (empty segments allowed).
 *   k           DEVICE int64[nseg], 8-byte aligned: k[s] >= 0; values above
 *               a segment's size keep the whole segment.
 *   k_total     capacity of idx/val; must be >= sum of min(k[s], size_s).
 *   idx, val    payload: segment s's pairs occupy
 *               [kout_s, kout_s + min(k[s], size_s)), kout the exclusive
 *               prefix of those counts; order within a segment unspecified.
 *   workspace   >= topk_segmented_workspace_bytes(nseg, k_total) bytes,
 *               16-byte aligned: per-segment tables and histograms (36 KiB per
 *               segment), a candidate region of 16*k_total + 4096*nseg
 *               (key, index) pairs, a work list of one 8-byte entry per
 *               512 of those pairs or payload slots, and 32 KiB of flags
 *               over groups of tiles.  Results never depend on its contents.
 *               Not shareable between concurrent calls.
 * Host-visible arguments are checked before anything is launched (EFS_EINVAL,
 * EFS_ESPACE).  offsets and k live on the device and are checked there: a
 * layout that breaks the rules above, or a k_total below the sum, makes the
 * call change nothing (no payload written, e untouched) and leaves the uint32
 * at topk_segmented_status_offset() in the workspace at 1 (0 after an
 * accepted call).  d == 0 is a no-op. */
#define EFS_SEG_MAX 65536
size_t topk_segmented_workspace_bytes(int32_t nseg, int64_t k_total);
size_t topk_segmented_status_offset(void);

/* Byte offset, within a layer-wise Top-k workspace, of a uint32 counting the
 * segments of the last completed call that selected among the keys in a
 * bracket around the threshold predicted from that segment's earlier calls
 * (instead of the full radix select; a diagnostic, read after the call has
 * completed). */
size_t topk_segmented_bracket_offset(void);
efs_status topk_segmented_compress(const float *g, float *e, int64_t d, float lr, int32_t nseg,
                                   const int64_t *offsets, const int64_t *k, int64_t k_total,
                                   int32_t *idx, float *val, void *workspace,
                                   size_t workspace_bytes, void *stream);

/* Exchange-and-average of n workers' payloads on one device (Algorithm 1:
 * the average (1/n) sum_i Delta_i of the compressed updates; App. C.6.2,
 * Algorithm 2: DECOMPRESS then AGGREGATE):
 *     out = (sum over w = 0..n-1, in that order, of decompress(payload_w)) / n
 * with fp32 adds in worker order and one IEEE division by (float)n at every
 * coordinate (untouched coordinates are +0).
 *
 *   idx, val   HOST arrays of n_workers device pointers; payload w has
 *              indices idx[w][0..c_w) (distinct within one payload) and
 *              values val[w][0..c_w).
 *   counts     HOST array of n_workers device pointers to the uint32 count of
 *              each payload (word 0 of ht_compress's counter object, which
 *              stays on the device), or NULL entries / a NULL array meaning
 *              c_w = caps[w].
 *   caps       HOST array of n_workers capacities; c_w = min(*counts[w],
 *              caps[w]).  A count above its capacity (a truncated
 *              hard-threshold payload) is averaged over its caps[w] pairs and
 *              reported in the status word (EFS_SPARSE_TRUNCATED).
 *   n_workers  1 <= n_workers <= EFS_MAX_WORKERS; sum of caps <= 2^32 - 1.
 *   d          length of out; d == 0 is a no-op.
 *   out        [d] fp32, 16-byte aligned, overwritten.
 *   workspace  device memory, 16-byte aligned, in one of two layouts chosen
 *              by workspace_bytes:
 *                bucketed, when workspace_bytes >=
 *                sparse_bucket_workspace_bytes(n_workers, d) (about 8 n d
 *                bytes): a 256-byte control block, an 8-byte counter per
 *                (range of 4096 coordinates, worker) and a bucket of 4096
 *                8-byte slots per counter.  Two launches.
 *                packed, otherwise; needs at least
 *                sparse_accumulate_workspace_bytes(n_workers, d, sum of caps)
 *                bytes: the control block, an 8-byte counter and a 4-byte
 *                segment start per (range, worker), and 8 bytes per payload
 *                slot for the pairs grouped by range.  Four launches.
 *              Both give the same bits.  Contents need no initialisation:
 *              each counter carries the 40-bit epoch of the call that wrote
 *              it (the control block's epoch, advanced by every call), so a
 *              counter of an earlier call reads as zero, as does arbitrary
 *              content except when its epoch bits equal the current epoch
 *              (probability 2^-40 per counter for random bytes).  Calls on
 *              one workspace must be ordered (one stream, or synchronised
 *              streams); concurrent calls on one workspace race.
 * Payload entries with an index outside [0, d) are skipped and reported in
 * the status word (EFS_SPARSE_BAD_INDEX).  The status word is the uint32 at
 * sparse_status_offset() in the workspace: the EFS_SPARSE_* bits of the last
 * completed call (0: every payload was whole and in range).  The counts are
 * read on the device, so these are reported there and not as an efs_status. */
#define EFS_MAX_WORKERS 64
#define EFS_SPARSE_TRUNCATED 1u
#define EFS_SPARSE_BAD_INDEX 2u
/* Bytes of the packed and of the bucketed workspace layout; 0 if the
 * arguments are out of range. */
size_t sparse_accumulate_workspace_bytes(int32_t n_workers, int64_t d, int64_t total_cap);
size_t sparse_bucket_workspace_bytes(int32_t n_workers, int64_t d);
size_t sparse_status_offset(void);
efs_status sparse_accumulate(const int32_t *const *idx, const float *const *val,
                             const uint32_t *const *counts, const int64_t *caps,
                             int32_t n_workers, int64_t d, float *out, void *workspace,
                             size_t workspace_bytes, void *stream);

/* sparse_accumulate for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same operation with the same bits, the pairs grouped in a
 * scratch array of EFS_STATIC_SCRATCH_BYTES that the library holds on each
 * device it runs on (from the library's first use of that device until the
 * process ends) instead of in a caller's workspace.  The call allocates
 * nothing.
 *
 *   idx, val, counts, caps, n_workers, d, out, stream
 *              as for sparse_accumulate.
 * Returns EFS_ESPACE, with nothing launched, when the payloads need more
 * than EFS_STATIC_SCRATCH_BYTES: the bucketed layout is used when
 * sparse_bucket_workspace_bytes(n_workers, d) fits in the scratch, else the
 * packed one, which needs sparse_accumulate_workspace_bytes(n_workers, d,
 * sum of caps).  EFS_EINVAL on any other invalid argument, EFS_EHIP if the
 * scratch cannot be found on the current device.  Every call on one device
 * shares that device's scratch; nothing in it needs clearing between calls
 * (its counters carry epoch tags), but calls that overlap on one device
 * (from concurrent streams or host threads) race and must be ordered by the
 * caller.  The status word of these calls stays in the scratch and is not
 * reported. */
#define EFS_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
efs_status sparse_accumulate_static(const int32_t *const *idx, const float *const *val,
                                    const uint32_t *const *counts, const int64_t *caps,
                                    int32_t n_workers, int64_t d, float *out, void *stream);

/* Exchange-and-average fused with the model update that follows it.
 *
 *   avg = (sum over w = 0..n-1, in that order, of decompress(payload_w)) / n
 * exactly as sparse_accumulate computes it (fp32 adds in worker order, one
 * IEEE division by (float)n), then, by mode:
 *   EFS_APPLY_AVERAGE   x = avg at every coordinate (x is the output; the
 *                       same call as sparse_accumulate).
 *   EFS_APPLY_SGD       x = x - avg (Algorithm 1, model update).  Only
 *                       coordinates that some payload touches are written;
 *                       the others keep x, which equals x - (+0) for every
 *                       value except a signalling NaN.
 *   EFS_APPLY_MOMENTUM  m = beta*m + avg, then x = x - gamma*(avg + m) with the
 *                       new m, at every coordinate (Appendix C.6.2,
 *                       Algorithm 2: EF SGD with momentum and gradient
 *                       compression; the paper writes the momentum factor
 *                       as lambda and the learning rate as gamma).
 * Every operation is one separately rounded fp32 operation, in the order
 * written (no fused multiply-add).
 *
 *   idx, val, counts, caps, n_workers, d, workspace, status word
 *              as for sparse_accumulate (the same workspace layouts, chosen
 *              the same way).
 *   x          [d] fp32, 16-byte aligned, read and written in place (mode
 *              EFS_APPLY_AVERAGE only writes it).  Must not overlap a payload.
 *   m          [d] fp32 momentum, 16-byte aligned, read and written in place;
 *              used by EFS_APPLY_MOMENTUM only (may be NULL otherwise).
 *   beta, gamma  momentum factor and learning rate (finite); used by
 *              EFS_APPLY_MOMENTUM only.
 * Returns EFS_ESPACE if the workspace is too small, EFS_EINVAL on any other
 * invalid argument; nothing is launched then.  d == 0 is a no-op. */
enum { EFS_APPLY_AVERAGE = 0, EFS_APPLY_SGD = 1, EFS_APPLY_MOMENTUM = 2 };

/* Workspace bytes of sparse_apply's packed layout (the same as
 * sparse_accumulate_workspace_bytes); 0 if the arguments are out of range. */
size_t sparse_apply_workspace_bytes(int32_t n_workers, int64_t d, int64_t total_cap);

efs_status sparse_apply(const int32_t *const *idx, const float *const *val,
                        const uint32_t *const *counts, const int64_t *caps, int32_t n_workers,
                        int64_t d, int mode, float *x, float *m, float beta, float gamma,
                        void *workspace, size_t workspace_bytes, void *stream);

/* Streaming copy dst[0..n) = src[0..n) with the same 16-byte access pattern
 * and grid as the hard-threshold kernel: the reference transfer for
 * measurements, not part of the method.  src and dst 16-byte aligned,
 * 0 <= n <= INT32_MAX * 4096. */
efs_status efs_copy_probe(const float *src, float *dst, int64_t n, void *stream);

/* Streaming bandwidth probes over n floats with the same tile shape as the
 * compression kernels (measurement aids, not part of the method):
 *   mode 0  copy       y = x                (4n bytes read, 4n written)
 *   mode 1  read       sum of x, discarded  (4n read; y[0..255] reserved)
 *   mode 2  write      y = constant         (4n written)
 *   mode 3  2R1W       y = y + 0.5 x        (8n read, 4n written; the
 *                                            access pattern of ht_compress)
 * plus 4: the same traffic with one workgroup per 4096-element tile instead
 * of the hard threshold's persistent grid.  Modes 1-3 (5-7) cover whole
 * 4096-element tiles only.  x and y 16-byte aligned, 0 <= n <=
 * INT32_MAX * 4096; for mode 1 (5), y must hold at least 256 floats.  Other
 * modes: EFS_EINVAL. */
efs_status efs_stream_probe(const float *x, float *y, int64_t n, int mode, void *stream);

/* Static text for a status code. */
const char *efs_status_string(efs_status status);

/* Detail of the last non-OK status returned on the calling thread. */
const char *efs_last_error_message(void);

/* Sticky status for callers that check once after a sequence of calls:
 * EFS_EHIP when the HIP runtime holds an error left by an earlier
 * asynchronous launch on this thread (hipPeekAtLastError, not cleared);
 * otherwise the last non-OK status any call returned on this thread since
 * the previous efs_last_error (which clears it), or EFS_OK.  Conditions
 * that only the device sees are reported on the device: a hard-threshold
 * count above the capacity in the counter object (compare it with cap), a
 * truncated payload or an index out of range in the average's status word. */
efs_status efs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EFSPARSE_H */
