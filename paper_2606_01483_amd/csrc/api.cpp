// C ABI of libmurmur (include/murmur.h): argument validation, workspace
// planning, error text, and dispatch to the gfx950 kernels.  Every check runs
// before the first HIP call, so rejected calls leave the device untouched.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "internal.h"
#include "murmur.h"
#include "policy.h"

#define MURMUR_EXPORT extern "C" __attribute__((visibility("default")))

static_assert(sizeof(murmur_seg) == 4 * sizeof(int32_t), "the kernels read murmur_seg as four int32");
static_assert(sizeof(murmur_policy) == 5 * sizeof(int32_t), "the kernels read murmur_policy as five int32");

namespace murmur {
namespace {

thread_local char g_last_error[512];

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_last_error[0] = '\0';
    return MURMUR_OK;
}

bool aligned(const void *p, size_t n) { return ((uintptr_t)p % n) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

size_t ticket_region(size_t ws_bytes) { return round_up(4 * kTicketStride * ((ws_bytes + 1023) / 1024), 256); }

namespace {

// ceil(2^32 / d) - 1: the kernel's x / d is the high word of (x + 1) times it,
// exact for x < 2^16 and 1 <= d < 2^16.  0 for d = 0 (an unused divisor).
uint32_t magic16(uint32_t d) { return d == 0 ? 0u : (uint32_t)((((uint64_t)1 << 32) + d - 1) / d - 1); }

// Estimated launch time (us) of a one-round split with at most len positions per
// workgroup and at most n splits per group (the model behind the automatic choice,
// with constants measured on MI355X): each compute unit streams its share at
// kCuBytesPerUs, in whole passes of kWaveTile rows (a wavefront issues a pass's
// loads whether it holds 2 rows or 32), and more than one split adds the merge
// chain, the merging workgroup's loads of n partials and a load round trip for
// every further two batches of partials.
double wide_cost(int64_t len, int64_t n, int64_t G) {
    const double part_bytes = (double)G * (kHeadDim + 2) * 4.0;
    const double trips = (double)((n - 1) / (2 * kMergeBatch)) * kMergeRoundTripUs;
    const int64_t rows = (len + kWaveTile - 1) / kWaveTile * kWaveTile;
    return (double)rows * 4.0 * kHeadDim / kCuBytesPerUs +
           (n > 1 ? kMergeChainUs + n * part_bytes / kCuBytesPerUs + trips : 0.0);
}

// The LDS-staged kernel's automatic split length: as many splits as keep one
// dispatch round (fewer when there are more groups than that, at most
// kMaxAutoSplits), counted in whole workgroup passes, then each split made as
// short as that count allows in whole wavefront passes: a split's time is
// bound by its compute unit's read rate, so rows past the longest sequence's
// share only cost (12 x 300 s dense: 768 -> 704 positions, five splits either way).
int64_t lds_auto_split(int64_t max_keep, int64_t groups) {
    const int64_t units = (max_keep + kSplitUnit - 1) / kSplitUnit;
    int64_t want = std::min<int64_t>(std::min<int64_t>(kRoundWorkgroups / groups, kMaxAutoSplits), units);
    if (want < 1) want = 1;
    const int64_t per = std::max<int64_t>((units + want - 1) / want, 2);
    const int64_t n = (max_keep + per * kSplitUnit - 1) / (per * kSplitUnit);
    const int64_t len = ((max_keep + n - 1) / n + kWaveTile - 1) / kWaveTile * kWaveTile;
    return std::max<int64_t>(len, 2 * kSplitUnit);
}

}  // namespace

WorkspacePlan plan_workspace(int32_t n_layers, int32_t B, int32_t Hq, int32_t Hkv, int32_t max_keep,
                             int32_t split_len) {
    WorkspacePlan p{};
    const int64_t groups = (int64_t)n_layers * B * Hkv;
    const int64_t G = Hkv > 0 ? Hq / Hkv : 0;
    p.groups = groups;
    // The wide schedule (splits of at most kWideSplit positions, a wavefront per
    // pass) needs its work indices below 2^16.
    const bool wide_ok = groups < 65536 && Hkv < 65536 && B < 65536;
    int64_t n_wide = 0, len_wide = 0;
    if (split_len == 0 && wide_ok && groups <= kRoundWorkgroups) {
        // One dispatch round: the number of splits per group with the lowest
        // estimate (fewer workgroups on a tie).  Giving some groups one split
        // more than the others never lowers it: the longest split stays and
        // those groups merge one partial more.
        double best = 0.0;
        for (int64_t n = 1; n * groups <= kRoundWorkgroups; ++n) {
            const int64_t len = ((int64_t)max_keep + n - 1) / n;
            if (len > kWideSplit) continue;
            const double t = wide_cost(len, n, G);
            if (n_wide == 0 || t < best - 1e-9) {
                best = t;
                n_wide = n;
                len_wide = len;
            }
        }
    } else if (split_len > 0 && split_len <= kWideSplit && wide_ok) {
        n_wide = ((int64_t)max_keep + split_len - 1) / split_len;
        len_wide = split_len;
    }
    if (split_len == 0 && n_wide > 0) {
        // The LDS-staged kernel's automatic split (below) when the model expects it to be faster.
        const int64_t len_lds = lds_auto_split(max_keep, groups);
        const int64_t n_lds = ((int64_t)max_keep + len_lds - 1) / len_lds;
        if (wide_cost(std::min<int64_t>(len_lds, max_keep), n_lds, G) < wide_cost(len_wide, n_wide, G)) n_wide = 0;
    }
    if (n_wide > 0 && n_wide <= kMaxMergeSplits && groups * n_wide < 65536) {
        p.wide_wg = (int32_t)(groups * n_wide);
        const uint32_t per = ((uint32_t)p.wide_wg + 7) / 8;
        p.sched.xcd = (per - 1) | ((uint32_t)p.wide_wg - 8 * (per - 1)) << 16;
        p.sched.magic_n = magic16((uint32_t)n_wide);
        p.sched.len = (uint32_t)len_wide | (uint32_t)n_wide << 9 | (uint32_t)G << 18;
        p.sched.hkv_b = (uint32_t)Hkv | (uint32_t)B << 16;
        p.sched.magic_hkv = magic16((uint32_t)Hkv);
        p.sched.magic_b = magic16((uint32_t)B);
        p.n_split = (int32_t)n_wide;
        p.split_len = (int32_t)len_wide;
        if (p.n_split > 1) {
            p.tickets = groups;
            p.ml_bytes = round_up((size_t)p.wide_wg * G * 2 * sizeof(float), 256);
            p.o_bytes = round_up((size_t)p.wide_wg * G * kHeadDim * sizeof(float), 256);
        }
    } else {
        if (split_len <= 0) split_len = (int32_t)lds_auto_split(max_keep, groups);  // a whole compute unit each
        p.split_len = split_len;
        p.n_split = (int32_t)(((int64_t)max_keep + split_len - 1) / split_len);
        if (p.n_split > 1) {
            // a counter per group, and for a two-level merge one per set of
            // kSubSplits splits after them
            const int64_t n_sub = (p.n_split + kSubSplits - 1) / kSubSplits;
            const bool two_level = p.n_split > 2 * kMergeBatch && p.n_split <= kTwoLevelMax;
            p.tickets = groups * (two_level ? 1 + n_sub : 1);
            p.ml_bytes = round_up((size_t)groups * p.n_split * G * 2 * sizeof(float), 256);
            p.o_bytes = round_up((size_t)groups * p.n_split * G * kHeadDim * sizeof(float), 256);
        }
    }
    // The smallest size whose ticket region holds the tickets and leaves room
    // for the partials, with 256 bytes to spare so that any larger size does
    // too (the region grows by 256 bytes at a time).
    const size_t part = p.ml_bytes + p.o_bytes;
    if (part == 0 && p.tickets == 0) {
        p.total = 256;
        return p;
    }
    size_t total = round_up(part + 512, 256);
    if (total < (size_t)p.tickets * 1024) total = round_up((size_t)p.tickets * 1024, 256);
    while (total < ticket_region(total) + part + 256) total += 256;
    p.total = total;
    return p;
}

namespace {

int check_host_policy(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B,
                      int32_t *counts, int32_t *max_count) {
    int32_t mx = 0;
    for (int32_t b = 0; b < B; ++b) {
        const murmur_seg &s = seg[b];
        const murmur_policy &p = pol[pol_per_seq ? b : 0];
        Pieces pc;
        if (retained_pieces(s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window, p.speech_delay,
                            p.speech_sink, p.out_window, p.out_sink, &pc) != 0)
            return fail(MURMUR_EINVAL,
                        "sequence %d: invalid layout or policy (seg %d/%d/%d/%d, policy %d/%d/%d/%d/%d)", b,
                        s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window, p.speech_delay,
                        p.speech_sink, p.out_window, p.out_sink);
        if (counts) counts[b] = pc.count;
        if (pc.count > mx) mx = pc.count;
    }
    if (max_count) *max_count = mx;
    return ok();
}

}  // namespace
}  // namespace murmur

namespace murmur {
namespace {

// Tickets in the ticket region at the start of the workspace, partials after
// it; the region depends only on ws_bytes (see murmur_decode_attn_workspace).
void bind_workspace(AttnLaunch &a, void *ws_dev, size_t ws_bytes) {
    uint8_t *ws = (uint8_t *)ws_dev;
    const size_t region = ticket_region(ws_bytes);
    a.ticket = (int32_t *)ws;
    a.part_ml = a.part_ml_bytes ? (float *)(ws + region) : nullptr;
    a.part_o = a.part_ml_bytes ? (float *)(ws + region + a.part_ml_bytes) : nullptr;
}

// Validation and launch description shared by murmur_decode_attn and the
// decode steps (everything but where the retained sets come from).  With
// ws_dev NULL and static_ws set, the workspace is the library's scratch array
// of ws_bytes (bound by the caller after these checks); otherwise ws_dev.
int prepare_attn(const void *q_dev, const murmur_kv *kv, int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv,
                 int32_t D, float scale, int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                 void *ws_dev, size_t ws_bytes, AttnLaunch &a, bool static_ws = false) {
    if (!q_dev || !kv || !out_dev || (!ws_dev && !static_ws))
        return fail(MURMUR_EINVAL, "q_dev, kv, out_dev and ws_dev must not be NULL");
    if (!kv->k || !kv->v) return fail(MURMUR_EINVAL, "kv->k and kv->v must not be NULL");
    if (B < 1 || Hq < 1 || Hkv < 1 || max_keep < 1 || kv->n_layers < 1 || kv->max_len < 1)
        return fail(MURMUR_EINVAL, "B, Hq, Hkv, max_keep, kv->n_layers and kv->max_len must be >= 1");
    if (Hq % Hkv != 0) return fail(MURMUR_EINVAL, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
    if (max_keep > kMaxKeep)
        return fail(MURMUR_EUNSUPPORTED, "max_keep %d exceeds %d (index-list offsets are 32-bit byte offsets)",
                    max_keep, kMaxKeep);
    if (D != kHeadDim) return fail(MURMUR_EUNSUPPORTED, "head_dim %d is not supported (only %d)", D, kHeadDim);
    if (Hq / Hkv > kMaxGroup)
        return fail(MURMUR_EUNSUPPORTED, "query heads per KV head %d exceeds %d", Hq / Hkv, kMaxGroup);
    if (out_dtype != MURMUR_DTYPE_BF16 && out_dtype != MURMUR_DTYPE_F32)
        return fail(MURMUR_EINVAL, "out_dtype must be MURMUR_DTYPE_BF16 or MURMUR_DTYPE_F32 (got %d)", out_dtype);
    if (!isfinite(scale)) return fail(MURMUR_EINVAL, "scale must be finite");
    if (split_len < 0 || split_len % kWaveTile != 0)
        return fail(MURMUR_EINVAL, "split_len must be 0 or a positive multiple of %d (got %d)", kWaveTile, split_len);
    const int64_t strides[4] = {kv->stride_layer, kv->stride_b, kv->stride_h, kv->stride_pos};
    for (int i = 0; i < 4; ++i)
        if (strides[i] < 0 || strides[i] % 8 != 0)
            return fail(MURMUR_EINVAL, "KV strides must be non-negative multiples of 8 elements");
    if (kv->stride_pos < kHeadDim && kv->max_len > 1)
        return fail(MURMUR_EINVAL, "kv->stride_pos (%lld) must be >= head_dim", (long long)kv->stride_pos);
    if (!aligned(q_dev, 16) || !aligned(kv->k, 16) || !aligned(kv->v, 16))
        return fail(MURMUR_EINVAL, "q_dev, kv->k and kv->v must be 16-byte aligned");
    if (!aligned(out_dev, 16) || !aligned(lse_dev, 4))
        return fail(MURMUR_EINVAL, "out_dev must be 16-byte and lse_dev 4-byte aligned");
    if (!aligned(ws_dev, 256)) return fail(MURMUR_EINVAL, "ws_dev must be 256-byte aligned");

    const WorkspacePlan plan = plan_workspace(kv->n_layers, B, Hq, Hkv, max_keep, split_len);
    if (ws_bytes < plan.total && static_ws)
        return fail(MURMUR_ENOSPACE, "this call needs %zu bytes of scratch; the allocation-free step has %zu "
                    "(use murmur_decode_step with a workspace)", plan.total, ws_bytes);
    if (ws_bytes < plan.total)
        return fail(MURMUR_ENOSPACE, "workspace of %zu bytes is too small (%zu needed)", ws_bytes, plan.total);
    if (plan.n_split > kMaxMergeSplits)
        return fail(MURMUR_EINVAL, "split_len %d gives %d splits for max_keep %d; at most %d are supported",
                    plan.split_len, plan.n_split, max_keep, kMaxMergeSplits);
    if (plan.o_bytes >= ((size_t)1 << 31))
        return fail(MURMUR_EINVAL, "split partials of %zu bytes exceed the 2 GiB a launch can address; use a longer "
                    "split_len", plan.o_bytes);
    if ((int64_t)kv->n_layers * Hkv > 65535 || B > 65535 || (int64_t)kv->n_layers * B * Hq > 0x7fffffffLL)
        return fail(MURMUR_EINVAL, "problem too large for one launch (n_layers * Hkv = %lld, B = %d)",
                    (long long)kv->n_layers * Hkv, B);

    a = AttnLaunch{};
    a.q = (const uint16_t *)q_dev;
    a.k = (const uint16_t *)kv->k;
    a.v = (const uint16_t *)kv->v;
    a.s_layer = kv->stride_layer;
    a.s_b = kv->stride_b;
    a.s_h = kv->stride_h;
    a.s_pos = kv->stride_pos;
    a.out = out_dev;
    a.lse = lse_dev;
    // Partials exist when a group has more than one split.
    const size_t region = ticket_region(ws_bytes);
    const bool partials = plan.ml_bytes > 0;
    if (partials != (plan.n_split > 1) || region < (size_t)plan.tickets * 4 * kTicketStride ||
        region + plan.ml_bytes + plan.o_bytes > ws_bytes)
        return fail(MURMUR_EINVAL, "internal: inconsistent workspace plan");
    a.part_ml_bytes = (uint32_t)plan.ml_bytes;
    a.part_o_bytes = (uint32_t)plan.o_bytes;
    if (!static_ws) bind_workspace(a, ws_dev, ws_bytes);
    a.max_len = kv->max_len;
    a.max_keep = max_keep;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.G = Hq / Hkv;
    a.NL = kv->n_layers;
    a.split_len = plan.split_len;
    a.n_split = plan.n_split;
    a.wide_wg = plan.wide_wg;
    a.sched = plan.sched;
    a.out_f32 = out_dtype == MURMUR_DTYPE_F32;
    a.scale_log2 = scale * 1.4426950408889634f;
    return ok();
}

}  // namespace
}  // namespace murmur

using namespace murmur;

MURMUR_EXPORT int murmur_abi_version(void) { return MURMUR_ABI_VERSION; }

MURMUR_EXPORT const char *murmur_last_error(void) { return g_last_error; }

MURMUR_EXPORT int murmur_retained_count_host(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq,
                                             int32_t B, int32_t *counts, int32_t *max_count) {
    if (!seg || !pol) return fail(MURMUR_EINVAL, "seg and pol must not be NULL");
    if (B < 1) return fail(MURMUR_EINVAL, "B must be >= 1 (got %d)", B);
    if (pol_per_seq != 0 && pol_per_seq != 1) return fail(MURMUR_EINVAL, "pol_per_seq must be 0 or 1");
    return check_host_policy(seg, pol, pol_per_seq, B, counts, max_count);
}

MURMUR_EXPORT int murmur_evict_compact(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                                       int32_t B, int32_t *idx_dev, int32_t max_keep, int32_t *count_dev,
                                       int32_t *ranges_dev, murmur_stream_t stream) {
    if (!seg_dev || !pol_dev || !idx_dev || !count_dev)
        return fail(MURMUR_EINVAL, "seg_dev, pol_dev, idx_dev and count_dev must not be NULL");
    if (B < 1) return fail(MURMUR_EINVAL, "B must be >= 1 (got %d)", B);
    if (max_keep < 1) return fail(MURMUR_EINVAL, "max_keep must be >= 1 (got %d)", max_keep);
    if (pol_per_seq != 0 && pol_per_seq != 1) return fail(MURMUR_EINVAL, "pol_per_seq must be 0 or 1");
    if (!aligned(seg_dev, 4) || !aligned(pol_dev, 4) || !aligned(idx_dev, 4) || !aligned(count_dev, 4) ||
        !aligned(ranges_dev, 4))
        return fail(MURMUR_EINVAL, "device pointers must be 4-byte aligned");
    if ((int64_t)B * max_keep > ((int64_t)1 << 40)) return fail(MURMUR_EINVAL, "B * max_keep too large");
    const int e = launch_evict_compact(seg_dev, pol_dev, pol_per_seq, B, idx_dev, max_keep, count_dev, ranges_dev,
                                       nullptr, 0, 0, stream);
    if (e != 0) return fail(MURMUR_EHIP, "evict_compact launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_evict_compact_paged(const murmur_seg *seg_dev, const murmur_policy *pol_dev,
                                             int32_t pol_per_seq, int32_t B, const int32_t *block_table_dev,
                                             int32_t max_blocks, int32_t block_size, int32_t *idx_dev,
                                             int32_t max_keep, int32_t *count_dev, int32_t *ranges_dev,
                                             murmur_stream_t stream) {
    if (!seg_dev || !pol_dev || !idx_dev || !count_dev || !block_table_dev)
        return fail(MURMUR_EINVAL, "seg_dev, pol_dev, block_table_dev, idx_dev and count_dev must not be NULL");
    if (B < 1) return fail(MURMUR_EINVAL, "B must be >= 1 (got %d)", B);
    if (max_keep < 1) return fail(MURMUR_EINVAL, "max_keep must be >= 1 (got %d)", max_keep);
    if (max_blocks < 1) return fail(MURMUR_EINVAL, "max_blocks must be >= 1 (got %d)", max_blocks);
    if (pol_per_seq != 0 && pol_per_seq != 1) return fail(MURMUR_EINVAL, "pol_per_seq must be 0 or 1");
    if (block_size < 1 || block_size > (1 << 20) || (block_size & (block_size - 1)) != 0)
        return fail(MURMUR_EINVAL, "block_size must be a power of two in [1, 2^20] (got %d)", block_size);
    if (!aligned(seg_dev, 4) || !aligned(pol_dev, 4) || !aligned(idx_dev, 4) || !aligned(count_dev, 4) ||
        !aligned(ranges_dev, 4) || !aligned(block_table_dev, 4))
        return fail(MURMUR_EINVAL, "device pointers must be 4-byte aligned");
    if ((int64_t)B * max_keep > ((int64_t)1 << 40) || (int64_t)B * max_blocks > ((int64_t)1 << 40))
        return fail(MURMUR_EINVAL, "B * max_keep or B * max_blocks too large");
    int log2_bs = 0;
    while ((1 << log2_bs) < block_size) ++log2_bs;
    const int e = launch_evict_compact(seg_dev, pol_dev, pol_per_seq, B, idx_dev, max_keep, count_dev, ranges_dev,
                                       block_table_dev, max_blocks, log2_bs, stream);
    if (e != 0) return fail(MURMUR_EHIP, "evict_compact_paged launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_freeable_blocks_host(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq,
                                             int32_t B, int32_t block_size, int32_t *blocks) {
    if (!seg || !pol || !blocks) return fail(MURMUR_EINVAL, "seg, pol and blocks must not be NULL");
    if (B < 1) return fail(MURMUR_EINVAL, "B must be >= 1 (got %d)", B);
    if (pol_per_seq != 0 && pol_per_seq != 1) return fail(MURMUR_EINVAL, "pol_per_seq must be 0 or 1");
    if (block_size < 1) return fail(MURMUR_EINVAL, "block_size must be >= 1 (got %d)", block_size);
    for (int32_t b = 0; b < B; ++b) {
        const murmur_seg &s = seg[b];
        const murmur_policy &p = pol[pol_per_seq ? b : 0];
        int32_t ranges[2][2];
        if (evicted_ranges(s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window, p.speech_delay,
                           p.speech_sink, p.out_window, p.out_sink, ranges[0], ranges[1]) != 0)
            return fail(MURMUR_EINVAL,
                        "sequence %d: invalid layout or policy (seg %d/%d/%d/%d, policy %d/%d/%d/%d/%d)", b,
                        s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window, p.speech_delay,
                        p.speech_sink, p.out_window, p.out_sink);
        // Whole blocks inside each range: from the first block that starts in it to the last that ends in it.
        for (int k = 0; k < 2; ++k) {
            const int64_t lo = ranges[k][0], hi = (int64_t)ranges[k][0] + ranges[k][1];
            const int64_t first = (lo + block_size - 1) / block_size, end = hi / block_size;
            int32_t *out = blocks + (int64_t)b * 4 + 2 * k;
            out[0] = end > first ? (int32_t)first : 0;
            out[1] = end > first ? (int32_t)(end - first) : 0;
        }
    }
    return ok();
}

MURMUR_EXPORT int murmur_paged_step(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                                    int32_t B, int32_t *block_table_dev, int32_t max_blocks, int32_t block_size,
                                    int32_t *free_stack_dev, int32_t *free_top_dev, int32_t capacity,
                                    int32_t full_scan, const murmur_kv *pool, int32_t Hkv, const void *k_new_dev,
                                    const void *v_new_dev, murmur_stream_t stream) {
    if (!seg_dev || !pol_dev || !block_table_dev || !free_stack_dev || !free_top_dev)
        return fail(MURMUR_EINVAL, "seg_dev, pol_dev, block_table_dev, free_stack_dev and free_top_dev must not be NULL");
    if (B < 1) return fail(MURMUR_EINVAL, "B must be >= 1 (got %d)", B);
    if (max_blocks < 1) return fail(MURMUR_EINVAL, "max_blocks must be >= 1 (got %d)", max_blocks);
    if (capacity < 1) return fail(MURMUR_EINVAL, "capacity must be >= 1 (got %d)", capacity);
    if (pol_per_seq != 0 && pol_per_seq != 1) return fail(MURMUR_EINVAL, "pol_per_seq must be 0 or 1");
    if (full_scan != 0 && full_scan != 1) return fail(MURMUR_EINVAL, "full_scan must be 0 or 1");
    if (block_size < 1 || block_size > (1 << 20) || (block_size & (block_size - 1)) != 0)
        return fail(MURMUR_EINVAL, "block_size must be a power of two in [1, 2^20] (got %d)", block_size);
    if (!aligned(seg_dev, 4) || !aligned(pol_dev, 4) || !aligned(block_table_dev, 4) || !aligned(free_stack_dev, 4) ||
        !aligned(free_top_dev, 4))
        return fail(MURMUR_EINVAL, "device pointers must be 4-byte aligned");
    if ((int64_t)B * max_blocks > ((int64_t)1 << 40)) return fail(MURMUR_EINVAL, "B * max_blocks too large");
    if (pool) {
        if (!pool->k || !pool->v || !k_new_dev || !v_new_dev)
            return fail(MURMUR_EINVAL, "with a pool, pool->k, pool->v, k_new_dev and v_new_dev must not be NULL");
        if (Hkv < 1 || pool->n_layers < 1 || pool->max_len < 1)
            return fail(MURMUR_EINVAL, "Hkv, pool->n_layers and pool->max_len must be >= 1");
        const int64_t strides[3] = {pool->stride_layer, pool->stride_h, pool->stride_pos};
        for (int i = 0; i < 3; ++i)
            if (strides[i] < 0 || strides[i] % 8 != 0)
                return fail(MURMUR_EINVAL, "pool strides must be non-negative multiples of 8 elements");
        if (pool->stride_pos < kHeadDim && pool->max_len > 1)
            return fail(MURMUR_EINVAL, "pool->stride_pos (%lld) must be >= head_dim", (long long)pool->stride_pos);
        if (!aligned(pool->k, 16) || !aligned(pool->v, 16) || !aligned(k_new_dev, 16) || !aligned(v_new_dev, 16))
            return fail(MURMUR_EINVAL, "pool->k, pool->v, k_new_dev and v_new_dev must be 16-byte aligned");
        if ((int64_t)B * pool->n_layers * Hkv > ((int64_t)1 << 36))
            return fail(MURMUR_EINVAL, "B * n_layers * Hkv too large");
    }
    int log2_bs = 0;
    while ((1 << log2_bs) < block_size) ++log2_bs;
    int e = launch_paged_step(seg_dev, pol_dev, pol_per_seq, B, block_table_dev, max_blocks, log2_bs, free_stack_dev,
                              free_top_dev, capacity, full_scan, stream);
    if (e != 0) return fail(MURMUR_EHIP, "paged_step launch failed: %s", hip_error_text(e));
    if (pool) {
        e = launch_paged_append(seg_dev, B, block_table_dev, max_blocks, log2_bs, *pool, Hkv, k_new_dev, v_new_dev,
                                stream);
        if (e != 0) return fail(MURMUR_EHIP, "paged_step append launch failed: %s", hip_error_text(e));
    }
    return ok();
}

MURMUR_EXPORT int murmur_decode_attn_workspace(int32_t n_layers, int32_t B, int32_t Hq, int32_t Hkv,
                                               int32_t max_keep, int32_t split_len, size_t *bytes) {
    if (!bytes) return fail(MURMUR_EINVAL, "bytes must not be NULL");
    if (n_layers < 1 || B < 1 || Hq < 1 || Hkv < 1 || max_keep < 1)
        return fail(MURMUR_EINVAL, "n_layers, B, Hq, Hkv and max_keep must be >= 1");
    if (Hq % Hkv != 0) return fail(MURMUR_EINVAL, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
    if (split_len < 0 || split_len % kWaveTile != 0)
        return fail(MURMUR_EINVAL, "split_len must be 0 or a positive multiple of %d (got %d)", kWaveTile, split_len);
    *bytes = plan_workspace(n_layers, B, Hq, Hkv, max_keep, split_len).total;
    return ok();
}

MURMUR_EXPORT int murmur_decode_attn_workspace_init(void *ws_dev, size_t ws_bytes, murmur_stream_t stream) {
    if (!ws_dev) return fail(MURMUR_EINVAL, "ws_dev must not be NULL");
    if (!aligned(ws_dev, 256)) return fail(MURMUR_EINVAL, "ws_dev must be 256-byte aligned");
    const int64_t n = (int64_t)(ws_bytes / sizeof(int32_t));
    if (n < 1) return ok();
    const int e = launch_workspace_init((int32_t *)ws_dev, n, stream);
    if (e != 0) return fail(MURMUR_EHIP, "workspace_init launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_decode_attn(const void *q_dev, const murmur_kv *kv, const int32_t *idx_dev, const int32_t *ranges_dev,
                                     const int32_t *count_dev, int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                     float scale, int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                                     void *ws_dev, size_t ws_bytes, murmur_stream_t stream) {
    if (!idx_dev && !ranges_dev) return fail(MURMUR_EINVAL, "one of idx_dev and ranges_dev is required");
    if (!ranges_dev && !count_dev) return fail(MURMUR_EINVAL, "count_dev is required with an index list");
    if (!aligned(count_dev, 4) || !aligned(idx_dev, 4) || !aligned(ranges_dev, 4))
        return fail(MURMUR_EINVAL, "count/idx/ranges pointers must be 4-byte aligned");
    AttnLaunch a;
    const int rc = prepare_attn(q_dev, kv, max_keep, B, Hq, Hkv, D, scale, split_len, out_dev, out_dtype, lse_dev,
                                ws_dev, ws_bytes, a);
    if (rc != MURMUR_OK) return rc;
    a.src0 = ranges_dev ? nullptr : count_dev;  // a range table carries its own counts
    a.src1 = ranges_dev;
    a.idx = idx_dev;
    a.src_mode = ranges_dev ? kSrcRanges : kSrcIndex;
    const int e = launch_decode_attn(a, stream);
    if (e != 0) return fail(MURMUR_EHIP, "decode_attn launch failed: %s", hip_error_text(e));
    return ok();
}

namespace {

// Checks and launch description of murmur_decode_step and its allocation-free
// variant (static_ws: the workspace is bound by the caller).
int prepare_step(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq, const void *q_dev,
                 const murmur_kv *kv, int32_t *idx_dev, int32_t *count_dev, int32_t *ranges_dev, int32_t max_keep,
                 int32_t B, int32_t Hq, int32_t Hkv, int32_t D, float scale, int32_t split_len, void *out_dev,
                 int32_t out_dtype, float *lse_dev, void *ws_dev, size_t ws_bytes, bool static_ws, AttnLaunch &a) {
    if (!seg_dev || !pol_dev) return fail(MURMUR_EINVAL, "seg_dev and pol_dev must not be NULL");
    if (pol_per_seq < 0 || pol_per_seq > (MURMUR_POL_PER_SEQ | MURMUR_POL_PER_LAYER))
        return fail(MURMUR_EINVAL, "pol_per_seq must be a set of MURMUR_POL_* bits (0..3, got %d)", pol_per_seq);
    if (!aligned(seg_dev, 4) || !aligned(pol_dev, 4) || !aligned(idx_dev, 4) || !aligned(count_dev, 4) ||
        !aligned(ranges_dev, 4))
        return fail(MURMUR_EINVAL, "seg/pol/idx/count/ranges pointers must be 4-byte aligned");
    if ((int64_t)B * max_keep > ((int64_t)1 << 40)) return fail(MURMUR_EINVAL, "B * max_keep too large");
    const int rc = prepare_attn(q_dev, kv, max_keep, B, Hq, Hkv, D, scale, split_len, out_dev, out_dtype, lse_dev,
                                ws_dev, ws_bytes, a, static_ws);
    if (rc != MURMUR_OK) return rc;
    a.src0 = reinterpret_cast<const int32_t *>(seg_dev);
    a.src1 = reinterpret_cast<const int32_t *>(pol_dev);
    a.pol_per_seq = pol_per_seq;
    a.src_mode = kSrcLayout;
    a.idx_out = idx_dev;
    a.count_out = count_dev;
    a.ranges_out = ranges_dev;
    return ok();
}

}  // namespace

MURMUR_EXPORT int murmur_decode_step(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                                     const void *q_dev, const murmur_kv *kv, int32_t *idx_dev, int32_t *count_dev,
                                     int32_t *ranges_dev, int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                     float scale, int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                                     void *ws_dev, size_t ws_bytes, murmur_stream_t stream) {
    AttnLaunch a;
    const int rc = prepare_step(seg_dev, pol_dev, pol_per_seq, q_dev, kv, idx_dev, count_dev, ranges_dev, max_keep, B,
                                Hq, Hkv, D, scale, split_len, out_dev, out_dtype, lse_dev, ws_dev, ws_bytes, false, a);
    if (rc != MURMUR_OK) return rc;
    const int e = launch_decode_attn(a, stream);
    if (e != 0) return fail(MURMUR_EHIP, "decode_step launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_decode_step_static(const murmur_seg *seg_dev, const murmur_policy *pol_dev,
                                            int32_t pol_per_seq, const void *q_dev, const murmur_kv *kv,
                                            int32_t *idx_dev, int32_t *count_dev, int32_t *ranges_dev,
                                            int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                                            float scale, int32_t split_len, void *out_dev, int32_t out_dtype,
                                            float *lse_dev, murmur_stream_t stream) {
    AttnLaunch a;
    const int rc = prepare_step(seg_dev, pol_dev, pol_per_seq, q_dev, kv, idx_dev, count_dev, ranges_dev, max_keep, B,
                                Hq, Hkv, D, scale, split_len, out_dev, out_dtype, lse_dev, nullptr,
                                MURMUR_STATIC_SCRATCH_BYTES, true, a);
    if (rc != MURMUR_OK) return rc;
    void *scratch = nullptr;
    bool fresh = false;
    int e = static_scratch(&scratch, &fresh);
    if (e != 0) return fail(MURMUR_EHIP, "looking up the scratch array failed: %s", hip_error_text(e));
    if (fresh) {  // first call on this device: the tickets start at zero (later calls leave them at zero)
        e = launch_workspace_init((int32_t *)scratch, (int64_t)(ticket_region(MURMUR_STATIC_SCRATCH_BYTES) / 4),
                                  stream);
        if (e != 0) return fail(MURMUR_EHIP, "scratch ticket reset failed: %s", hip_error_text(e));
    }
    bind_workspace(a, scratch, MURMUR_STATIC_SCRATCH_BYTES);
    e = launch_decode_attn(a, stream);
    if (e != 0) return fail(MURMUR_EHIP, "decode_step_static launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_ring_layout_host(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq,
                                          int32_t B, int32_t out_capacity, int32_t *ranges, int32_t *cur_row) {
    if (!seg || !pol) return fail(MURMUR_EINVAL, "seg and pol must not be NULL");
    if (B < 1) return fail(MURMUR_EINVAL, "B must be >= 1 (got %d)", B);
    if (pol_per_seq != 0 && pol_per_seq != 1) return fail(MURMUR_EINVAL, "pol_per_seq must be 0 or 1");
    if (out_capacity < 1) return fail(MURMUR_EINVAL, "out_capacity must be >= 1 (got %d)", out_capacity);
    for (int32_t b = 0; b < B; ++b) {
        const murmur_seg &s = seg[b];
        const murmur_policy &p = pol[pol_per_seq ? b : 0];
        Pieces pc;
        int32_t cur = 0;
        const int rc = ring_pieces(s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window,
                                   p.speech_delay, p.speech_sink, p.out_window, p.out_sink, out_capacity, &pc, &cur);
        if (rc == -2)
            return fail(MURMUR_EINVAL, "sequence %d: a ring of %d rows cannot hold the retained outputs (out_len %d, "
                        "out_window %d, out_sink %d)", b, out_capacity, s.out_len, p.out_window, p.out_sink);
        if (rc != 0)
            return fail(MURMUR_EINVAL,
                        "sequence %d: invalid layout or policy (seg %d/%d/%d/%d, policy %d/%d/%d/%d/%d)", b,
                        s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window, p.speech_delay,
                        p.speech_sink, p.out_window, p.out_sink);
        if (ranges)
            for (int k = 0; k < kPieces; ++k) {
                ranges[(int64_t)b * 2 * kPieces + 2 * k] = pc.start[k];
                ranges[(int64_t)b * 2 * kPieces + 2 * k + 1] = pc.len[k];
            }
        if (cur_row) cur_row[b] = cur;
    }
    return ok();
}

MURMUR_EXPORT int murmur_decode_step_ring(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                                          const murmur_ring *ring, const void *q_dev, const murmur_kv *kv,
                                          int32_t *idx_dev, int32_t *count_dev, int32_t *ranges_dev, int32_t max_keep,
                                          int32_t B, int32_t Hq, int32_t Hkv, int32_t D, float scale,
                                          int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                                          void *ws_dev, size_t ws_bytes, murmur_stream_t stream) {
    if (!seg_dev || !pol_dev || !ring) return fail(MURMUR_EINVAL, "seg_dev, pol_dev and ring must not be NULL");
    if (pol_per_seq < 0 || pol_per_seq > (MURMUR_POL_PER_SEQ | MURMUR_POL_PER_LAYER))
        return fail(MURMUR_EINVAL, "pol_per_seq must be a set of MURMUR_POL_* bits (0..3, got %d)", pol_per_seq);
    if (!ring->k_new || !ring->v_new) return fail(MURMUR_EINVAL, "ring->k_new and ring->v_new must not be NULL");
    if (!aligned(ring->k_new, 16) || !aligned(ring->v_new, 16))
        return fail(MURMUR_EINVAL, "ring->k_new and ring->v_new must be 16-byte aligned");
    if (ring->out_capacity < 1)
        return fail(MURMUR_EINVAL, "ring->out_capacity must be >= 1 (got %d)", ring->out_capacity);
    if (!aligned(seg_dev, 4) || !aligned(pol_dev, 4) || !aligned(idx_dev, 4) || !aligned(count_dev, 4) ||
        !aligned(ranges_dev, 4))
        return fail(MURMUR_EINVAL, "seg/pol/idx/count/ranges pointers must be 4-byte aligned");
    if ((int64_t)B * max_keep > ((int64_t)1 << 40)) return fail(MURMUR_EINVAL, "B * max_keep too large");
    AttnLaunch a;
    const int rc = prepare_attn(q_dev, kv, max_keep, B, Hq, Hkv, D, scale, split_len, out_dev, out_dtype, lse_dev,
                                ws_dev, ws_bytes, a);
    if (rc != MURMUR_OK) return rc;
    a.src0 = reinterpret_cast<const int32_t *>(seg_dev);
    a.src1 = reinterpret_cast<const int32_t *>(pol_dev);
    a.pol_per_seq = pol_per_seq;
    a.src_mode = kSrcRing;
    a.idx_out = idx_dev;
    a.count_out = count_dev;
    a.ranges_out = ranges_dev;
    a.ring_cap = ring->out_capacity;
    a.k_new = (const uint16_t *)ring->k_new;
    a.v_new = (const uint16_t *)ring->v_new;
    const int e = launch_decode_attn(a, stream);
    if (e != 0) return fail(MURMUR_EHIP, "decode_step_ring launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_plan_chunks(const double *seg_start, const double *seg_end, int32_t n_seg,
                                     double audio_len, double max_chunk, double tokens_per_s, int32_t *chunk_of_seg,
                                     double *chunk_start, double *chunk_len, int32_t *speech_tokens,
                                     int32_t max_chunks, int32_t *n_chunks) {
    if (!n_chunks || (n_seg > 0 && (!seg_start || !seg_end)) || (max_chunks > 0 && (!chunk_start || !chunk_len)))
        return fail(MURMUR_EINVAL, "missing segment or chunk arrays");
    if (n_seg < 0 || max_chunks < 0) return fail(MURMUR_EINVAL, "n_seg and max_chunks must be >= 0");
    if (!(max_chunk > 0) || !(audio_len >= 0) || !(tokens_per_s >= 0) || !isfinite(audio_len) ||
        !isfinite(max_chunk) || !isfinite(tokens_per_s))
        return fail(MURMUR_EINVAL, "audio_len and tokens_per_s must be >= 0 and max_chunk > 0, all finite");
    if (audio_len / max_chunk > (double)(1 << 24) || max_chunk * tokens_per_s > 2e9 || n_seg > (1 << 24))
        return fail(MURMUR_EINVAL, "more than 2^24 chunks or segments, or more than 2e9 speech tokens per chunk");
    for (int32_t i = 0; i < n_seg; ++i) {
        if (!(seg_start[i] >= 0) || !(seg_end[i] > seg_start[i]) || !(seg_end[i] <= audio_len))
            return fail(MURMUR_EINVAL, "segment %d [%g, %g) is empty or outside [0, %g]", i, seg_start[i], seg_end[i],
                        audio_len);
        if (i > 0 && seg_start[i] < seg_end[i - 1])
            return fail(MURMUR_EINVAL, "segment %d starts before segment %d ends (unsorted or overlapping)", i, i - 1);
    }
    // Pass 1: chunk boundaries.  `speech`: the open chunk holds (part of) a segment.
    int32_t n = 0;
    auto emit = [&](double start, double len) {
        if (n < max_chunks) {
            chunk_start[n] = start;
            chunk_len[n] = len;
            if (speech_tokens) speech_tokens[n] = (int32_t)llround(len * tokens_per_s);
        }
        ++n;
    };
    double start = 0.0;
    bool speech = false;
    for (int32_t i = 0; i < n_seg;) {
        if (seg_end[i] - start <= max_chunk) {  // segment i (or what is left of it) ends within the chunk
            speech = true;
            ++i;
            continue;
        }
        // Segment i does not end within the chunk: close the chunk max_chunk after its start, unless that
        // falls inside segment i and the segment can stay whole (it fits a chunk of its own) or the chunk
        // already holds speech before it: then where the segment begins.
        double end = start + max_chunk;
        const bool whole = seg_end[i] - seg_start[i] <= max_chunk;
        if ((speech || whole) && seg_start[i] < end) end = seg_start[i];
        emit(start, end - start);
        start = end;
        speech = false;
    }
    // The last chunk keeps the silence after the last segment, up to audio_len or max_chunk after its start.
    if (n_seg > 0) emit(start, (audio_len < start + max_chunk ? audio_len : start + max_chunk) - start);
    *n_chunks = n;
    if (n > max_chunks) return fail(MURMUR_ENOSPACE, "%d chunks needed, %d allowed", n, max_chunks);
    // Pass 2: the chunk holding each segment's start (chunks are in time order).
    if (chunk_of_seg) {
        int32_t c = 0;
        for (int32_t i = 0; i < n_seg; ++i) {
            while (c + 1 < n && chunk_start[c + 1] <= seg_start[i]) ++c;
            chunk_of_seg[i] = c;
        }
    }
    return ok();
}

MURMUR_EXPORT int murmur_chunk_timestamps(const double *t_local, const int32_t *chunk, int32_t n,
                                          const double *chunk_len, int32_t n_chunks, double *t) {
    if (n < 0 || n_chunks < 0) return fail(MURMUR_EINVAL, "n and n_chunks must be >= 0");
    if (n > 0 && (!t_local || !chunk || !t || !chunk_len)) return fail(MURMUR_EINVAL, "missing arrays");
    for (int32_t c = 0; c < n_chunks; ++c)
        if (!(chunk_len[c] >= 0)) return fail(MURMUR_EINVAL, "chunk %d has a negative length", c);
    for (int32_t k = 0; k < n; ++k)
        if (chunk[k] < 0 || chunk[k] >= n_chunks)
            return fail(MURMUR_EINVAL, "timestamp %d names chunk %d of %d", k, chunk[k], n_chunks);
    // offset(i): the lengths of the chunks before i, accumulated in order.
    double *offset = new double[n_chunks > 0 ? n_chunks : 1];
    double acc = 0.0;
    for (int32_t c = 0; c < n_chunks; ++c) {
        offset[c] = acc;
        acc += chunk_len[c];
    }
    for (int32_t k = 0; k < n; ++k) t[k] = t_local[k] + offset[chunk[k]];
    delete[] offset;
    return ok();
}

MURMUR_EXPORT int murmur_read_probe(const void *buf_dev, size_t bytes, int32_t n_workgroups, int32_t threads,
                                    int32_t depth, int32_t mode, uint32_t *sink_dev, murmur_stream_t stream) {
    if (!buf_dev || !sink_dev) return fail(MURMUR_EINVAL, "buf_dev and sink_dev must not be NULL");
    if (!aligned(buf_dev, 16) || !aligned(sink_dev, 4))
        return fail(MURMUR_EINVAL, "buf_dev must be 16-byte and sink_dev 4-byte aligned");
    if (bytes == 0 || bytes % 16 != 0) return fail(MURMUR_EINVAL, "bytes must be a positive multiple of 16");
    if (n_workgroups < 1 || n_workgroups > 65535) return fail(MURMUR_EINVAL, "n_workgroups must be in [1, 65535]");
    if (threads < 64 || threads > 1024 || threads % 64 != 0)
        return fail(MURMUR_EINVAL, "threads must be a multiple of 64 in [64, 1024]");
    if (depth != 1 && depth != 2 && depth != 4 && depth != 8 && depth != 16)
        return fail(MURMUR_EINVAL, "depth must be 1, 2, 4, 8 or 16");
    if (mode != MURMUR_PROBE_REGISTERS && mode != MURMUR_PROBE_LDS)
        return fail(MURMUR_EINVAL, "mode must be MURMUR_PROBE_REGISTERS or MURMUR_PROBE_LDS");
    if (mode == MURMUR_PROBE_LDS && (threads / 64) * depth > 64)
        return fail(MURMUR_EINVAL, "MURMUR_PROBE_LDS needs (threads / 64) * depth KiB of LDS, at most 64");
    const int e = launch_read_probe(buf_dev, (int64_t)(bytes / 16), n_workgroups, threads, depth,
                                    mode == MURMUR_PROBE_LDS, sink_dev, stream);
    if (e != 0) return fail(MURMUR_EHIP, "read_probe launch failed: %s", hip_error_text(e));
    return ok();
}

MURMUR_EXPORT int murmur_device_error(murmur_stream_t stream, int32_t *code) {
    if (!code) return fail(MURMUR_EINVAL, "code must not be NULL");
    const int e = read_and_clear_device_error(stream, code);
    if (e != 0) return fail(MURMUR_EHIP, "reading the device error word failed: %s", hip_error_text(e));
    return ok();
}
