// Internal interface between the C ABI layer (api.cpp) and the gfx950 kernels
// (kernels.hip).  Not installed; include/murmur.h is the public surface.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "murmur.h"

namespace murmur {

constexpr int kHeadDim = 128;     // head_dim supported by the attention kernel
constexpr int kMaxGroup = 16;     // query heads per KV head (MFMA tile height)
constexpr int kWaveTile = 32;     // retained positions one wavefront handles per pass
constexpr int kWavesPerWg = 4;
constexpr int kSplitUnit = kWaveTile * kWavesPerWg;  // 128 positions: one pass of a workgroup
constexpr int kMaxAutoSplits = 64;
constexpr int kRoundWorkgroups = 256;     // one workgroup per compute unit
// Splits one merge can combine: it stages 2 * n_split * G + 2 * G floats in
// the workgroup's 32 KiB of V-tile LDS.
constexpr int kMaxMergeSplits = 240;
constexpr int kMaxKeep = 1 << 28;  // retained positions per sequence the attention accepts
constexpr int kMergeBatch = 8;  // splits whose partials one merging thread loads at once
// The LDS-staged schedule merges groups of more than 2 * kMergeBatch and at
// most kTwoLevelMax splits in two levels, sets of kSubSplits splits first (so
// that the second level folds at most 16 partials too).
constexpr int kSubSplits = 8;
constexpr int kTwoLevelMax = 128;
// Split-choice model (measured on MI355X): one compute unit streams about 40 GB/s from HBM however many
// wavefronts it runs, and the split-K merge chain (partial stores, ticket, loading the partials) costs
// about 2.3 us on top of the data phase.
constexpr double kCuBytesPerUs = 40e3;
constexpr double kMergeChainUs = 2.3;
// The wide schedule's merge keeps two batches of kMergeBatch partials in flight: every further
// 2 * kMergeBatch partials of a group add one serial load round trip (measured: 14 splits of 192
// positions 8.5 us, 17 of 160 9.0 us on 4 groups of 2592).
constexpr double kMergeRoundTripUs = 0.5;

// Wide schedule: workgroups of kWideWaves wavefronts, each wavefront one pass
// of kWaveTile retained positions, so a split holds at most kWideSplit.
constexpr int kWideWaves = 8;
constexpr int kWideSplit = kWideWaves * kWaveTile;  // 256

// Work of the wide schedule's workgroups, decoded on the device with exact
// multiply-high divisions (values below 2^16, multipliers ceil(2^32 / d), 0
// for d = 1): every (layer, sequence, KV head) group is cut into n splits of
// len positions; the w-th (group, split) in that order goes to the workgroup
// that xcd_order maps to w and, when its group has more than one split,
// leaves its partial in slot w.
struct WideSched {
    uint32_t xcd;       // (per - 1) | tall << 16 for W workgroups: per = ceil(W / 8) and tall = W - 8 (per - 1)
                        // (see xcd_order)
    uint32_t magic_n;   // ceil(2^32 / n)
    uint32_t len;       // len | n << 9 | G << 18 (split lengths <= 256, n <= kMaxMergeSplits, G query heads
                        // per KV head); the launch adds the policy mode (MURMUR_POL_* bits) << 23, at
                        // bit 25 whether stride_pos < kRunRowLimit and at bit 26 whether every group's
                        // first K/V element lies below 2^31 elements
    uint32_t hkv_b;     // Hkv | B << 16
    uint32_t magic_hkv;
    uint32_t magic_b;
};

// Row strides (elements) below this let a pass of kWaveTile consecutive rows
// address its K/V rows with 32-bit byte offsets from its first row.
constexpr int64_t kRunRowLimit = (int64_t)1 << 23;

// Launch description of one decode_attn call, fully validated by the caller.
// Where the attention takes the retained sets from (see AttnLaunch::src0/src1).
enum SrcMode : int32_t { kSrcIndex = 0, kSrcRanges = 1, kSrcLayout = 2, kSrcRing = 3 };

struct AttnLaunch {
    // kSrcIndex / kSrcRanges: src0 = counts [B], src1 = range tables [B][6][2]
    // (kSrcRanges); kSrcLayout and kSrcRing: src0 = layouts (murmur_seg [B]),
    // src1 = policies (murmur_policy [1] or [B], pol_per_seq).
    const int32_t *src0;
    const int32_t *src1;
    int32_t src_mode, pol_per_seq;
    int32_t *idx_out, *count_out, *ranges_out;  // kSrcLayout / kSrcRing: optional evict_compact outputs
    // kSrcRing: output ring rows, and the current token's K/V [NL][B][Hkv][D]
    // (read instead of its ring row, then appended there).
    int32_t ring_cap;
    const uint16_t *k_new;
    const uint16_t *v_new;
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    int64_t s_layer, s_b, s_h, s_pos;
    const int32_t *idx;
    void *out;
    float *lse;
    int32_t *ticket;   // [groups][kTicketStride]: one counter per group (layer, sequence, KV head), then
                       // for a two-level merge one per set of kSubSplits splits, [groups][n_sub]
    float *part_ml;    // [groups][n_split][G][2]  (running max in log2 units, sum)
    float *part_o;     // [groups][n_split][G][128]
    uint32_t part_ml_bytes, part_o_bytes;  // extents of the two partial arrays (< 2^31)
    int32_t max_len, max_keep, B, Hq, Hkv, G, NL;
    int32_t split_len, n_split, out_f32;
    float scale_log2;  // logit scale times log2(e)
    int32_t wide_wg;   // > 0: the wide schedule with this many workgroups (sched)
    WideSched sched;
};

struct WorkspacePlan {
    int32_t split_len;
    int32_t n_split;  // splits per group (the wide schedule: of the groups with the most)
    int32_t wide_wg;  // > 0: the wide schedule's workgroups
    WideSched sched;
    int64_t groups;
    int64_t tickets;  // ticket counters the launch uses
    size_t ml_bytes, o_bytes, total;
};

// Ticket counters sit kTicketStride int32 apart (one 128-byte cache line
// each), so that the atomics of different groups do not queue on one line.
constexpr int kTicketStride = 32;
// Bytes at the start of a workspace of ws_bytes that hold the tickets (the
// partials follow): 128 bytes per KiB, rounded up to 256, room for a ticket
// per KiB.  Depends on the size alone, so calls of different shapes that share
// a workspace place their tickets alike, and never where another call left
// partials.
size_t ticket_region(size_t ws_bytes);

// Split choice and workspace layout; deterministic in its arguments.
WorkspacePlan plan_workspace(int32_t n_layers, int32_t B, int32_t Hq, int32_t Hkv, int32_t max_keep,
                             int32_t split_len);

// Kernel launchers (kernels.hip).  They return a hipError_t value as int.
int launch_evict_compact(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B,
                         int32_t *idx, int32_t max_keep, int32_t *count, int32_t *ranges, const int32_t *bt,
                         int32_t max_blocks, int32_t log2_bs, murmur_stream_t stream);
int launch_decode_attn(const AttnLaunch &a, murmur_stream_t stream);
int launch_workspace_init(int32_t *ticket, int64_t n, murmur_stream_t stream);
// Device address of the current device's scratch array (MURMUR_STATIC_SCRATCH_BYTES,
// 256-byte aligned), looked up once per device; *fresh is true on that first
// lookup, when the caller must zero the ticket region.  Returns a hipError_t value.
int static_scratch(void **ptr, bool *fresh);
int launch_read_probe(const void *buf, int64_t n16, int32_t n_workgroups, int32_t threads, int32_t depth, bool lds,
                      uint32_t *sink, murmur_stream_t stream);
int launch_paged_step(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B, int32_t *bt,
                      int32_t max_blocks, int32_t log2_bs, int32_t *stack, int32_t *top, int32_t capacity,
                      int32_t full_scan, murmur_stream_t stream);
int launch_paged_append(const murmur_seg *seg, int32_t B, const int32_t *bt, int32_t max_blocks, int32_t log2_bs,
                        const murmur_kv &pool, int32_t Hkv, const void *k_new, const void *v_new,
                        murmur_stream_t stream);
int read_and_clear_device_error(murmur_stream_t stream, int32_t *code);
const char *hip_error_text(int err);

}  // namespace murmur
