// gfx950 (MI355X, CDNA4) kernels of libmurmur.
//
//   evict_compact_kernel     Section 3.2, Algorithms 1-2 and Equation 2: the
//                            retained set of every sequence as an ascending
//                            index list, a count and a six-piece range table.
//   decode_attn_wide_kernel  Section 3.2, Equation 1: split-K grouped-query
//                            decode attention over the retained positions,
//                            splits of up to 256 positions, eight wavefronts
//                            per workgroup, one 32-position pass each.
//   decode_attn_lds_kernel   the same for longer splits: each wavefront
//                            streams its passes through LDS stages.
//   Both accumulate in fp32 and fuse the log-sum-exp merge of the splits into
//   the last workgroup of each (layer, sequence, KV head).
//   paged_step_kernel, paged_append_kernel: the device block manager of the
//   paged cache (freeing behind the windows, appending the current token).
//
// Attention data flow per 64-wide wavefront and pass of 32 retained positions:
//   K, V rows --global_load_lds_dwordx4--> LDS stage (XOR-swizzled 16 B chunks)
//   K: ds_read_b128 --> MFMA A operands      S^T = K Q^T (16x16x32 bf16)
//   V: ds_read_b64_tr_b16 (transposing) --> MFMA B operands
//   P = exp2(S - m) stays in registers: the S^T accumulator layout is already
//   the A-operand layout of O = P V, split into bf16 hi + lo parts so the
//   product keeps ~16 mantissa bits.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "internal.h"
#include "policy.h"

namespace murmur {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Per-device error word (MURMUR_DEVERR_* bits); read and cleared by the host.
__device__ int32_t g_device_error;

static __device__ __forceinline__ void raise_device_error(int32_t bit) { atomicOr(&g_device_error, bit); }

// ---------------------------------------------------------------------------
// evict_compact: one workgroup per sequence.
// ---------------------------------------------------------------------------
// With a block table (paged cache, bt != null) the index list holds pool rows
// (paged_pool_row): a position past the table's max_blocks entries, in a freed
// block (negative entry) or in a row beyond 2^31 - 1 gives -1 and
// MURMUR_DEVERR_BLOCK.
static __device__ __forceinline__ int32_t paged_row(const int32_t *bt_row, int32_t max_blocks, int32_t log2_bs,
                                                    int32_t p, int &bad) {
    const int32_t row = paged_pool_row(bt_row, max_blocks, log2_bs, p);
    bad |= row < 0;
    return row;
}

__global__ __launch_bounds__(256) void evict_compact_kernel(const murmur_seg *__restrict__ seg,
                                                            const murmur_policy *__restrict__ pol,
                                                            int32_t pol_per_seq, int32_t max_keep,
                                                            int32_t *__restrict__ idx, int32_t *__restrict__ count,
                                                            int32_t *__restrict__ ranges,
                                                            const int32_t *__restrict__ bt, int32_t max_blocks,
                                                            int32_t log2_bs) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const murmur_seg s = seg[b];
    const murmur_policy p = pol[pol_per_seq ? b : 0];
    Pieces pc;
    const int rc = retained_pieces(s.prompt_pre, s.speech_len, s.prompt_mid, s.out_len, p.speech_window,
                                   p.speech_delay, p.speech_sink, p.out_window, p.out_sink, &pc);
    int32_t *row = idx + (int64_t)b * max_keep;
    if (rc != 0) {
        if (tid == 0) {
            count[b] = 0;
            raise_device_error(MURMUR_DEVERR_POLICY);
        }
        if (ranges && tid < 2 * kPieces) ranges[b * 2 * kPieces + tid] = 0;
        for (int r = tid; r < max_keep; r += blockDim.x) row[r] = -1;
        return;
    }
    if (tid == 0) {
        count[b] = pc.count;
        if (pc.count > max_keep) raise_device_error(MURMUR_DEVERR_OVERFLOW);
    }
    if (ranges && tid < 2 * kPieces) {
        const int k = tid >> 1;
        ranges[b * 2 * kPieces + tid] = (tid & 1) ? pc.len[k] : pc.start[k];
    }
    int off = 0;
    int bad_block = 0;
    const int32_t *bt_row = bt ? bt + (int64_t)b * max_blocks : nullptr;
#pragma unroll
    for (int k = 0; k < kPieces; ++k) {
        const int n = pc.len[k] < max_keep - off ? pc.len[k] : max_keep - off;
        for (int t = tid; t < n; t += blockDim.x) {
            const int32_t p = pc.start[k] + t;
            row[off + t] = bt_row ? paged_row(bt_row, max_blocks, log2_bs, p, bad_block) : p;
        }
        off += pc.len[k];
        if (off >= max_keep) break;
    }
    for (int r = pc.count + tid; r < max_keep; r += blockDim.x) row[r] = -1;
    if (bad_block) raise_device_error(MURMUR_DEVERR_BLOCK);
}

// ---------------------------------------------------------------------------
// paged_step: the block manager of a paged cache, one decode step, on the
// device.  One workgroup handles every sequence, 256 at a time: it returns to
// the free stack each still-allocated block that no step from out_len on
// retains (evicted_ranges: the speech behind the window and the outputs older
// than the window, minus sinks), then pops a block for the current token if
// its logical block has none.  Pushes and pops are placed with block-wide
// exclusive scans, so the stack stays dense and the result does not depend on
// thread timing.  A full scan frees every allocated block inside the ranges;
// otherwise only the blocks that became whole since step out_len - 1 are
// looked at (one call per step, in order).
// ---------------------------------------------------------------------------
static __device__ __forceinline__ int block_exclusive_scan(int v, int *s, int tid, int &total) {
    s[tid] = v;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int t = tid >= off ? s[tid - off] : 0;
        __syncthreads();
        s[tid] += t;
        __syncthreads();
    }
    total = s[255];
    const int excl = s[tid] - v;
    __syncthreads();
    return excl;
}

// One sequence's view for paged_step: whether its layout and policy are
// valid, the logical block of its current token, and the logical blocks
// [lo[k], hi[k]) to look at for freeing in the speech (k = 0) and output
// (k = 1) ranges: the whole ranges with a full scan, else from the previous
// step's last whole block on (a range's start stays put while it is not
// empty, and its end only grows).  Blocks past the table are clipped.
struct PagedSeq {
    bool valid;
    int32_t cur;
    int32_t lo[2], hi[2];
};

static __device__ __forceinline__ PagedSeq paged_seq(const murmur_seg *seg, const murmur_policy *pol,
                                                     int32_t pol_per_seq, int b, int B, int32_t max_blocks,
                                                     int32_t log2_bs, int32_t full_scan, int &err) {
    PagedSeq q{false, 0, {0, 0}, {0, 0}};
    if (b >= B) return q;
    const murmur_seg sq = seg[b];
    const murmur_policy p = pol[pol_per_seq ? b : 0];
    int32_t ranges[2][2], before[2][2] = {{0, 0}, {0, 0}};
    if (evicted_ranges(sq.prompt_pre, sq.speech_len, sq.prompt_mid, sq.out_len, p.speech_window, p.speech_delay,
                       p.speech_sink, p.out_window, p.out_sink, ranges[0], ranges[1]) != 0) {
        err |= MURMUR_DEVERR_POLICY;
        return q;
    }
    if (!full_scan && sq.out_len > 1)
        evicted_ranges(sq.prompt_pre, sq.speech_len, sq.prompt_mid, sq.out_len - 1, p.speech_window, p.speech_delay,
                       p.speech_sink, p.out_window, p.out_sink, before[0], before[1]);
    q.valid = true;
    const int64_t len = (int64_t)sq.prompt_pre + sq.speech_len + sq.prompt_mid + sq.out_len;
    q.cur = (int32_t)((len - 1) >> log2_bs);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        int64_t first = ((int64_t)ranges[k][0] + (1 << log2_bs) - 1) >> log2_bs;
        const int64_t end = ((int64_t)ranges[k][0] + ranges[k][1]) >> log2_bs;
        if (!full_scan && before[k][1] > 0) {
            const int64_t end_before = ((int64_t)before[k][0] + before[k][1]) >> log2_bs;
            if (end_before > first) first = end_before;
        }
        q.lo[k] = (int32_t)first;
        q.hi[k] = (int32_t)(end < max_blocks ? end : max_blocks);
    }
    return q;
}

// Two passes over the sequences, 256 at a time: every push first, then every
// pop, both in sequence order, so a step's allocations can use any block freed
// in that step.
__global__ __launch_bounds__(256) void paged_step_kernel(const murmur_seg *__restrict__ seg,
                                                         const murmur_policy *__restrict__ pol, int32_t pol_per_seq,
                                                         int32_t B, int32_t *__restrict__ bt, int32_t max_blocks,
                                                         int32_t log2_bs, int32_t *__restrict__ stack,
                                                         int32_t *__restrict__ top, int32_t capacity,
                                                         int32_t full_scan) {
    __shared__ int s_scan[256];
    __shared__ int s_top;
    const int tid = threadIdx.x;
    if (tid == 0) s_top = *top;
    __syncthreads();
    int err = 0;
    for (int b0 = 0; b0 < B; b0 += 256) {  // frees
        const int b = b0 + tid;
        const PagedSeq q = paged_seq(seg, pol, pol_per_seq, b, B, max_blocks, log2_bs, full_scan, err);
        int32_t *row = bt + (int64_t)(q.valid ? b : 0) * max_blocks;
        int npush = 0;
#pragma unroll
        for (int k = 0; k < 2; ++k)
            for (int32_t blk = q.lo[k]; blk < q.hi[k]; ++blk) npush += row[blk] >= 0;
        int pushed;
        int at = s_top + block_exclusive_scan(npush, s_scan, tid, pushed);
#pragma unroll
        for (int k = 0; k < 2; ++k)
            for (int32_t blk = q.lo[k]; blk < q.hi[k]; ++blk) {
                const int32_t phys = row[blk];
                if (phys < 0) continue;
                if (at < capacity) stack[at] = phys;
                else err |= MURMUR_DEVERR_POOL;
                ++at;
                row[blk] = -1;
            }
        __syncthreads();  // every thread has read s_top
        if (tid == 0) s_top = s_top + pushed < capacity ? s_top + pushed : capacity;
        __syncthreads();
    }
    for (int b0 = 0; b0 < B; b0 += 256) {  // allocations
        const int b = b0 + tid;
        int no_err = 0;  // the first pass has reported invalid sequences
        const PagedSeq q = paged_seq(seg, pol, pol_per_seq, b, B, max_blocks, log2_bs, 1, no_err);
        int32_t *row = bt + (int64_t)(q.valid ? b : 0) * max_blocks;
        if (q.valid && q.cur >= max_blocks) err |= MURMUR_DEVERR_BLOCK;
        const int need = q.valid && q.cur < max_blocks && row[q.cur] < 0;
        int taken;
        const int off = block_exclusive_scan(need, s_scan, tid, taken);
        if (need) {
            const int from = s_top - 1 - off;
            if (from >= 0) row[q.cur] = stack[from];
            else err |= MURMUR_DEVERR_POOL;
        }
        __syncthreads();  // every thread has read s_top and the stack
        if (tid == 0) s_top = s_top - taken > 0 ? s_top - taken : 0;
        __syncthreads();
    }
    if (tid == 0) *top = s_top;
    if (err) raise_device_error(err);
}

// The current token's K and V rows (256 bytes each per layer and KV head) into
// the pool row its block table gives; 16 bytes per thread.  A sequence whose
// block is missing (an error paged_step has reported) or whose row lies
// outside the pool is skipped.
__global__ __launch_bounds__(256) void paged_append_kernel(const murmur_seg *__restrict__ seg, int32_t B,
                                                           const int32_t *__restrict__ bt, int32_t max_blocks,
                                                           int32_t log2_bs, uint16_t *__restrict__ k,
                                                           uint16_t *__restrict__ v, int64_t s_layer, int64_t s_h,
                                                           int64_t s_pos, int64_t rows,
                                                           const uint16_t *__restrict__ k_new,
                                                           const uint16_t *__restrict__ v_new, int32_t NL,
                                                           int32_t Hkv) {
    const int64_t items = (int64_t)B * NL * Hkv * 2 * 16;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < items; i += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(i & 15);
        int64_t r = i >> 4;
        const int is_v = (int)(r & 1);
        r >>= 1;
        const int h = (int)(r % Hkv);
        r /= Hkv;
        const int layer = (int)(r % NL);
        const int b = (int)(r / NL);
        const murmur_seg sq = seg[b];
        const int64_t p = (int64_t)sq.prompt_pre + sq.speech_len + sq.prompt_mid + sq.out_len - 1;
        const int64_t blk = p >> log2_bs;
        if (p < 0 || blk >= max_blocks) continue;
        const int32_t phys = bt[(int64_t)b * max_blocks + blk];
        if (phys < 0) continue;
        const int64_t prow = ((int64_t)phys << log2_bs) | (p & ((1 << log2_bs) - 1));
        if (prow >= rows) continue;
        const uint16_t *src = (is_v ? v_new : k_new) + (((int64_t)layer * B + b) * Hkv + h) * kHeadDim + 8 * c;
        uint16_t *dst = (is_v ? v : k) + layer * s_layer + h * s_h + prow * s_pos + 8 * c;
        *reinterpret_cast<u32x4 *>(dst) = *reinterpret_cast<const u32x4 *>(src);
    }
}

// ---------------------------------------------------------------------------
// decode_attn helpers
// ---------------------------------------------------------------------------
static __device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

static __device__ __forceinline__ u32x4 load16(const uint16_t *p) { return *reinterpret_cast<const u32x4 *>(p); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two fp32 values -> packed bf16 pair (x in the low half), round to nearest
// even: one v_cvt_pk_bf16_f32 on gfx950.
static __device__ __forceinline__ uint32_t pack_bf16(float x, float y) {
    const bf16x2 v = {(__bf16)x, (__bf16)y};
    return __builtin_bit_cast(uint32_t, v);
}

constexpr float kNegInf = -__builtin_huge_valf();

// Device-coherent accesses for the split partials: raw buffer loads and stores
// with the sc1 cache-policy bit, which bypass the per-XCD L2's non-coherent
// copies, so the partials need no L2 writeback or invalidate (the
// __threadfence() route costs a full L2 write-back per wavefront).  The buffer
// resource's byte count also bounds every access in hardware.
constexpr int kCoherent = 16;  // sc1
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
static __device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, 0x00020000);
}
static __device__ __forceinline__ void store_coherent4(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kCoherent);
}
static __device__ __forceinline__ void store_coherent1(__amdgpu_buffer_rsrc_t r, uint32_t off, float x) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), r, off, 0, kCoherent);
}
static __device__ __forceinline__ f32x4 load_coherent4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCoherent));
}
static __device__ __forceinline__ float load_coherent1(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kCoherent));
}
// The same with a scalar byte offset added to the vector one (the split slot
// of a partial, so that the loads of all slots share one vector offset).
static __device__ __forceinline__ f32x4 load_coherent4_s(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t soff) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, kCoherent));
}
static __device__ __forceinline__ float load_coherent1_s(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, soff, kCoherent));
}
// Wait until every vector-memory access of this wavefront has completed; also a
// compiler barrier, so no store is moved past it.
static __device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Reductions over the four lanes n16 + 16*c4 (c4 = 0..3) that share a head
// column, with the gfx950 lane-swap instructions: after
// v_permlane16_swap(a, b) with a == b on entry, {a, b} holds {x[l], x[l^16]}
// in every lane l; v_permlane32_swap likewise pairs lane l with l^32.  Pure
// VALU, no LDS round trip.  Written as inline assembly: the compiler's own
// builtins for these instructions fold the two results of a swap into one
// when both feed a commutative operation.  The s_nop pairs cover the wait
// states these instructions need around VALU writes and reads of their
// operands.
static __device__ __forceinline__ void swap16(uint32_t &a, uint32_t &b) {
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
static __device__ __forceinline__ void swap32(uint32_t &a, uint32_t &b) {
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
static __device__ __forceinline__ float max_over_c4(float x) {
    uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
    swap16(a, b);
    x = fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
    a = b = __builtin_bit_cast(uint32_t, x);
    swap32(a, b);
    return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
static __device__ __forceinline__ float sum_over_c4(float x) {
    uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
    swap16(a, b);
    x = __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
    a = b = __builtin_bit_cast(uint32_t, x);
    swap32(a, b);
    return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

// Running softmax state of one wavefront for one (layer, sequence, KV head):
// lane (head n16, c4) holds the max (log2 units) and sum of head n16; acc holds
// O rows 4*c4 + i (heads) at head dims 16*db + n16.
struct WaveAcc {
    float m_run, l_run;
    f32x4 acc[8];
    int bad_pos;
};

static __device__ __forceinline__ void wave_acc_reset(WaveAcc &w) {
    w.m_run = kNegInf;
    w.l_run = 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) w.acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    w.bad_pos = 0;
}

// Q^T as the MFMA B operand: lane (head n16, k-group c4) holds head dims
// kc*32 + 8*c4 .. +8 for kc = 0..3.  Lanes past the group read the group's
// last head, so every lane loads (no branch around the loads); their logits
// fill S^T columns of no head of the group, which are never stored.
static __device__ __forceinline__ void load_q(u32x4 (&qf)[4], const uint16_t *q, int64_t row_of_head0, int G,
                                              int n16, int c4) {
    const int hq = n16 < G ? n16 : G - 1;
    const uint16_t *qrow = q + (row_of_head0 + hq) * kHeadDim + 8 * c4;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) qf[kc] = load16(qrow + kc * 32);
}

// The six-piece range table in cumulative form: rank r belongs to the last
// piece k with r >= lo[k] (empty pieces are passed over by the next one) and
// sits at position r + off[k].
struct RangeTab {
    int32_t lo[kPieces];
    int32_t off[kPieces];
};

static __device__ __forceinline__ RangeTab make_tab(const int32_t (&rg)[2 * kPieces]) {
    RangeTab t;
    int32_t acc = 0;
#pragma unroll
    for (int k = 0; k < kPieces; ++k) {
        t.lo[k] = acc;
        t.off[k] = rg[2 * k] - acc;
        acc += rg[2 * k + 1];
    }
    return t;
}

// Position of rank r, and its piece, by a select chain (no branches).
static __device__ __forceinline__ int tab_pos(const RangeTab &t, int r, int &piece) {
    int p = r + t.off[0];
    piece = 0;
#pragma unroll
    for (int k = 1; k < kPieces; ++k) {
        const bool in = r >= t.lo[k];
        p = in ? r + t.off[k] : p;
        piece = in ? k : piece;
    }
    return p;
}

// The current token in ring storage: rows at position `cur` are read from
// the K/V passed with the call instead of the cache, whose row `cur` this
// launch overwrites (kRing only; otherwise cur is never compared).
struct NewRows {
    int32_t cur;
    const uint16_t *k;
    const uint16_t *v;
};

// Forces uniform values into scalar registers at this point: the scalar loads
// they come from are then issued together, ahead of one wait, instead of
// being sunk to their first use behind earlier waits.
template <typename T>
static __device__ __forceinline__ void materialize_one(const T &x) {
    asm volatile("" ::"s"(x));
}
template <typename... T>
static __device__ __forceinline__ void materialize(const T &...x) {
    (materialize_one(x), ...);
}


// Softmax update of one pass from its S^T tile (lane (head n16, c4), register
// i of block blk: logit of rank 16*blk + 4*c4 + i of the pass): masks ranks
// at or past `valid`, folds the pass into the running (max, sum) and rescales
// O, and returns P as the A operand of O = P V in k order (4*c4 + 0..3,
// 16 + 4*c4 + 0..3), split into bf16 hi + lo so that hi + lo carries ~16
// mantissa bits.  kOnline: fold into a running state; otherwise the state is
// known to be empty.
template <bool kOnline>
static __device__ __forceinline__ void softmax_step(const f32x4 (&s)[2], int valid, float scale_log2, WaveAcc &w,
                                                    int c4, u32x4 &p_hi, u32x4 &p_lo) {
    // Logits in log2 units; ranks past `valid` are masked (a partial pass).
    float x[2][4];
    const bool partial = valid < kWaveTile;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[blk][i] = s[blk][i] * scale_log2;
            if (partial && 16 * blk + 4 * c4 + i >= valid) x[blk][i] = kNegInf;
        }
    float tmax = fmaxf(fmaxf(fmaxf(x[0][0], x[0][1]), fmaxf(x[0][2], x[0][3])),
                       fmaxf(fmaxf(x[1][0], x[1][1]), fmaxf(x[1][2], x[1][3])));
    tmax = max_over_c4(tmax);
    const float m_new = kOnline ? fmaxf(w.m_run, tmax) : tmax;  // finite: rank 0 of the pass is valid
    float psum = 0.f;
    float pr[2][4];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            pr[blk][i] = __builtin_amdgcn_exp2f(x[blk][i] - m_new);  // in [0, 1]
            psum += pr[blk][i];
        }
    psum = sum_over_c4(psum);
    if (kOnline) {
        const float alpha = __builtin_amdgcn_exp2f(w.m_run - m_new);  // 0 while the state is empty
        w.l_run = w.l_run * alpha + psum;
        // Rescale O rows: row 4*c4 + i belongs to head 4*c4 + i.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float ai = __shfl(alpha, 4 * c4 + i);
#pragma unroll
            for (int db = 0; db < 8; ++db) w.acc[db][i] *= ai;
        }
    } else {
        w.l_run = psum;
    }
    w.m_run = m_new;
#pragma unroll
    for (int wd = 0; wd < 4; ++wd) {
        const int blk = wd >> 1, i0 = (wd & 1) * 2;
        const float e0 = pr[blk][i0], e1 = pr[blk][i0 + 1];
        const uint32_t hi = pack_bf16(e0, e1);
        p_hi[wd] = hi;
        p_lo[wd] = pack_bf16(e0 - __builtin_bit_cast(float, hi << 16), e1 - __builtin_bit_cast(float, hi & 0xffff0000u));
    }
}

// ---------------------------------------------------------------------------
// LDS-staged passes.  K and V rows go from HBM straight into LDS with gfx950's
// direct-to-LDS loads (no registers hold data in flight, so a wavefront can
// keep a whole pass loading while it computes the previous one), the MFMA K
// operands come back with ds_read_b128 and the V operands with the
// transposing ds_read_b64_tr_b16, which needs no VALU transpose.
//
// Tile of one pass (K or V): 32 rows of 256 bytes; 16-byte chunk c of row r
// sits at slot c ^ (r & 15), which keeps both operand reads bank-conflict
// free.  A direct-to-LDS load writes lane l's 16 bytes at base + 16*l, so load
// j (0..7) fills rows 4j .. 4j+3 and lane l fetches chunk (l & 15) ^ (row & 15)
// of row 4j + (l >> 4).
//
// The LDS reads run in inline assembly that ends with its own lgkmcnt wait
// (outputs early-clobber: a read's result may land before a later read of the
// same block has taken its address):
// the compiler's wait insertion assumes any LDS read may depend on every
// direct-to-LDS load in flight and would drain the pipeline; the waits for
// the loads are placed by hand instead (wait_vm), counting only loads issued
// by this wavefront after the ones awaited, so a wait can be longer than
// needed but never shorter.
// ---------------------------------------------------------------------------
constexpr int kTileRowBytes = kHeadDim * 2;            // 256
constexpr int kTileBytes = kWaveTile * kTileRowBytes;  // 8 KiB
constexpr int kStageBytes = 2 * kTileBytes;            // K tile, then V tile
constexpr int kIdxSlotBytes = 256;                     // index entries of one pass (32 of 64 words used)
constexpr int kStageLoads = 16;                        // direct-to-LDS loads of one pass (dma_pass)

typedef __attribute__((address_space(3))) void lds_void_t;

static __device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
}

template <int N>
static __device__ __forceinline__ void wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// The 16 direct-to-LDS loads of one pass (8 for K, then 8 for V) into `stage`.
// pos[j]: in-bounds position of the row whose rank is r0 + 4j + (lane >> 4).
// ring: compare positions with nr.cur (a constant at every call site).
static __device__ __forceinline__ void dma_pass(uint8_t *stage, const uint16_t *kbase, const uint16_t *vbase,
                                                int64_t s_pos, const int32_t (&pos)[8], int lane, bool ring,
                                                const NewRows &nr) {
    const int q = lane >> 4, sl = lane & 15;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int c = sl ^ ((4 * j + q) & 15);
        const uint16_t *kr = kbase + (int64_t)pos[j] * s_pos;
        __builtin_amdgcn_global_load_lds((ring && pos[j] == nr.cur ? nr.k : kr) + 8 * c,
                                         (lds_void_t *)(stage + j * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int c = sl ^ ((4 * j + q) & 15);
        const uint16_t *vr = vbase + (int64_t)pos[j] * s_pos;
        __builtin_amdgcn_global_load_lds((ring && pos[j] == nr.cur ? nr.v : vr) + 8 * c,
                                         (lds_void_t *)(stage + kTileBytes + j * 1024), 16, 0, 0);
    }
}

// Positions for dma_pass from the range table.  Ranks at or past r_end read
// the row of rank r0 (their logits are masked and their weights are exactly
// zero); a retained rank outside [0, max_len) sets `bad` and reads a clamped
// row.  When the pass lies in one piece (the common case; the test is uniform
// over the wavefront) the rows are consecutive.
static __device__ __forceinline__ void dma_pos_ranges(const RangeTab &t, int r0, int r_end, int max_len, int q,
                                                      int32_t (&pos)[8], int &bad) {
    const int valid = min(kWaveTile, r_end - r0);
    int pc0, pcl;
    const int p0 = tab_pos(t, r0, pc0);
    const int pl = tab_pos(t, r0 + valid - 1, pcl);
    const bool p0ok = (uint32_t)p0 < (uint32_t)max_len;
    if (pc0 == pcl && p0ok && pl < max_len) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int d = 4 * j + q;
            pos[j] = p0 + (d < valid ? d : 0);
        }
    } else {
        const int fb = p0ok ? p0 : 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int r = r0 + 4 * j + q;
            int pc;
            const int p = tab_pos(t, r, pc);
            const bool live = r < r_end, inb = (uint32_t)p < (uint32_t)max_len;
            bad |= live && !inb;
            pos[j] = live && inb ? p : fb;
        }
    }
}

// Whether the ranks r0 .. r0+valid-1 of a pass lie in one piece of the range
// table, and if so the position p0 of rank r0: the pass then reads the
// consecutive rows p0 .. p0+valid-1, all inside [0, max_len).  One piece: no piece starts at a rank in
// (r0, r0+valid-1], so every rank of the pass has the piece of r0 (the last k
// with rank >= lo[k]), whatever the table.  Every argument is uniform over the
// wavefront, so the test is scalar code.
static __device__ __forceinline__ bool tab_run(const RangeTab &t, int r0, int valid, int max_len, int &p0) {
    // (readfirstlane: the entries stay separate scalars; a select chain over the
    // table's fields could otherwise become an indexed load of a copy of it)
    int p = r0 + __builtin_amdgcn_readfirstlane(t.off[0]);
    uint32_t first_in = 0xffffffffu;  // min over pieces k >= 1 of lo[k] - r0 - 1 (unsigned)
#pragma unroll
    for (int k = 1; k < kPieces; ++k) {
        const int lo = __builtin_amdgcn_readfirstlane(t.lo[k]), off = __builtin_amdgcn_readfirstlane(t.off[k]);
        p = r0 >= lo ? r0 + off : p;
        first_in = min(first_in, (uint32_t)(lo - r0 - 1));
    }
    p0 = p;
    // lo[k] in (r0, r0 + valid - 1] exactly when lo[k] - r0 - 1 < valid - 1 unsigned
    return first_in >= (uint32_t)(valid - 1) && p >= 0 && p <= max_len - valid;
}

// dma_pass for a pass whose rows are consecutive (tab_run): the loads take the
// wavefront's first K (V) row as a scalar base and a 32-bit offset per lane,
// one offset per row shared by K and V, so issuing them costs one vector add
// each instead of a 64-bit address computation.  Ranks at or past `valid`
// read row p0, as in dma_pos_ranges.  Lane (q, sl) of load j reads chunk
// sl ^ ((4j + q) & 15) of row 4j + q, as in dma_pass; that chunk's byte
// offset 16 * (sl ^ q) ^ 64 * (j & 3) repeats with period 4 in j.
template <bool kFull>
static __device__ __forceinline__ void dma_pass_run(uint8_t *stage, const uint16_t *kbase, const uint16_t *vbase,
                                                    int64_t s_pos, int p0, int valid, int lane) {
    const int q = lane >> 4, sl = lane & 15;
    const uint32_t row_bytes = (uint32_t)s_pos * 2u;
    const uint8_t *kb = reinterpret_cast<const uint8_t *>(kbase + (int64_t)p0 * s_pos);
    const uint8_t *vb = reinterpret_cast<const uint8_t *>(vbase + (int64_t)p0 * s_pos);
    const uint32_t qrow = (uint32_t)q * row_bytes, chunk = (uint32_t)(sl ^ q) * 16u;
    uint32_t voff[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t row = qrow + (uint32_t)(4 * j) * row_bytes;
        const uint32_t c = chunk ^ (64u * (uint32_t)(j & 3));
        voff[j] = (kFull || 4 * j + q < valid ? row : 0u) + c;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
        __builtin_amdgcn_global_load_lds(kb + voff[j], (lds_void_t *)(stage + j * 1024), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < 8; ++j)
        __builtin_amdgcn_global_load_lds(vb + voff[j], (lds_void_t *)(stage + kTileBytes + j * 1024), 16, 0, 0);
    // Ends the path with a statement of its own: the compiler would otherwise
    // sink the last load of this and dma_pass's path into one shared block,
    // which takes a 64-bit address.
    asm volatile("" ::: "memory");
}

// The 16 K/V loads of the pass at ranks r0 .. min(r0 + kWaveTile, r_end) - 1
// from the range table: consecutive rows through dma_pass_run (tab_run; not
// for ring storage, whose current row comes from another buffer), else
// per-row positions through dma_pass.  short_rows: stride_pos < kRunRowLimit.
template <bool kRing>
static __device__ __forceinline__ void dma_pass_ranges(uint8_t *stage, const RangeTab &tab, int r0, int r_end,
                                                       int max_len, bool short_rows, const uint16_t *kbase,
                                                       const uint16_t *vbase, int64_t s_pos, int lane, int c4,
                                                       int &bad, const NewRows &nr) {
    const int valid = min(kWaveTile, r_end - r0);
    int p0;
    if (!kRing && short_rows && tab_run(tab, r0, valid, max_len, p0)) {
        if (valid == kWaveTile)
            dma_pass_run<true>(stage, kbase, vbase, s_pos, p0, valid, lane);
        else
            dma_pass_run<false>(stage, kbase, vbase, s_pos, p0, valid, lane);
    } else {
        int32_t pos[8];
        dma_pos_ranges(tab, r0, r_end, max_len, c4, pos, bad);
        dma_pass(stage, kbase, vbase, s_pos, pos, lane, kRing, nr);
    }
}

// Index entries of one pass into an LDS slot with one direct-to-LDS load:
// word 8q + j holds the entry of rank r0 + 4j + q (q = 0..3, j = 0..7), so a
// lane reads its eight entries as two 16-byte words.  The buffer resource
// spans the row's count; lanes past it (and lanes 32..63) read zeros.
static __device__ __forceinline__ void dma_idx(uint8_t *slot, __amdgpu_buffer_rsrc_t irow, int r0, int lane) {
    const uint32_t voff = lane < 32 ? (uint32_t)(r0 + (lane & 7) * 4 + (lane >> 3)) * 4u : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(irow, (lds_void_t *)slot, 4, voff, 0, 0, 0);
}

static __device__ __forceinline__ void dma_pos_index(const uint8_t *slot, int r0, int r_end, int max_len, int q,
                                                     int32_t (&pos)[8], int &bad) {
    u32x4 e0, e1;
    uint32_t w0;
    asm volatile("ds_read_b128 %0, %3\n\tds_read_b128 %1, %3 offset:16\n\tds_read_b32 %2, %4\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(e0), "=&v"(e1), "=&v"(w0)
                 : "v"(lds_addr(slot) + 32u * q), "v"(lds_addr(slot))
                 : "memory");
    const int p0 = (int)w0;  // entry of rank r0
    const int fb = (uint32_t)p0 < (uint32_t)max_len ? p0 : 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int r = r0 + 4 * j + q;
        const int p = (int)(j < 4 ? e0[j] : e1[j - 4]);
        const bool live = r < r_end, inb = (uint32_t)p < (uint32_t)max_len;
        bad |= live && !inb;
        pos[j] = live && inb ? p : fb;
    }
}

// One pass from an LDS stage: operand reads, S^T = K Q^T, softmax update,
// O += P V.  kWaitDma: the stage's direct-to-LDS loads (dma_pass: the K tile's,
// then the V tile's, the last loads this wavefront issued) may still be in
// flight; the K operands are read once the K loads are in, and S^T and the
// softmax are computed while the V loads land.
template <bool kOnline, bool kWaitDma = false>
static __device__ __forceinline__ void compute_pass_lds(const uint8_t *stage, const u32x4 (&qf)[4], int valid,
                                                        float scale_log2, WaveAcc &w, int n16, int c4) {
    const uint32_t kt = lds_addr(stage), vt = kt + kTileBytes;
    // K operand (blk, kc): row 16*blk + n16, chunk 4*kc + c4 (row & 15 == n16);
    // blk 1 is 16 rows (4096 bytes) further.
    uint32_t ka[4];
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) ka[kc] = kt + n16 * kTileRowBytes + (((4 * kc + c4) ^ n16) << 4);
    // V operand (db, h) of lane (i = n16, c4): row 16*h + 4*c4 + i/4, head dims
    // 16*db + 4*(i%4) .. +3, i.e. chunk 2*db + (i%4)/2, half i & 1; the row's
    // low four bits are 4*c4 + i/4 for both h (h = 1 is 4096 bytes further).
    const int vr = 4 * c4 + (n16 >> 2);
    uint32_t va[8];
#pragma unroll
    for (int db = 0; db < 8; ++db)
        va[db] = vt + vr * kTileRowBytes + (((2 * db + ((n16 & 3) >> 1)) ^ vr) << 4) + (n16 & 1) * 8;
    u32x4 kf[8];
    u32x2 vf[16];
    if constexpr (!kWaitDma) {
        asm volatile(
            "ds_read_b128 %0, %24\n\t"
            "ds_read_b128 %1, %25\n\t"
            "ds_read_b128 %2, %26\n\t"
            "ds_read_b128 %3, %27\n\t"
            "ds_read_b128 %4, %24 offset:4096\n\t"
            "ds_read_b128 %5, %25 offset:4096\n\t"
            "ds_read_b128 %6, %26 offset:4096\n\t"
            "ds_read_b128 %7, %27 offset:4096\n\t"
            "ds_read_b64_tr_b16 %8, %28\n\t"
            "ds_read_b64_tr_b16 %9, %28 offset:4096\n\t"
            "ds_read_b64_tr_b16 %10, %29\n\t"
            "ds_read_b64_tr_b16 %11, %29 offset:4096\n\t"
            "ds_read_b64_tr_b16 %12, %30\n\t"
            "ds_read_b64_tr_b16 %13, %30 offset:4096\n\t"
            "ds_read_b64_tr_b16 %14, %31\n\t"
            "ds_read_b64_tr_b16 %15, %31 offset:4096\n\t"
            "ds_read_b64_tr_b16 %16, %32\n\t"
            "ds_read_b64_tr_b16 %17, %32 offset:4096\n\t"
            "ds_read_b64_tr_b16 %18, %33\n\t"
            "ds_read_b64_tr_b16 %19, %33 offset:4096\n\t"
            "ds_read_b64_tr_b16 %20, %34\n\t"
            "ds_read_b64_tr_b16 %21, %34 offset:4096\n\t"
            "ds_read_b64_tr_b16 %22, %35\n\t"
            "ds_read_b64_tr_b16 %23, %35 offset:4096\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(kf[0]), "=&v"(kf[1]), "=&v"(kf[2]), "=&v"(kf[3]), "=&v"(kf[4]), "=&v"(kf[5]), "=&v"(kf[6]), "=&v"(kf[7]),
              "=&v"(vf[0]), "=&v"(vf[1]), "=&v"(vf[2]), "=&v"(vf[3]), "=&v"(vf[4]), "=&v"(vf[5]), "=&v"(vf[6]), "=&v"(vf[7]),
              "=&v"(vf[8]), "=&v"(vf[9]), "=&v"(vf[10]), "=&v"(vf[11]), "=&v"(vf[12]), "=&v"(vf[13]), "=&v"(vf[14]),
              "=&v"(vf[15])
            : "v"(ka[0]), "v"(ka[1]), "v"(ka[2]), "v"(ka[3]), "v"(va[0]), "v"(va[1]), "v"(va[2]), "v"(va[3]), "v"(va[4]),
              "v"(va[5]), "v"(va[6]), "v"(va[7])
            : "memory");
    } else {
        wait_vm<kStageLoads / 2>();  // the K tile's loads (issued before the V tile's)
        asm volatile(
            "ds_read_b128 %0, %8\n\t"
            "ds_read_b128 %1, %9\n\t"
            "ds_read_b128 %2, %10\n\t"
            "ds_read_b128 %3, %11\n\t"
            "ds_read_b128 %4, %8 offset:4096\n\t"
            "ds_read_b128 %5, %9 offset:4096\n\t"
            "ds_read_b128 %6, %10 offset:4096\n\t"
            "ds_read_b128 %7, %11 offset:4096\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(kf[0]), "=&v"(kf[1]), "=&v"(kf[2]), "=&v"(kf[3]), "=&v"(kf[4]), "=&v"(kf[5]), "=&v"(kf[6]),
              "=&v"(kf[7])
            : "v"(ka[0]), "v"(ka[1]), "v"(ka[2]), "v"(ka[3])
            : "memory");
    }
    f32x4 s[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
        s[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) s[blk] = mfma16x16x32(kf[4 * blk + kc], qf[kc], s[blk]);
    }
    u32x4 p_hi, p_lo;
    softmax_step<kOnline>(s, valid, scale_log2, w, c4, p_hi, p_lo);
    if constexpr (kWaitDma) {
        wait_vm<0>();  // the V tile's loads
        asm volatile(
            "ds_read_b64_tr_b16 %0, %16\n\t"
            "ds_read_b64_tr_b16 %1, %16 offset:4096\n\t"
            "ds_read_b64_tr_b16 %2, %17\n\t"
            "ds_read_b64_tr_b16 %3, %17 offset:4096\n\t"
            "ds_read_b64_tr_b16 %4, %18\n\t"
            "ds_read_b64_tr_b16 %5, %18 offset:4096\n\t"
            "ds_read_b64_tr_b16 %6, %19\n\t"
            "ds_read_b64_tr_b16 %7, %19 offset:4096\n\t"
            "ds_read_b64_tr_b16 %8, %20\n\t"
            "ds_read_b64_tr_b16 %9, %20 offset:4096\n\t"
            "ds_read_b64_tr_b16 %10, %21\n\t"
            "ds_read_b64_tr_b16 %11, %21 offset:4096\n\t"
            "ds_read_b64_tr_b16 %12, %22\n\t"
            "ds_read_b64_tr_b16 %13, %22 offset:4096\n\t"
            "ds_read_b64_tr_b16 %14, %23\n\t"
            "ds_read_b64_tr_b16 %15, %23 offset:4096\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(vf[0]), "=&v"(vf[1]), "=&v"(vf[2]), "=&v"(vf[3]), "=&v"(vf[4]), "=&v"(vf[5]), "=&v"(vf[6]),
              "=&v"(vf[7]), "=&v"(vf[8]), "=&v"(vf[9]), "=&v"(vf[10]), "=&v"(vf[11]), "=&v"(vf[12]), "=&v"(vf[13]),
              "=&v"(vf[14]), "=&v"(vf[15])
            : "v"(va[0]), "v"(va[1]), "v"(va[2]), "v"(va[3]), "v"(va[4]), "v"(va[5]), "v"(va[6]), "v"(va[7])
            : "memory");
    }
    // B operand of head dims 16*db .. +15: positions 4*c4 .. +3 (h = 0) and
    // 16 + 4*c4 .. +3 (h = 1), the k order of P.
#pragma unroll
    for (int db = 0; db < 8; ++db) {
        const u32x4 bv = u32x4{vf[2 * db][0], vf[2 * db][1], vf[2 * db + 1][0], vf[2 * db + 1][1]};
        w.acc[db] = mfma16x16x32(p_hi, bv, w.acc[db]);
        w.acc[db] = mfma16x16x32(p_lo, bv, w.acc[db]);
    }
}

// ---------------------------------------------------------------------------
// Where the retained set of a sequence comes from.  kSrcIndex: counts and the
// index list; kSrcRanges: counts and the six-piece range table; kSrcLayout
// (the fused decode step): the layouts and policies themselves, the pieces
// computed in closed form by every workgroup that needs them, and the
// evict_compact outputs written by one workgroup per sequence.
// ---------------------------------------------------------------------------
// Row of the policy array that applies to (layer, sequence b): the array is
// [per layer ? NL : 1][per sequence ? B : 1] policies (MURMUR_POL_* bits).
static __device__ __forceinline__ int policy_row(int32_t pol_mode, int layer, int b, int B) {
    const int per_seq = pol_mode & MURMUR_POL_PER_SEQ;
    return ((pol_mode & MURMUR_POL_PER_LAYER) ? layer * (per_seq ? B : 1) : 0) + (per_seq ? b : 0);
}

// Count of sequence b and, unless kSrcIndex, its range table.  p0/p1: counts
// (kSrcIndex) or range tables (kSrcRanges, the count being the table's total
// length), or (kSrcLayout, kSrcRing) layouts (murmur_seg [B]) and policies
// (murmur_policy rows, see policy_row).  kSrcRing gives the pieces in ring-storage rows
// of ring_cap output slots and the row of the current token in `cur`.  An
// invalid layout or policy gives count 0 and sets policy_bad to 1 (2: the
// ring cannot hold the retained outputs).
// The few words a workgroup needs to find its sequence's retained set are
// fetched with one vector load (lane k reads the word at its own address) and
// made wavefront-uniform with readlane.  Scalar loads would share their wait
// counter with the scalar loads of the launch description, and a scalar wait
// cannot be partial: the compiler's first wait for a launch field would then
// put a second memory round trip in front of the first K/V loads.  Vector
// loads have a counter of their own, so both round trips overlap.  seq_words
// issues the load, seq_count_from uses its result: in between, the caller pins
// the launch fields it needs.
static __device__ __forceinline__ int32_t word_of_lane(const int32_t *addr) { return *addr; }

// 0 in a vector register the compiler cannot see through: an address offset by
// it stays a per-lane address, so its load stays a vector load.
static __device__ __forceinline__ int opaque_lane_zero() {
    int z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    return z;
}

// Words of sequence b (see seq_count_from): kSrcLayout / kSrcRing: lanes 0-3
// its layout, lanes 4-8 its policy; kSrcRanges: lanes 0-11 its range table;
// kSrcIndex: its count.
template <int kSrc>
static __device__ __forceinline__ int32_t seq_words(const int32_t *p0, const int32_t *p1, int b, int32_t pol_mode,
                                                    int layer, int B) {
    const int lane = threadIdx.x & 63;
    if (kSrc == kSrcLayout || kSrc == kSrcRing) {
        const int32_t *sg = p0 + 4 * b;
        const int32_t *pl = p1 + 5 * policy_row(pol_mode, layer, b, B);
        return word_of_lane(lane < 4 ? sg + lane : (lane < 9 ? pl + (lane - 4) : sg));
    }
    if (kSrc == kSrcRanges) return word_of_lane(p1 + b * 2 * kPieces + (lane < 2 * kPieces ? lane : 0));
    return word_of_lane(p0 + b + opaque_lane_zero());
}

// Count of sequence b and, unless kSrcIndex, its range table, from the words
// seq_words loaded.  Their sources: counts (kSrcIndex) or range tables
// (kSrcRanges, the count being the table's total length), or (kSrcLayout,
// kSrcRing) layouts (murmur_seg [B]) and policies (murmur_policy rows, see
// policy_row).  kSrcRing gives the pieces in ring-storage rows of ring_cap
// output slots and the row of the current token in `cur`; an invalid layout or
// policy gives count 0 and sets policy_bad to 1 (2: the ring cannot hold the
// retained outputs).  kSrcLayout gives the pieces without the validity test,
// whose nine input words it leaves in lw for layout_valid once the first loads
// are out (the positions read are bounded whatever the table says).
template <int kSrc>
static __device__ __forceinline__ int seq_count_from(int32_t x, int32_t ring_cap, int32_t (&rg)[2 * kPieces],
                                                     int &policy_bad, int32_t &cur, int32_t (&lw)[9]) {
    if (kSrc == kSrcLayout || kSrc == kSrcRing) {
        const int32_t s0 = __builtin_amdgcn_readlane(x, 0), s1 = __builtin_amdgcn_readlane(x, 1),
                      s2 = __builtin_amdgcn_readlane(x, 2), s3 = __builtin_amdgcn_readlane(x, 3);
        const int32_t w0 = __builtin_amdgcn_readlane(x, 4), w1 = __builtin_amdgcn_readlane(x, 5),
                      w2 = __builtin_amdgcn_readlane(x, 6), w3 = __builtin_amdgcn_readlane(x, 7),
                      w4 = __builtin_amdgcn_readlane(x, 8);
        Pieces pc;
        if (kSrc == kSrcLayout) {
            retained_pieces_unchecked(s0, s1, s2, s3, w0, w1, w2, w3, w4, &pc);
            const int32_t words[9] = {s0, s1, s2, s3, w0, w1, w2, w3, w4};
#pragma unroll
            for (int k = 0; k < 9; ++k) lw[k] = words[k];
#pragma unroll
            for (int k = 0; k < kPieces; ++k) {
                rg[2 * k] = pc.start[k];
                rg[2 * k + 1] = pc.len[k];
            }
            return pc.count;
        }
        const int rc = ring_pieces(s0, s1, s2, s3, w0, w1, w2, w3, w4, ring_cap, &pc, &cur);
        if (rc != 0) {
            policy_bad = rc == -2 ? 2 : 1;
#pragma unroll
            for (int k = 0; k < 2 * kPieces; ++k) rg[k] = 0;
            return 0;
        }
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            rg[2 * k] = pc.start[k];
            rg[2 * k + 1] = pc.len[k];
        }
        return pc.count;
    }
    if (kSrc == kSrcRanges) {  // the count is the table's total length
        int c = 0;
#pragma unroll
        for (int k = 0; k < 2 * kPieces; ++k) rg[k] = __builtin_amdgcn_readlane(x, k);
#pragma unroll
        for (int k = 0; k < kPieces; ++k) c += rg[2 * k + 1];
        return c;
    }
    return __builtin_amdgcn_readfirstlane(x);
}

// layout_valid of the words seq_count_from left, evaluated where it is called:
// the words pass through an opaque statement that also orders memory, so the
// compiler neither hoists the test in front of the loads issued before it nor
// reuses earlier work.
static __device__ __forceinline__ bool layout_valid_late(const int32_t (&lw)[9]) {
    int32_t v0 = lw[0], v1 = lw[1], v2 = lw[2], v3 = lw[3], v4 = lw[4], v5 = lw[5], v6 = lw[6], v7 = lw[7], v8 = lw[8];
    asm volatile("" : "+s"(v0), "+s"(v1), "+s"(v2), "+s"(v3), "+s"(v4), "+s"(v5), "+s"(v6), "+s"(v7), "+s"(v8)::"memory");
    return layout_valid(v0, v1, v2, v3, v4, v5, v6, v7, v8);
}

// Count of sequence b and, unless kSrcIndex, its range table, read with
// scalar loads (the LDS-staged kernel, whose other scalar loads go out in the
// same batch).  Sources as for seq_count_from.
template <int kSrc>
static __device__ __forceinline__ int seq_count_scalar(const int32_t *p0, const int32_t *p1, int b, int32_t pol_mode,
                                                int layer, int B, int32_t ring_cap, int32_t (&rg)[2 * kPieces],
                                                int &policy_bad, int32_t &cur) {
    if (kSrc == kSrcLayout || kSrc == kSrcRing) {
        const int32_t *sg = p0 + 4 * b;
        const int32_t *pl = p1 + 5 * policy_row(pol_mode, layer, b, B);
        const int32_t s0 = sg[0], s1 = sg[1], s2 = sg[2], s3 = sg[3];
        const int32_t w0 = pl[0], w1 = pl[1], w2 = pl[2], w3 = pl[3], w4 = pl[4];
        if (kSrc == kSrcRing)
            materialize(s0, s1, s2, s3, w0, w1, w2, w3, w4, ring_cap);  // one round trip
        else
            materialize(s0, s1, s2, s3, w0, w1, w2, w3, w4);  // both rows in one round trip
        Pieces pc;
        const int rc = kSrc == kSrcRing ? ring_pieces(s0, s1, s2, s3, w0, w1, w2, w3, w4, ring_cap, &pc, &cur)
                                        : retained_pieces(s0, s1, s2, s3, w0, w1, w2, w3, w4, &pc);
        if (rc != 0) {
            policy_bad = rc == -2 ? 2 : 1;
#pragma unroll
            for (int k = 0; k < 2 * kPieces; ++k) rg[k] = 0;
            return 0;
        }
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            rg[2 * k] = pc.start[k];
            rg[2 * k + 1] = pc.len[k];
        }
        return pc.count;
    }
    if (kSrc == kSrcRanges) {  // the count is the table's total length
        int c = 0;
#pragma unroll
        for (int k = 0; k < 2 * kPieces; ++k) rg[k] = p1[b * 2 * kPieces + k];
#pragma unroll
        for (int k = 0; k < kPieces; ++k) c += rg[2 * k + 1];
        return c;
    }
    return p0[b];
}

// The evict_compact outputs of sequence b (each one only if the caller passed
// its buffer) and its device errors: count (0 for an invalid layout or
// policy), range table, ascending index list padded with -1 (its first
// max_keep entries when the count exceeds max_keep).  Each caller writes the
// index-list entries of ranks [r_lo, r_hi) (the splits of a sequence share
// the list between them); the one with r_lo == 0 also writes the count, the
// table and the errors.  Block-wide.
template <int kThreads>
static __device__ __forceinline__ void write_retained(const AttnLaunch &a, int b, int cnt, int policy_bad,
                                                      const int32_t (&rg)[2 * kPieces], int max_keep, int tid,
                                                      int r_lo, int r_hi) {
    if (r_lo == 0 && tid == 0) {
        if (a.count_out) a.count_out[b] = cnt;
        if (policy_bad) raise_device_error(policy_bad == 2 ? MURMUR_DEVERR_CAPACITY : MURMUR_DEVERR_POLICY);
        else if (cnt > max_keep) raise_device_error(MURMUR_DEVERR_OVERFLOW);
    }
    if (r_lo == 0 && a.ranges_out && tid < 2 * kPieces) {
        int32_t v = 0;
#pragma unroll
        for (int k = 0; k < 2 * kPieces; ++k) v = tid == k ? rg[k] : v;
        a.ranges_out[b * 2 * kPieces + tid] = v;
    }
    if (a.idx_out) {
        int32_t *row = a.idx_out + (int64_t)b * max_keep;
        const int hi = r_hi < max_keep ? r_hi : max_keep;
        int off = 0;  // first rank of piece k
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            const int n = rg[2 * k + 1] < max_keep - off ? rg[2 * k + 1] : max_keep - off;
            const int lo = off > r_lo ? off : r_lo, e = off + n < hi ? off + n : hi;
            for (int r = lo + tid; r < e; r += kThreads) row[r] = rg[2 * k] + (r - off);
            off += n;
        }
        for (int r = (off > r_lo ? off : r_lo) + tid; r < hi; r += kThreads) row[r] = -1;
    }
}

// Ring storage: the current token's K and V rows (256 bytes each) of this
// (layer, sequence, KV head) go into its ring row `cur`, by split 0's first
// wavefront (lanes 0-15 K, 16-31 V; lanes 32-63 load the same chunks and store
// nothing), unless the layout, policy or ring is invalid or the row lies
// outside the cache.  The rows are loaded when the kernel starts and stored
// once the passes are done, so neither the load's round trip nor the store
// lengthens the workgroup.  No workgroup of this launch reads row `cur`
// (positions equal to cur read nr.k / nr.v) and the token it held is no longer
// retained, so the store may land at any time.
struct NewRowCopy {
    u32x4 x;
    bool on;
};
static __device__ __forceinline__ NewRowCopy load_new_row(const AttnLaunch &a, const NewRows &nr, int policy_bad,
                                                          int lane, bool first_wave_of_split0) {
    NewRowCopy c{{0u, 0u, 0u, 0u}, false};
    if (first_wave_of_split0) {
        const int l = lane & 31;
        c.x = load16(((l >= 16) ? nr.v : nr.k) + 8 * (l & 15));
        c.on = lane < 32 && !policy_bad && (uint32_t)nr.cur < (uint32_t)a.max_len;
    }
    return c;
}
static __device__ __forceinline__ void store_new_row(const AttnLaunch &a, const NewRowCopy &c, const NewRows &nr,
                                                     const uint16_t *kbase, const uint16_t *vbase, int lane) {
    if (!c.on) return;
    uint16_t *dst = const_cast<uint16_t *>(lane >= 16 ? vbase : kbase) + (int64_t)nr.cur * a.s_pos + 8 * (lane & 15);
    *reinterpret_cast<u32x4 *>(dst) = c.x;
}

// Workgroup barrier that also ORs a per-thread flag over the workgroup: each
// wavefront writes whether any of its lanes holds the flag into its own LDS
// slot before the barrier.  (__syncthreads_or would load the block size from
// the kernel arguments at this point: a scalar memory round trip in front of
// the barrier.)
template <int kWaves>
static __device__ __forceinline__ int barrier_or(int flag, int *s_wave_flag, int wave, int lane) {
    const int any = __ballot(flag != 0) != 0;
    if (lane == 0) s_wave_flag[wave] = any;
    __syncthreads();
    int r = 0;
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) r |= s_wave_flag[wv];
    return r;
}

// Combine of a workgroup's four wavefronts.  Each wavefront publishes its
// state -- (max, sum) per head and its unscaled O rows -- into LDS regions no
// other wavefront touches before the workgroup barrier that follows; after
// the barrier the threads writing the result rescale and add the four states
// as they read them.  One barrier and no dependent LDS round trip between.
template <int kWaves>
struct __attribute__((aligned(16))) CombineLdsT {
    float ml[kMaxGroup][kWaves][2];  // per head and wavefront: max (log2 units), sum
};
using CombineLds = CombineLdsT<kWavesPerWg>;
constexpr int kOStride = kHeadDim + 4;                  // floats per published O row (padded: conflict-free stores)
constexpr int kOWaveBytes = kMaxGroup * kOStride * 4;   // 8448: a wavefront's published rows

template <int kWaves>
static __device__ __forceinline__ void publish_wave(const WaveAcc &w, float *o_w, CombineLdsT<kWaves> &cl, int wave,
                                                    int n16, int c4) {
    if (c4 == 0) {
        cl.ml[n16][wave][0] = w.m_run;
        cl.ml[n16][wave][1] = w.l_run;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int db = 0; db < 8; ++db) o_w[(4 * c4 + i) * kOStride + 16 * db + n16] = w.acc[db][i];
}

// The workgroup's state of head h, head dims d0 .. d0+3, from the published
// states: M = max over the wavefronts, L and O rescaled to M.  wave_stride:
// floats between consecutive wavefronts' regions.
template <int kWaves>
static __device__ __forceinline__ void gather_head(const float *o_lds, int wave_stride, const CombineLdsT<kWaves> &cl,
                                                   int h, int d0, float &M, float &L, f32x4 &O) {
    float m[kWaves], l[kWaves];
#pragma unroll
    for (int p = 0; p < kWaves / 2; ++p) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(&cl.ml[h][2 * p][0]);
        m[2 * p] = v[0];
        l[2 * p] = v[1];
        m[2 * p + 1] = v[2];
        l[2 * p + 1] = v[3];
    }
    M = m[0];
#pragma unroll
    for (int wv = 1; wv < kWaves; ++wv) M = fmaxf(M, m[wv]);
    L = 0.f;
    O = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int wv = 0; wv < kWaves; ++wv) {
        const float f = m[wv] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m[wv] - M);
        L += l[wv] * f;
        O += f * *reinterpret_cast<const f32x4 *>(&o_lds[wv * wave_stride + h * kOStride + d0]);
    }
}

// Normalised output of four head dims and, from the thread owning d0 == 0, the lse.
static __device__ __forceinline__ void store_output(const AttnLaunch &a, int64_t row, int d0, f32x4 O, float M, float L) {
    const int64_t orow = row * kHeadDim + d0;
    const float inv = 1.f / L;
    if (a.out_f32)
        *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(a.out) + orow) = O * inv;
    else
        *reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(a.out) + orow) =
            u32x2{pack_bf16(O[0] * inv, O[1] * inv), pack_bf16(O[2] * inv, O[3] * inv)};
    if (d0 == 0 && a.lse) a.lse[row] = (M + __builtin_log2f(L)) * 0.69314718055994530942f;
}

// Writes the workgroup's combined result: the output itself when it covered
// the whole (layer, sequence, KV head), else a partial in slot `slot`.  bad:
// the sum becomes NaN (and so do the outputs).
template <int kWaves>
static __device__ __forceinline__ void write_result(const AttnLaunch &a, const float *o_lds, int wave_stride,
                                                    const CombineLdsT<kWaves> &cl, bool bad, int G, int tid,
                                                    int64_t row0, bool whole, uint32_t slot) {
    for (int c = tid; c < G * (kHeadDim / 4); c += kWaves * 64) {
        const int h = c / (kHeadDim / 4), d0 = (c % (kHeadDim / 4)) * 4;
        float mx, L;
        f32x4 O;
        gather_head(o_lds, wave_stride, cl, h, d0, mx, L, O);
        if (bad) L = __builtin_nanf("");
        if (whole) {
            store_output(a, row0 + h, d0, O, mx, L);
        } else {
            const uint32_t prow = slot * G + h;
            store_coherent4(raw_buffer(a.part_o, a.part_o_bytes), (prow * kHeadDim + d0) * 4, O);
            if (d0 == 0) {
                const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
                store_coherent1(rml, prow * 8, mx);
                store_coherent1(rml, prow * 8 + 4, L);
            }
        }
    }
}

// Takes a ticket for group `grp` after this workgroup's partial stores have
// completed; true in the workgroup that draws the last of `n` tickets (which
// also resets the counter for the next call).  Block-wide.
static __device__ __forceinline__ bool take_ticket(const AttnLaunch &a, int counter, int n, int tid, int &s_last) {
    wait_vmem();
    __syncthreads();
    if (tid == 0) {
        int *t = &a.ticket[(int64_t)counter * kTicketStride];
        const int prev = __hip_atomic_fetch_add(t, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = prev == n - 1;
        if (s_last) __hip_atomic_store(t, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    return s_last != 0;
}

// Where a load past the last partial must stay unconditional (a branch around a
// load lets the compiler wait for it inside the branch), it gets this offset,
// outside the buffer resource's range, which the hardware answers with zero
// and no memory access; a select or a zero weight drops it.
constexpr uint32_t kNoPartial = 0x80000000u;  // a byte offset past both partial arrays (each < 2^31 bytes)

// Cross-split log-sum-exp merges of the n partials of one group.  Each thread
// owns four consecutive head dims of one head and folds the partials in
// batches whose loads are all in flight together.  Block-wide.
// Many partials (more than 2 * kMergeBatch), slots slot0 .. slot0+n-1.  Three
// steps, none of them a chain of dependent round trips:
// * the (max, sum) pairs of every partial and head are staged in LDS, each
//   thread's loads (up to kManyPairLoads) in flight together;
// * per head, its 32 threads take the slots t, t + 32, ... each: their max, a
//   lane-shuffle max over the 32, each slot's weight exp2(m - M) (which
//   replaces the max in LDS) and its weighted sum, and a shuffle sum: no thread
//   walks all n slots;
// * the O values stream through two register batches of kManyBatch slots, the
//   next batch's loads in flight while the current one is accumulated with the
//   staged weights (a slot past the last takes an out-of-range offset and
//   weight 0).
// A head's 32 threads are one half of a wavefront, whose LDS accesses complete
// in order, so the weights need no barrier.  The sums run in slot order and in
// a fixed shuffle tree: the result does not depend on which split merges.
// s_ml: LDS scratch of n * G * 2 floats, free by the time the merge runs.
constexpr int kManyBatch = 16;
constexpr int kManyPairLoads = 4;
template <int kThreads>
static __device__ __forceinline__ void merge_many(const AttnLaunch &a, int n, uint32_t slot0, int G, int tid,
                                               int64_t row0, float *s_ml) {
    const __amdgpu_buffer_rsrc_t ro = raw_buffer(a.part_o, a.part_o_bytes);
    const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
    // The pairs of the group lie in consecutive slots: entry e = i * G + h is
    // pair slot0 * G + e.
    const int total = n * G;
    const uint32_t ml0 = slot0 * (uint32_t)G * 8;
    for (int e0 = tid; e0 < total; e0 += kManyPairLoads * kThreads) {
        float pm[kManyPairLoads], pl[kManyPairLoads];
#pragma unroll
        for (int j = 0; j < kManyPairLoads; ++j) {
            const int e = e0 + j * kThreads;
            const uint32_t off = e < total ? ml0 + (uint32_t)e * 8 : kNoPartial;
            pm[j] = load_coherent1(rml, off);
            pl[j] = load_coherent1(rml, off + 4);
        }
#pragma unroll
        for (int j = 0; j < kManyPairLoads; ++j) {
            const int e = e0 + j * kThreads;
            if (e < total) {
                s_ml[2 * e] = pm[j];
                s_ml[2 * e + 1] = pl[j];
            }
        }
    }
    __syncthreads();
    const uint32_t so = (uint32_t)G * kHeadDim * 4;  // bytes from one slot's O rows to the next
    for (int c = tid; c < G * (kHeadDim / 4); c += kThreads) {
        const int h = c / (kHeadDim / 4), t = c % (kHeadDim / 4), d0 = t * 4;
        float M = kNegInf;
        for (int i = t; i < n; i += 32) M = fmaxf(M, s_ml[2 * (i * G + h)]);
#pragma unroll
        for (int x = 16; x >= 1; x /= 2) M = fmaxf(M, __shfl_xor(M, x, 32));
        float L = 0.f;
        for (int i = t; i < n; i += 32) {
            const float m = s_ml[2 * (i * G + h)];
            const float f = m == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m - M);
            L += s_ml[2 * (i * G + h) + 1] * f;
            s_ml[2 * (i * G + h)] = f;
        }
#pragma unroll
        for (int x = 16; x >= 1; x /= 2) L += __shfl_xor(L, x, 32);
        asm volatile("" ::: "memory");  // the weights' stores stay ahead of their loads below
        const uint32_t vo = ((slot0 * (uint32_t)G + (uint32_t)h) * kHeadDim + d0) * 4;
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
        auto load_batch = [&](int base, f32x4 (&o)[kManyBatch]) {
#pragma unroll
            for (int k = 0; k < kManyBatch; ++k) {
                const bool in = base + k < n;
                o[k] = load_coherent4_s(ro, in ? vo : kNoPartial, in ? (uint32_t)(base + k) * so : 0u);
            }
        };
        auto add_batch = [&](int base, const f32x4 (&o)[kManyBatch]) {
#pragma unroll
            for (int k = 0; k < kManyBatch; ++k) {
                const int i = base + k;
                const float f = i < n ? s_ml[2 * (i * G + h)] : 0.f;
                O += o[k] * f;
            }
        };
        f32x4 ba[kManyBatch], bb[kManyBatch];
        load_batch(0, ba);
        for (int base = 0;; base += 2 * kManyBatch) {
            if (base + kManyBatch < n) load_batch(base + kManyBatch, bb);
            add_batch(base, ba);
            if (base + kManyBatch >= n) break;
            if (base + 2 * kManyBatch < n) load_batch(base + 2 * kManyBatch, ba);
            add_batch(base + kManyBatch, bb);
            if (base + 2 * kManyBatch >= n) break;
        }
        store_output(a, row0 + h, d0, O, M, L);
    }
}

// Folds the kCnt slots base .. base+kCnt-1 into (M, L, O); pair j of the
// current chunk of pairs (pm, pl) sits in lane (lane & 32) + j, for
// j = base - cb + k.
template <int kCnt, int kLen>
static __device__ __forceinline__ void merge_fold_n(const f32x4 (&o)[kLen], float pm, float pl, int cb, int base,
                                                    int lane, float &M, float &L, f32x4 &O) {
    static_assert(kCnt <= kLen && kCnt <= 32, "the slots lie in the array and in one chunk of pairs");
    float m[kCnt], l[kCnt];
#pragma unroll
    for (int k = 0; k < kCnt; ++k) {
        const int src = (lane & 32) + ((base - cb + k) & 31);
        m[k] = __shfl(pm, src);
        l[k] = __shfl(pl, src);
    }
    float mx = M;
#pragma unroll
    for (int k = 0; k < kCnt; ++k) mx = fmaxf(mx, m[k]);
    // every factor first (independent exp2s), then sums in a tree
    float lf[kCnt + 1];
    f32x4 of[kCnt + 1];
    const float sc = M == kNegInf ? 0.f : __builtin_amdgcn_exp2f(M - mx);
#pragma unroll
    for (int k = 0; k < kCnt; ++k) {
        const float f = m[k] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m[k] - mx);
        lf[k] = l[k] * f;
        of[k] = o[k] * f;
    }
    lf[kCnt] = L * sc;
    of[kCnt] = O * sc;
#pragma unroll
    for (int w = 1; w < kCnt + 1; w *= 2)
#pragma unroll
        for (int k = 0; k + w < kCnt + 1; k += 2 * w) {
            lf[k] += lf[k + w];
            of[k] += of[k + w];
        }
    L = lf[0];
    O = of[0];
    M = mx;
}

// Up to kMergeBatch partials (every group of the 12 x 300 s workloads): one
// batch, all loads of a thread in flight at once.

template <int kThreads, int kCnt, typename SlotOf, typename Emit>
static __device__ __forceinline__ void merge_one_batch_n(const AttnLaunch &a, SlotOf slot_of, int G, int tid,
                                                         Emit emit) {
    const __amdgpu_buffer_rsrc_t ro = raw_buffer(a.part_o, a.part_o_bytes);
    const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
    const int lane = tid & 63;
    for (int c = tid; c < G * (kHeadDim / 4); c += kThreads) {
        const int h = c / (kHeadDim / 4), d0 = (c % (kHeadDim / 4)) * 4;
        // the (max, sum) pairs with one load: lane j of the head's half-wavefront
        // takes slot j's, the fold shares them by lane shuffle
        const int j = lane & 31;
        const uint32_t vml = j < kCnt ? (slot_of(j) * G + h) * 8 : kNoPartial;
        const float pm = load_coherent1(rml, vml);
        const float pl = load_coherent1(rml, vml + 4);
        f32x4 oo[kCnt];
#pragma unroll
        for (int k = 0; k < kCnt; ++k) oo[k] = load_coherent4(ro, ((slot_of(k) * G + h) * kHeadDim + d0) * 4);
        float M = kNegInf, L = 0.f;
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
        merge_fold_n<kCnt>(oo, pm, pl, 0, 0, lane, M, L, O);
        emit(h, d0, O, M, L);
    }
}

// Up to kMergeBatch partials in one batch of loads, specialised on the count:
// exactly n loads of each kind (a load past the last partial, even one the
// hardware answers with zeros, still passes through the address unit).
template <int kThreads, typename SlotOf, typename Emit>
static __device__ __forceinline__ void merge_one_batch(const AttnLaunch &a, int n, SlotOf slot_of, int G, int tid,
                                                       Emit emit) {
    static_assert(kMergeBatch == 8, "one case per batch size");
    switch (n) {
    case 1: merge_one_batch_n<kThreads, 1>(a, slot_of, G, tid, emit); break;
    case 2: merge_one_batch_n<kThreads, 2>(a, slot_of, G, tid, emit); break;
    case 3: merge_one_batch_n<kThreads, 3>(a, slot_of, G, tid, emit); break;
    case 4: merge_one_batch_n<kThreads, 4>(a, slot_of, G, tid, emit); break;
    case 5: merge_one_batch_n<kThreads, 5>(a, slot_of, G, tid, emit); break;
    case 6: merge_one_batch_n<kThreads, 6>(a, slot_of, G, tid, emit); break;
    case 7: merge_one_batch_n<kThreads, 7>(a, slot_of, G, tid, emit); break;
    default: merge_one_batch_n<kThreads, 8>(a, slot_of, G, tid, emit); break;
    }
}

// The n partials lie in the slots slot0 + i * stride; emit(h, d0, O, M, L)
// takes each thread's merged state.  More than 2 * kMergeBatch partials only
// in consecutive slots (stride 1) and into the output.
template <int kThreads, typename Emit>
static __device__ __forceinline__ void merge_partials(const AttnLaunch &a, int n, uint32_t slot0, uint32_t stride,
                                                      int G, int tid, int64_t row0, float *s_ml, Emit emit) {
    if (n > 2 * kMergeBatch) {
        merge_many<kThreads>(a, n, slot0, G, tid, row0, s_ml);
        return;
    }
    const auto slot_of = [slot0, stride](int i) { return slot0 + (uint32_t)i * stride; };
    if (n <= kMergeBatch) {
        merge_one_batch<kThreads>(a, n, slot_of, G, tid, emit);
        return;
    }
    const __amdgpu_buffer_rsrc_t ro = raw_buffer(a.part_o, a.part_o_bytes);
    const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
    for (int c = tid; c < G * (kHeadDim / 4); c += kThreads) {
        const int h = c / (kHeadDim / 4), d0 = (c % (kHeadDim / 4)) * 4;
        float M = kNegInf, L = 0.f;
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
        for (int base = 0; base < n; base += kMergeBatch) {
            float mm[kMergeBatch], ll[kMergeBatch];
            f32x4 oo[kMergeBatch];
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                const uint32_t prow = slot_of(base + k < n ? base + k : 0) * G + h;
                mm[k] = load_coherent1(rml, prow * 8);
                ll[k] = load_coherent1(rml, prow * 8 + 4);
                oo[k] = load_coherent4(ro, (prow * kHeadDim + d0) * 4);
            }
            float bm = M;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k)
                if (base + k < n) bm = fmaxf(bm, mm[k]);
            const float sc = M == kNegInf ? 0.f : __builtin_amdgcn_exp2f(M - bm);
            L *= sc;
            O *= sc;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                const float f = (base + k >= n || mm[k] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mm[k] - bm);
                L += ll[k] * f;
                O += oo[k] * f;
            }
            M = bm;
        }
        emit(h, d0, O, M, L);
    }
}

// ---------------------------------------------------------------------------
// decode_attn, split schedule with LDS-staged passes, for splits longer than
// the wide schedule's: one workgroup of four wavefronts per (split, layer and
// KV head, sequence), wavefront w taking passes w, w + 4, ...  With
// kStages = 2 each wavefront double-buffers its passes in two LDS stages (K
// and V, 16 KiB per stage), issuing the next pass's direct-to-LDS loads before
// computing the current one; the workgroup takes 128 KiB of LDS, a compute
// unit to itself.  With kStages = 1 (grids of more than one dispatch round)
// each wavefront loads a pass, waits and computes it: 64 KiB, so two
// workgroups share a compute unit and one's prologue, epilogue and dispatch
// gap overlap the other's loads.  Index lists are staged too, one pass ahead
// of the rows.
// ---------------------------------------------------------------------------
template <int kSrc, int kStages>
__global__ __launch_bounds__(256) void decode_attn_lds_kernel(const int32_t *__restrict__ src0,
                                                              const int32_t *__restrict__ src1,
                                                              const int32_t *__restrict__ idx,
                                                              const uint16_t *__restrict__ q, int32_t max_keep,
                                                              int32_t B, int32_t pol_per_seq, int32_t Hkv, int32_t G,
                                                          const AttnLaunch a) {
    __shared__ __attribute__((aligned(16))) uint8_t stages[kWavesPerWg][kStages][kStageBytes];
    __shared__ __attribute__((aligned(16))) uint8_t idx_ring[kSrc != kSrcIndex ? 1 : kWavesPerWg][2][kIdxSlotBytes];
    __shared__ CombineLds cl;
    __shared__ int s_last;
    __shared__ int s_wave_flag[kWavesPerWg];
    static_assert(kMaxMergeSplits * kMaxGroup * 2 * 4 <= sizeof(stages) && kOWaveBytes <= kStages * kStageBytes,
                  "merge scratch and published rows fit the stages");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the passes' rank arithmetic is scalar
    const int n16 = lane & 15;
    const int c4 = lane >> 4;

    // Grid: x = split, y = layer * Hkv + KV head, z = sequence.  The
    // sequence's retained-set description is loaded first: the first K/V loads
    // wait for it and for nothing else.
    const int split = blockIdx.x;
    const int b = blockIdx.z;
    int32_t rg[2 * kPieces];
    int policy_bad = 0;
    int32_t cur_row = -1;  // ring storage: the current token's row
    const int layer = (int)blockIdx.y / Hkv;
    const int cnt_seq = seq_count_scalar<kSrc>(src0, src1, b, pol_per_seq, layer, B, a.ring_cap, rg, policy_bad, cur_row);
    const int g = (int)blockIdx.y - layer * Hkv;
    const int lb = layer * B + b;
    const int grp = lb * Hkv + g;  // ((layer * B) + b) * Hkv + g
    const int Hq = Hkv * G;
    const bool bad_count = cnt_seq < 1 || cnt_seq > max_keep;
    const int cnt = cnt_seq < 0 ? 0 : (cnt_seq > max_keep ? max_keep : cnt_seq);
    const int r_begin = split * a.split_len;
    const int r_end = min(r_begin + a.split_len, cnt);

    RangeTab tab;
    __amdgpu_buffer_rsrc_t irow;
    if (kSrc != kSrcIndex) tab = make_tab(rg);
    else irow = raw_buffer(idx + (int64_t)b * max_keep, (uint32_t)max_keep * 4u);  // ranks past the count are masked

    const int64_t row0 = (int64_t)lb * Hq + g * G;
    u32x4 qf[4];
    load_q(qf, q, row0, G, n16, c4);
    const int64_t kv_off = layer * a.s_layer + b * a.s_b + g * a.s_h;
    const uint16_t *kbase = a.k + kv_off;
    const uint16_t *vbase = a.v + kv_off;
    constexpr bool kRing = kSrc == kSrcRing;
    NewRows nr{cur_row, nullptr, nullptr};
    if (kRing) {
        nr.k = a.k_new + (int64_t)grp * kHeadDim;
        nr.v = a.v_new + (int64_t)grp * kHeadDim;
    }
    uint8_t *st[2] = {&stages[wave][0][0], &stages[wave][kStages - 1][0]};
    uint8_t *ring[2] = {&idx_ring[kSrc != kSrcIndex ? 0 : wave][0][0], &idx_ring[kSrc != kSrcIndex ? 0 : wave][1][0]};

    WaveAcc w;
    wave_acc_reset(w);
    int r = r_begin + wave * kWaveTile;
    materialize(kbase, vbase, a.s_pos, a.max_len, a.scale_log2, cnt);
    if (kRing) materialize(nr.k, nr.v, nr.cur);
    NewRowCopy app{};
    if (kRing) app = load_new_row(a, nr, policy_bad, lane, split == 0 && wave == 0);
    if (kSrc != kSrcIndex)
        materialize(tab.lo[1], tab.lo[2], tab.lo[3], tab.lo[4], tab.lo[5], tab.off[0], tab.off[1], tab.off[2],
                    tab.off[3], tab.off[4], tab.off[5]);
    const bool short_rows = a.s_pos < kRunRowLimit;
    if (r < r_end && kStages == 1) {
        int32_t pos[8];
        if (kSrc == kSrcIndex) {
            dma_idx(ring[0], irow, r, lane);
            dma_idx(ring[1], irow, r + kSplitUnit, lane);
        }
        for (int k = 0;; r += kSplitUnit, ++k) {
            if (kSrc != kSrcIndex) {
                dma_pass_ranges<kRing>(st[0], tab, r, r_end, a.max_len, short_rows, kbase, vbase, a.s_pos, lane, c4,
                                       w.bad_pos, nr);
            } else {
                wait_vm<1>();  // this pass's entries; the next pass's may stay in flight
                dma_pos_index(ring[k & 1], r, r_end, a.max_len, c4, pos, w.bad_pos);
                dma_pass(st[0], kbase, vbase, a.s_pos, pos, lane, kRing, nr);
            }
            wait_vm<0>();
            compute_pass_lds<true>(st[0], qf, min(kWaveTile, r_end - r), a.scale_log2, w, n16, c4);
            if (r + kSplitUnit >= r_end) break;
            if (kSrc == kSrcIndex) dma_idx(ring[k & 1], irow, r + 2 * kSplitUnit, lane);  // its slot is read
        }
    } else if (r < r_end) {
        int32_t pos[8];
        if (kSrc != kSrcIndex) {
            dma_pass_ranges<kRing>(st[0], tab, r, r_end, a.max_len, short_rows, kbase, vbase, a.s_pos, lane, c4,
                                   w.bad_pos, nr);
        } else {
            dma_idx(ring[0], irow, r, lane);
            dma_idx(ring[1], irow, r + kSplitUnit, lane);
            wait_vm<1>();
            dma_pos_index(ring[0], r, r_end, a.max_len, c4, pos, w.bad_pos);
            dma_pass(st[0], kbase, vbase, a.s_pos, pos, lane, kRing, nr);
        }
        for (int k = 0;; r += kSplitUnit, ++k) {
            const uint8_t *cur = st[k & 1];
            if (r + kSplitUnit < r_end) {
                if (kSrc != kSrcIndex) {
                    dma_pass_ranges<kRing>(st[(k + 1) & 1], tab, r + kSplitUnit, r_end, a.max_len, short_rows, kbase,
                                           vbase, a.s_pos, lane, c4, w.bad_pos, nr);
                } else {
                    wait_vm<kStageLoads>();  // entries of the next pass (issued before this pass's rows)
                    dma_pos_index(ring[(k + 1) & 1], r + kSplitUnit, r_end, a.max_len, c4, pos, w.bad_pos);
                    dma_idx(ring[k & 1], irow, r + 2 * kSplitUnit, lane);
                    dma_pass(st[(k + 1) & 1], kbase, vbase, a.s_pos, pos, lane, kRing, nr);
                }
                if (kSrc != kSrcIndex)
                    wait_vm<kStageLoads>();  // this pass's rows; the next pass's stay in flight
                else
                    wait_vm<kStageLoads + 1>();
                compute_pass_lds<true>(cur, qf, kWaveTile, a.scale_log2, w, n16, c4);
            } else {
                wait_vm<0>();
                compute_pass_lds<true>(cur, qf, min(kWaveTile, r_end - r), a.scale_log2, w, n16, c4);
                break;
            }
        }
    }

    if (kRing) store_new_row(a, app, nr, kbase, vbase, lane);
    float *o_lds = reinterpret_cast<float *>(&stages[0][0][0]);  // each wavefront's O rows in its own stages
    constexpr int kStageWaveFloats = kStages * kStageBytes / 4;
    publish_wave(w, o_lds + wave * kStageWaveFloats, cl, wave, n16, c4);
    const int wg_bad_pos = barrier_or<kWavesPerWg>(w.bad_pos, s_wave_flag, wave, lane);
    const bool bad = wg_bad_pos || bad_count;
    write_result(a, o_lds, kStageWaveFloats, cl, bad, G, tid, row0, a.n_split == 1,
                 (uint32_t)grp * a.n_split + split);
    if ((kSrc == kSrcLayout || kRing) && g == 0 &&
        (layer == 0 || (pol_per_seq & MURMUR_POL_PER_LAYER)))  // per-layer policies: one set per layer
        write_retained<kWavesPerWg * 64>(a, (pol_per_seq & MURMUR_POL_PER_LAYER) ? layer * B + b : b, cnt_seq,
                                         policy_bad, rg,
                       max_keep, tid, r_begin, r_begin + a.split_len);
    if (bad && tid == 0)
        raise_device_error((wg_bad_pos ? MURMUR_DEVERR_POSITION : 0) | (bad_count ? MURMUR_DEVERR_COUNT : 0));
    if (a.n_split == 1) return;
    constexpr int kThreads = kWavesPerWg * 64;
    const int n = a.n_split;
    const uint32_t pbase = (uint32_t)grp * n;
    float *s_ml = reinterpret_cast<float *>(&stages[0][0][0]);
    const auto to_output = [&a, row0](int h, int d0, f32x4 O, float M, float L) {
        store_output(a, row0 + h, d0, O, M, L);
    };
    if (n > 2 * kMergeBatch && n <= kTwoLevelMax) {
        // Two levels: the last split of every kSubSplits folds their partials
        // into the first one's slot (one ticket per such set, after the group
        // tickets), and the last of those sets folds theirs into the output.
        // Each merging workgroup then reads at most max(kSubSplits, n_sub)
        // partials instead of n: the merge of many partials is bound by one
        // compute unit's read rate.
        const int n_sub = (n + kSubSplits - 1) / kSubSplits;
        const int sub = (int)split / kSubSplits;
        const int sub_n = min(kSubSplits, n - sub * kSubSplits);
        const uint32_t sub0 = pbase + (uint32_t)(sub * kSubSplits);
        if (sub_n > 1) {
            const int groups = a.NL * a.B * a.Hkv;
            if (!take_ticket(a, groups + grp * n_sub + sub, sub_n, tid, s_last)) return;
            const __amdgpu_buffer_rsrc_t ro = raw_buffer(a.part_o, a.part_o_bytes);
            const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
            // Each thread reads the set's (h, d0) values and its head's pairs
            // before its own stores: a head's 32 threads are one half of a
            // wavefront, whose stores follow its loads.
            const auto to_slot = [ro, rml, sub0, G](int h, int d0, f32x4 O, float M, float L) {
                const uint32_t prow = sub0 * (uint32_t)G + (uint32_t)h;
                store_coherent4(ro, (prow * kHeadDim + d0) * 4, O);
                if (d0 == 0) {
                    store_coherent1(rml, prow * 8, M);
                    store_coherent1(rml, prow * 8 + 4, L);
                }
            };
            merge_partials<kThreads>(a, sub_n, sub0, 1, G, tid, row0, s_ml, to_slot);
        }
        if (!take_ticket(a, grp, n_sub, tid, s_last)) return;
        merge_partials<kThreads>(a, n_sub, pbase, kSubSplits, G, tid, row0, s_ml, to_output);
        return;
    }
    if (!take_ticket(a, grp, n, tid, s_last)) return;
    merge_partials<kThreads>(a, n, pbase, 1, G, tid, row0, s_ml, to_output);
}

// ---------------------------------------------------------------------------
// decode_attn, wide schedule: workgroups of kWideWaves wavefronts in a 1-D
// grid, one (layer, sequence, KV head) split each (WideSched decodes which),
// and every wavefront exactly one pass of 32 retained positions: it issues
// the direct-to-LDS loads of its K and V rows into its own 16 KiB stage and its
// query rows into registers, waits for them and computes.  A wavefront thus
// never stalls on issuing a later pass's loads before computing an earlier
// one, needs no online rescale (its state is one pass), and the workgroup's
// eight states are combined through LDS.  Splits hold at most 256 positions;
// the schedule spreads the groups' splits over one dispatch round with as
// equal shares as the group count allows.  Split partials sit in the slot of
// the workgroup's index; the last workgroup of a group merges them.
// ---------------------------------------------------------------------------
constexpr int kWideThreads = kWideWaves * 64;

// The workgroup's state of head h, head dims d0 .. d0+3, from the eight
// published wavefront states (as gather_head, with every LDS read issued
// before the first is used).
static __device__ __forceinline__ void gather_wide(const float *o_lds, int wave_stride,
                                                   const CombineLdsT<kWideWaves> &cl, int h, int d0, float &M, float &L,
                                                   f32x4 &O) {
    f32x4 ml[kWideWaves / 2], o[kWideWaves];
#pragma unroll
    for (int p = 0; p < kWideWaves / 2; ++p) ml[p] = *reinterpret_cast<const f32x4 *>(&cl.ml[h][2 * p][0]);
#pragma unroll
    for (int wv = 0; wv < kWideWaves; ++wv)
        o[wv] = *reinterpret_cast<const f32x4 *>(&o_lds[wv * wave_stride + h * kOStride + d0]);
    M = kNegInf;
#pragma unroll
    for (int p = 0; p < kWideWaves / 2; ++p) M = fmaxf(M, fmaxf(ml[p][0], ml[p][2]));
    // every factor first (independent exp2s), then sums in a tree: no chain of
    // dependent exp2 and multiply-add through the eight states
    float f[kWideWaves], lf[kWideWaves];
    f32x4 of[kWideWaves];
#pragma unroll
    for (int wv = 0; wv < kWideWaves; ++wv) {
        const float m = ml[wv / 2][(wv & 1) * 2];
        f[wv] = m == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m - M);
    }
#pragma unroll
    for (int wv = 0; wv < kWideWaves; ++wv) {
        lf[wv] = ml[wv / 2][(wv & 1) * 2 + 1] * f[wv];
        of[wv] = o[wv] * f[wv];
    }
#pragma unroll
    for (int w2 = kWideWaves / 2; w2 >= 1; w2 /= 2)
#pragma unroll
        for (int wv = 0; wv < w2; ++wv) {
            lf[wv] += lf[wv + w2];
            of[wv] += of[wv + w2];
        }
    L = lf[0];
    O = of[0];
}

// Log-sum-exp merge of the n partials of a group (slots slot0 .. slot0+n-1),
// head h, head dims d0 .. d0+3, by one thread of a wavefront whose two halves
// hold two heads (32 threads each).  The (max, sum) pairs come in chunks of 32
// slots with one load per chunk: lane j loads the pair of slot j of its half's
// head, and the others take them by lane shuffle.  The O values of all slots
// share one vector offset; each load adds its slot's distance as a scalar
// offset (inside the partial arrays: the slots are the group's own).  A load
// past the last slot takes a vector offset outside the buffer instead (the
// hardware's range check covers the vector offset, not the scalar one) and
// scalar offset 0, which the hardware answers with zero without a memory
// access.  Batches of kMergeBatch slots, the next batch's loads in flight
// while the current one is folded in.  Few load instructions matter: the
// compute unit's address unit takes them one by one for all wavefronts.
static __device__ __forceinline__ void merge_o_load(f32x4 (&o)[kMergeBatch], __amdgpu_buffer_rsrc_t ro, uint32_t vo,
                                                    uint32_t so, int base, int n) {
#pragma unroll
    for (int k = 0; k < kMergeBatch; ++k) {
        const bool in = base + k < n;
        o[k] = load_coherent4_s(ro, in ? vo : kNoPartial, in ? (uint32_t)(base + k) * so : 0u);
    }
}

// Folds the slots of the batch at `base` that exist (fewer than kMergeBatch
// when it is the group's last): the work of absent slots is not done at all.
static __device__ __forceinline__ void merge_fold(const f32x4 (&o)[kMergeBatch], float pm, float pl, int cb,
                                                  int base, int n, int lane, float &M, float &L, f32x4 &O) {
    static_assert(kMergeBatch == 8, "one case per batch size");
    switch (min(n - base, kMergeBatch)) {
    case 1: merge_fold_n<1>(o, pm, pl, cb, base, lane, M, L, O); break;
    case 2: merge_fold_n<2>(o, pm, pl, cb, base, lane, M, L, O); break;
    case 3: merge_fold_n<3>(o, pm, pl, cb, base, lane, M, L, O); break;
    case 4: merge_fold_n<4>(o, pm, pl, cb, base, lane, M, L, O); break;
    case 5: merge_fold_n<5>(o, pm, pl, cb, base, lane, M, L, O); break;
    case 6: merge_fold_n<6>(o, pm, pl, cb, base, lane, M, L, O); break;
    case 7: merge_fold_n<7>(o, pm, pl, cb, base, lane, M, L, O); break;
    default: merge_fold_n<8>(o, pm, pl, cb, base, lane, M, L, O); break;
    }
}

static_assert(32 % kMergeBatch == 0, "a batch of slots lies in one chunk of pairs");

// The merge's load offsets for a group of at most kMergeDirect splits (all
// its pairs and O values loaded at once): the (max, sum) pair of slot lane & 31
// of the thread's head (out of the buffer past the last slot), the O values'
// vector offset, which every slot shares, and per slot its scalar distance.
// Computed before the ticket, while its atomic is in flight, so that the
// merging workgroup issues its loads right after the ticket.
constexpr int kMergeDirect = 2 * kMergeBatch;
struct MergeOffsets {
    uint32_t vml;
    uint32_t vo;
    uint32_t so[kMergeDirect];  // so[0] = 0
};
static __device__ __forceinline__ MergeOffsets merge_offsets(int n, uint32_t slot0, int G, int h, int d0, int lane) {
    MergeOffsets m;
    const uint32_t j = (uint32_t)(lane & 31);
    m.vml = j < (uint32_t)n ? ((slot0 + j) * (uint32_t)G + (uint32_t)h) * 8 : kNoPartial;
    m.vo = ((slot0 * (uint32_t)G + (uint32_t)h) * kHeadDim + d0) * 4;
    const uint32_t so = (uint32_t)G * kHeadDim * 4;  // bytes from one slot's rows to the next
#pragma unroll
    for (int k = 0; k < kMergeDirect; ++k) m.so[k] = (uint32_t)k * so;
    // opaque from here on: neither moved past the ticket nor computed again there
    asm volatile(""
                 : "+v"(m.vml), "+v"(m.vo), "+s"(m.so[1]), "+s"(m.so[2]), "+s"(m.so[3]), "+s"(m.so[4]),
                   "+s"(m.so[5]), "+s"(m.so[6]), "+s"(m.so[7]), "+s"(m.so[8]), "+s"(m.so[9]), "+s"(m.so[10]),
                   "+s"(m.so[11]), "+s"(m.so[12]), "+s"(m.so[13]), "+s"(m.so[14]), "+s"(m.so[15]));
    return m;
}

// Exactly kCnt loads of O, all in flight before the fold: a load past the last
// slot would be answered with zeros without a memory access, but it still
// passes through the compute unit's address unit, on the merging workgroup's
// critical path (three such loads per thread cost c3 0.2 us).
template <int kCnt>
static __device__ __forceinline__ void merge_wide_direct_n(const AttnLaunch &a, __amdgpu_buffer_rsrc_t ro,
                                                         __amdgpu_buffer_rsrc_t rml, const MergeOffsets &mo, int h,
                                                         int d0, int lane, int64_t row0) {
    static_assert(kCnt <= kMergeDirect, "offsets for every slot");
    const float pm = load_coherent1(rml, mo.vml);
    const float pl = load_coherent1(rml, mo.vml + 4);
    f32x4 o[kCnt];
#pragma unroll
    for (int k = 0; k < kCnt; ++k) o[k] = load_coherent4_s(ro, mo.vo, k == 0 ? 0u : mo.so[k]);
    float M = kNegInf, L = 0.f;
    f32x4 O = {0.f, 0.f, 0.f, 0.f};
    merge_fold_n<kCnt>(o, pm, pl, 0, 0, lane, M, L, O);
    store_output(a, row0 + h, d0, O, M, L);
}
static __device__ __forceinline__ void merge_wide_direct(const AttnLaunch &a, __amdgpu_buffer_rsrc_t ro,
                                                         __amdgpu_buffer_rsrc_t rml, const MergeOffsets &mo, int n,
                                                         int h, int d0, int lane, int64_t row0) {
    static_assert(kMergeDirect == 16, "one case per count");
    // two searches, so that the smaller counts take no more branches than
    // one over 2 .. 8
    if (n <= 8) {
        switch (n) {
        case 2: merge_wide_direct_n<2>(a, ro, rml, mo, h, d0, lane, row0); break;
        case 3: merge_wide_direct_n<3>(a, ro, rml, mo, h, d0, lane, row0); break;
        case 4: merge_wide_direct_n<4>(a, ro, rml, mo, h, d0, lane, row0); break;
        case 5: merge_wide_direct_n<5>(a, ro, rml, mo, h, d0, lane, row0); break;
        case 6: merge_wide_direct_n<6>(a, ro, rml, mo, h, d0, lane, row0); break;
        case 7: merge_wide_direct_n<7>(a, ro, rml, mo, h, d0, lane, row0); break;
        default: merge_wide_direct_n<8>(a, ro, rml, mo, h, d0, lane, row0); break;
        }
        return;
    }
    switch (n) {
    case 9: merge_wide_direct_n<9>(a, ro, rml, mo, h, d0, lane, row0); break;
    case 10: merge_wide_direct_n<10>(a, ro, rml, mo, h, d0, lane, row0); break;
    case 11: merge_wide_direct_n<11>(a, ro, rml, mo, h, d0, lane, row0); break;
    case 12: merge_wide_direct_n<12>(a, ro, rml, mo, h, d0, lane, row0); break;
    case 13: merge_wide_direct_n<13>(a, ro, rml, mo, h, d0, lane, row0); break;
    case 14: merge_wide_direct_n<14>(a, ro, rml, mo, h, d0, lane, row0); break;
    case 15: merge_wide_direct_n<15>(a, ro, rml, mo, h, d0, lane, row0); break;
    default: merge_wide_direct_n<16>(a, ro, rml, mo, h, d0, lane, row0); break;
    }
}

static __device__ __forceinline__ void merge_wide(const AttnLaunch &a, __amdgpu_buffer_rsrc_t ro,
                                                  __amdgpu_buffer_rsrc_t rml, int n, uint32_t slot0, int G, int h,
                                                  int d0, int lane, int64_t row0) {
    const uint32_t vo = ((slot0 * (uint32_t)G + (uint32_t)h) * kHeadDim + d0) * 4;
    const uint32_t so = (uint32_t)G * kHeadDim * 4;  // bytes from one slot's rows to the next
    float M = kNegInf, L = 0.f;
    f32x4 O = {0.f, 0.f, 0.f, 0.f};
    f32x4 b0[kMergeBatch], b1[kMergeBatch];
    for (int cb = 0; cb < n; cb += 32) {
        const int j = cb + (lane & 31);
        const uint32_t vml = ((slot0 + (uint32_t)j) * (uint32_t)G + (uint32_t)h) * 8;
        const float pm = load_coherent1(rml, j < n ? vml : kNoPartial);
        const float pl = load_coherent1(rml, j < n ? vml + 4 : kNoPartial);
        const int ce = min(cb + 32, n);
        merge_o_load(b0, ro, vo, so, cb, n);
        for (int base = cb; base < ce; base += 2 * kMergeBatch) {
            if (base + kMergeBatch < ce) merge_o_load(b1, ro, vo, so, base + kMergeBatch, n);
            merge_fold(b0, pm, pl, cb, base, n, lane, M, L, O);
            if (base + kMergeBatch >= ce) break;
            if (base + 2 * kMergeBatch < ce) merge_o_load(b0, ro, vo, so, base + 2 * kMergeBatch, n);
            merge_fold(b1, pm, pl, cb, base + kMergeBatch, n, lane, M, L, O);
        }
    }
    store_output(a, row0 + h, d0, O, M, L);
}

// The hardware hands workgroup w of a launch to XCD w mod 8.  The work items
// (in the order the schedule lists them) are dealt out XCD by XCD instead:
// XCD x takes a contiguous run of them, so the splits of a group, which trade
// partials, share one L2 where the counts allow.  Of W workgroups the first
// `tall` XCDs take per = ceil(W / 8) items and the others per - 1, so XCD x's
// run starts at x (per - 1) + min(x, tall); xcd = (per - 1) | tall << 16,
// from the launch.  A bijection of [0, W).
static __device__ __forceinline__ uint32_t xcd_order(uint32_t wg, uint32_t xcd) {
    const uint32_t x = wg & 7, local = wg >> 3;
    return x * (xcd & 0xffffu) + min(x, xcd >> 16) + local;
}

// x / d for x < 2^16 and 1 <= d < 2^16 from magic = ceil(2^32 / d) - 1,
// which fits in 32 bits for every such d: (x + 1) magic / 2^32 falls short of
// (x + 1) / d by more than 0 and at most 2^-16, less than the distance from
// x / d to the next integer unless x + 1 is a multiple of d, where it gives
// exactly the floor of x / d.
static __device__ __forceinline__ uint32_t div16(uint32_t x, uint32_t magic) { return __umulhi(x + 1u, magic); }

// The WideSched fields are separate scalar arguments (with the pointers, the
// first 16 dwords, which the build preloads into SGPRs; a struct argument
// would be loaded from memory first).
template <int kSrc>
__global__ __launch_bounds__(kWideThreads) void decode_attn_wide_kernel(
    const int32_t *__restrict__ src0, const int32_t *__restrict__ src1, uint32_t xcd, uint32_t magic_n,
    uint32_t len_g, uint32_t hkv_b, uint32_t magic_hkv, uint32_t magic_b,
    const int32_t *__restrict__ idx, const uint16_t *__restrict__ q, const AttnLaunch a) {
    const WideSched ws{xcd, magic_n, len_g, hkv_b, magic_hkv, magic_b};
    // G and the policy mode from a preloaded argument: loading them from memory
    // put a second round trip in front of the first K/V loads
    const int G = (int)((ws.len >> 18) & 0x1fu);
    const int32_t pol_per_seq = (int32_t)(ws.len >> 23) & 3;
    const bool short_rows = (ws.len >> 25) & 1u;  // a K/V row is under kRunRowLimit elements
    // from the launch description: every dword of the loads it takes is then in use, so no
    // scratch value lands in a register a scalar load is still filling (which forces a wait)
    const int32_t max_keep = a.max_keep;
    __shared__ __attribute__((aligned(16))) uint8_t stages[kWideWaves][kStageBytes];
    __shared__ __attribute__((aligned(16))) uint8_t idx_slot[kSrc != kSrcIndex ? 1 : kWideWaves][kIdxSlotBytes];
    __shared__ CombineLdsT<kWideWaves> cl;
    __shared__ int s_last;
    __shared__ int s_wave_flag[kWideWaves];
    static_assert(kMaxMergeSplits * kMaxGroup * 2 * 4 <= sizeof(stages) && kMaxGroup * kOStride * 4 <= kStageBytes,
                  "merge scratch and published rows fit the stages");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the pass's rank arithmetic is scalar
    const int n16 = lane & 15;
    const int c4 = lane >> 4;

    // Which split of which group: scalar arithmetic on preloaded arguments,
    // so the retained-set description is the first memory access.
    const uint32_t wg = xcd_order(blockIdx.x, ws.xcd);
    const uint32_t n = (ws.len >> 9) & 0x1ffu;
    const uint32_t grp = div16(wg, ws.magic_n);
    const uint32_t split = wg - grp * n;
    const uint32_t len = ws.len & 0x1ffu;
    const uint32_t slot0 = grp * n;
    const int Hkv = (int)(ws.hkv_b & 0xffffu), B = (int)(ws.hkv_b >> 16);
    const uint32_t lb = div16(grp, ws.magic_hkv);
    const int g = (int)(grp - lb * (uint32_t)Hkv);
    const int layer = (int)div16(lb, ws.magic_b);
    const int b = (int)lb - layer * B;
    int32_t rg[2 * kPieces];
    int policy_bad = 0;
    int32_t cur_row = -1;  // ring storage: the current token's row
    const int32_t seq_w = seq_words<kSrc>(src0, src1, b, pol_per_seq, layer, B);
    // Every launch field the kernel reads, pinned in scalar registers here: their
    // loads go out in one batch ahead of one wait, which the vector load above
    // overlaps, instead of later batches whose waits would each add a round trip
    // before the first K/V loads.
    materialize(a.k, a.v, a.s_layer, a.s_b, a.s_h, a.s_pos, a.max_len, a.scale_log2, a.max_keep, q, a.out, a.lse,
                a.ticket, a.part_ml, a.part_o, a.part_ml_bytes, a.part_o_bytes, a.out_f32);
    if (kSrc == kSrcLayout || kSrc == kSrcRing) materialize(a.idx_out, a.count_out, a.ranges_out);
    if (kSrc == kSrcRing) materialize(a.ring_cap, a.k_new, a.v_new);
    int32_t lw[9];  // kSrcLayout: the layout and policy words, tested once the first loads are out
    int cnt_seq = seq_count_from<kSrc>(seq_w, a.ring_cap, rg, policy_bad, cur_row, lw);
    const int cnt = cnt_seq < 0 ? 0 : (cnt_seq > max_keep ? max_keep : cnt_seq);
    const int r_begin = (int)(split * len);
    const int r_end = min(r_begin + (int)len, cnt);

    RangeTab tab;
    __amdgpu_buffer_rsrc_t irow;
    if (kSrc != kSrcIndex) tab = make_tab(rg);
    else irow = raw_buffer(idx + (int64_t)b * max_keep, (uint32_t)max_keep * 4u);  // ranks past the count are masked

    const int64_t row0 = (int64_t)lb * (Hkv * G) + g * G;  // first output row of the group
    // The group's first K/V element: in 32-bit arithmetic when the launch found
    // every group's offset below 2^31 elements (three 64-bit products cost
    // about 30 scalar instructions between the description's arrival and the
    // first K/V load).
    int64_t kv_off;
    if ((ws.len >> 26) & 1u)
        kv_off = (int64_t)((uint32_t)layer * (uint32_t)a.s_layer + (uint32_t)b * (uint32_t)a.s_b +
                           (uint32_t)g * (uint32_t)a.s_h);
    else
        kv_off = layer * a.s_layer + b * a.s_b + g * a.s_h;
    const uint16_t *kbase = a.k + kv_off;
    const uint16_t *vbase = a.v + kv_off;
    constexpr bool kRing = kSrc == kSrcRing;
    NewRows nr{cur_row, nullptr, nullptr};
    if (kRing) {
        nr.k = a.k_new + (int64_t)grp * kHeadDim;
        nr.v = a.v_new + (int64_t)grp * kHeadDim;
    }
    uint8_t *stage = &stages[wave][0];

    WaveAcc w;
    wave_acc_reset(w);
    const int r0 = r_begin + wave * kWaveTile;
    bool layout_ok = true;
    materialize(kbase, vbase, a.s_pos, a.max_len, a.scale_log2, cnt);
    if (kRing) materialize(nr.k, nr.v, nr.cur);
    NewRowCopy app{};
    if (kRing) app = load_new_row(a, nr, policy_bad, lane, split == 0 && wave == 0);
    if (kSrc != kSrcIndex)
        materialize(tab.lo[1], tab.lo[2], tab.lo[3], tab.lo[4], tab.lo[5], tab.off[0], tab.off[1], tab.off[2],
                    tab.off[3], tab.off[4], tab.off[5]);
    if (r0 < r_end) {
        const int valid = min(kWaveTile, r_end - r0);
        u32x4 qf[4];
        load_q(qf, q, row0, G, n16, c4);
        if (kSrc != kSrcIndex) {
            dma_pass_ranges<kRing>(stage, tab, r0, r_end, a.max_len, short_rows, kbase, vbase, a.s_pos, lane, c4,
                                   w.bad_pos, nr);
        } else {
            int32_t pos[8];
            dma_idx(&idx_slot[wave][0], irow, r0, lane);
            wait_vm<0>();
            dma_pos_index(&idx_slot[wave][0], r0, r_end, a.max_len, c4, pos, w.bad_pos);
            dma_pass(stage, kbase, vbase, a.s_pos, pos, lane, kRing, nr);
        }
        if (kSrc == kSrcLayout) layout_ok = layout_valid_late(lw);  // while this pass's rows are on their way
        compute_pass_lds<false, true>(stage, qf, valid, a.scale_log2, w, n16, c4);
    } else if (kSrc == kSrcLayout) {
        layout_ok = layout_valid_late(lw);
    }
    if (kSrc == kSrcLayout && !layout_ok) {  // as an invalid layout gives it: count 0, empty table, no positions
        policy_bad = 1;
        cnt_seq = 0;
#pragma unroll
        for (int k = 0; k < 2 * kPieces; ++k) rg[k] = 0;
        w.bad_pos = 0;
    }
    const bool bad_count = cnt_seq < 1 || cnt_seq > max_keep;

    if (kRing) store_new_row(a, app, nr, kbase, vbase, lane);
    float *o_lds = reinterpret_cast<float *>(&stages[0][0]);  // each wavefront's O rows in its own stage
    constexpr int kStageFloats = kStageBytes / 4;
    publish_wave(w, o_lds + wave * kStageFloats, cl, wave, n16, c4);
    const int wg_bad_pos = barrier_or<kWideWaves>(w.bad_pos, s_wave_flag, wave, lane);
    const bool bad = wg_bad_pos || bad_count;
    // The workgroup's state of head h, head dims d0 .. d0+3, per writer thread:
    // the output itself for a group of one split, else the partial in slot wg.
    const bool writer = tid < G * (kHeadDim / 4);
    const int h = tid >> 5, d0 = (tid & 31) * 4;
    const __amdgpu_buffer_rsrc_t ro = raw_buffer(a.part_o, a.part_o_bytes);
    const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
    if (writer) {
        float M, L;
        f32x4 O;
        gather_wide(o_lds, kStageFloats, cl, h, d0, M, L, O);
        if (bad) L = __builtin_nanf("");
        if (n == 1) {
            store_output(a, row0 + h, d0, O, M, L);
        } else {
            const uint32_t prow = wg * (uint32_t)G + (uint32_t)h;
            store_coherent4(ro, (prow * kHeadDim + d0) * 4, O);
            if (d0 == 0) {
                store_coherent1(rml, prow * 8, M);
                store_coherent1(rml, prow * 8 + 4, L);
            }
        }
    }
    // Wavefronts whose threads hold the workgroup's state (and store the partial).
    const int writer_waves = (G * (kHeadDim / 4) + 63) / 64;
    if ((kSrc == kSrcLayout || kRing) && g == 0 &&
        (layer == 0 || (pol_per_seq & MURMUR_POL_PER_LAYER))) {  // per-layer policies: one set per layer
        const int b_out = (pol_per_seq & MURMUR_POL_PER_LAYER) ? layer * B + b : b;
        const int r_hi = split == n - 1 ? max_keep : r_begin + (int)len;
        // By the wavefronts that store no partial when they are half of them:
        // the ticket then waits for the partial stores only, not for these.
        if (writer_waves <= kWideWaves / 2) {
            if (wave >= kWideWaves / 2)
                write_retained<kWideThreads / 2>(a, b_out, cnt_seq, policy_bad, rg, max_keep, tid - kWideThreads / 2,
                                                 r_begin, r_hi);
        } else {
            write_retained<kWideThreads>(a, b_out, cnt_seq, policy_bad, rg, max_keep, tid, r_begin, r_hi);
        }
    }
    if (bad && tid == 0)
        raise_device_error((wg_bad_pos ? MURMUR_DEVERR_POSITION : 0) | (bad_count ? MURMUR_DEVERR_COUNT : 0));
    if (n == 1) return;
    MergeOffsets mo;
    if (n <= (uint32_t)kMergeDirect) mo = merge_offsets((int)n, slot0, G, h, d0, lane);
    // Ticket: one per workgroup, once every writer wavefront's partial stores
    // have completed (each waits for its own, then the barrier); the workgroup
    // that takes the group's n-th merges.  (A ticket per writer wavefront saves
    // the barrier but queues four times the atomics on the group's counter,
    // which costs more.)  The other wavefronts' stores (the retained set) are
    // not waited for.
    if (wave < writer_waves) wait_vmem();
    __syncthreads();
    if (tid == 0) {
        const int prev = __hip_atomic_fetch_add(&a.ticket[grp * kTicketStride], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = prev == (int)n - 1;
        if (s_last) __hip_atomic_store(&a.ticket[grp * kTicketStride], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!s_last) return;
    if (writer) {
        if (n <= (uint32_t)kMergeDirect)
            merge_wide_direct(a, ro, rml, mo, (int)n, h, d0, lane, row0);
        else
            merge_wide(a, ro, rml, (int)n, slot0, G, h, d0, lane, row0);
    }
}

// Read-only streaming probe (measurement): workgroup w reads the 16-byte
// units [w * per, (w + 1) * per) of the buffer.  kLds false: each thread
// issues kDepth loads into registers (indexes clamped into the share, so every
// load is unconditional), then folds them into an XOR.  kLds true: the loads
// go straight to LDS (the attention kernels' load type), wavefront by
// wavefront, each into the next of kDepth 1 KiB slots of the wavefront's own
// ring, kDepth of them in flight at any time; the XOR is then taken over the
// last ring.  Block size: any multiple of 64 up to 1024.
template <int kDepth, bool kLds>
__global__ __launch_bounds__(1024) void read_probe_kernel(const u32x4 *__restrict__ p, int64_t n16,
                                                          uint32_t *__restrict__ sink) {
    extern __shared__ __align__(16) uint8_t probe_ring[];
    const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const int64_t lo = (int64_t)blockIdx.x * per;
    const int64_t hi = lo + per < n16 ? lo + per : n16;
    const int T = blockDim.x;
    u32x4 acc = {0, 0, 0, 0};
    if constexpr (!kLds) {
        for (int64_t i = lo + threadIdx.x; i < hi; i += (int64_t)kDepth * T) {
            u32x4 v[kDepth];
#pragma unroll
            for (int k = 0; k < kDepth; ++k) {
                const int64_t j = i + (int64_t)k * T;
                v[k] = p[j < hi ? j : hi - 1];
            }
#pragma unroll
            for (int k = 0; k < kDepth; ++k) acc ^= v[k];
        }
    } else {
        const int lane = threadIdx.x & 63;
        uint8_t *ring = probe_ring + (threadIdx.x >> 6) * kDepth * 1024;
        int slot = 0;
        // wavefront-uniform trip count: the last units of a share are clamped
        for (int64_t b = lo + (threadIdx.x & ~63); b < hi; b += T) {
            const int64_t j = b + lane < hi ? b + lane : hi - 1;
            __builtin_amdgcn_global_load_lds(p + j, (lds_void_t *)(ring + slot * 1024), 16, 0, 0);
            slot = slot + 1 == kDepth ? 0 : slot + 1;
            wait_vm<kDepth - 1>();
        }
        wait_vm<0>();
        acc = *(const u32x4 *)(ring + lane * 16);
    }
    const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    if (x == 0x9E3779B9u) sink[blockIdx.x] = x;
}

__global__ void workspace_init_kernel(int32_t *ticket, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        ticket[i] = 0;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
int launch_evict_compact(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B,
                         int32_t *idx, int32_t max_keep, int32_t *count, int32_t *ranges, const int32_t *bt,
                         int32_t max_blocks, int32_t log2_bs, murmur_stream_t stream) {
    hipLaunchKernelGGL(evict_compact_kernel, dim3(B), dim3(256), 0, (hipStream_t)stream, seg, pol, pol_per_seq,
                       max_keep, idx, count, ranges, bt, max_blocks, log2_bs);
    return (int)hipGetLastError();
}

// Whether every (layer, sequence, KV head) group's first K/V element lies
// below 2^31 elements from the cache's base (the strides are non-negative).
static bool small_group_offsets(const AttnLaunch &a) {
    const __int128 last = (__int128)(a.NL - 1) * a.s_layer + (__int128)(a.B - 1) * a.s_b + (__int128)(a.Hkv - 1) * a.s_h;
    return last < ((__int128)1 << 31);
}

template <int kSrc>
static void launch_decode_attn_mode(const AttnLaunch &a, hipStream_t stream) {
    if (a.wide_wg > 0) {
        const WideSched &w = a.sched;
        hipLaunchKernelGGL(decode_attn_wide_kernel<kSrc>, dim3((unsigned)a.wide_wg), dim3(kWideThreads), 0, stream,
                           a.src0, a.src1, w.xcd, w.magic_n,
                           w.len | (uint32_t)(a.pol_per_seq & 3) << 23 | (uint32_t)(a.s_pos < kRunRowLimit) << 25 |
                               (uint32_t)small_group_offsets(a) << 26,
                           w.hkv_b, w.magic_hkv, w.magic_b, a.idx,
                           a.q, a);
        return;
    }
    const dim3 grid((unsigned)a.n_split, (unsigned)(a.NL * a.Hkv), (unsigned)a.B);
    // Longer splits stage their passes in LDS, double-buffered within one
    // dispatch round, else one stage per wavefront and two workgroups per
    // compute unit.
    const bool one_round = (int64_t)a.n_split * a.NL * a.Hkv * a.B <= kRoundWorkgroups;
    if (one_round)
        hipLaunchKernelGGL((decode_attn_lds_kernel<kSrc, 2>), grid, dim3(kWavesPerWg * 64), 0, stream, a.src0, a.src1,
                           a.idx, a.q, a.max_keep, a.B, a.pol_per_seq, a.Hkv, a.G, a);
    else
        hipLaunchKernelGGL((decode_attn_lds_kernel<kSrc, 1>), grid, dim3(kWavesPerWg * 64), 0, stream, a.src0, a.src1,
                           a.idx, a.q, a.max_keep, a.B, a.pol_per_seq, a.Hkv, a.G, a);
}

int launch_decode_attn(const AttnLaunch &a, murmur_stream_t stream) {
    if (a.src_mode == kSrcRing)
        launch_decode_attn_mode<kSrcRing>(a, (hipStream_t)stream);
    else if (a.src_mode == kSrcLayout)
        launch_decode_attn_mode<kSrcLayout>(a, (hipStream_t)stream);
    else if (a.src_mode == kSrcRanges)
        launch_decode_attn_mode<kSrcRanges>(a, (hipStream_t)stream);
    else
        launch_decode_attn_mode<kSrcIndex>(a, (hipStream_t)stream);
    return (int)hipGetLastError();
}

int launch_paged_step(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B, int32_t *bt,
                      int32_t max_blocks, int32_t log2_bs, int32_t *stack, int32_t *top, int32_t capacity,
                      int32_t full_scan, murmur_stream_t stream) {
    hipLaunchKernelGGL(paged_step_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, seg, pol, pol_per_seq, B, bt,
                       max_blocks, log2_bs, stack, top, capacity, full_scan);
    return (int)hipGetLastError();
}

int launch_paged_append(const murmur_seg *seg, int32_t B, const int32_t *bt, int32_t max_blocks, int32_t log2_bs,
                        const murmur_kv &pool, int32_t Hkv, const void *k_new, const void *v_new,
                        murmur_stream_t stream) {
    const int64_t items = (int64_t)B * pool.n_layers * Hkv * 2 * 16;
    const int64_t blocks = (items + 255) / 256 < 1024 ? (items + 255) / 256 : 1024;
    hipLaunchKernelGGL(paged_append_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, seg, B, bt,
                       max_blocks, log2_bs, (uint16_t *)pool.k, (uint16_t *)pool.v, pool.stride_layer, pool.stride_h,
                       pool.stride_pos, (int64_t)pool.max_len, (const uint16_t *)k_new, (const uint16_t *)v_new,
                       pool.n_layers, Hkv);
    return (int)hipGetLastError();
}

template <int kDepth>
static int launch_read_probe_depth(const void *buf, int64_t n16, int32_t n_workgroups, int32_t threads, bool lds,
                                   uint32_t *sink, murmur_stream_t stream) {
    const size_t lds_bytes = lds ? (size_t)(threads / 64) * kDepth * 1024 : 0;
    if (lds)
        hipLaunchKernelGGL((read_probe_kernel<kDepth, true>), dim3((unsigned)n_workgroups), dim3((unsigned)threads),
                           lds_bytes, (hipStream_t)stream, (const u32x4 *)buf, n16, sink);
    else
        hipLaunchKernelGGL((read_probe_kernel<kDepth, false>), dim3((unsigned)n_workgroups), dim3((unsigned)threads),
                           0, (hipStream_t)stream, (const u32x4 *)buf, n16, sink);
    return (int)hipGetLastError();
}

int launch_read_probe(const void *buf, int64_t n16, int32_t n_workgroups, int32_t threads, int32_t depth, bool lds,
                      uint32_t *sink, murmur_stream_t stream) {
    switch (depth) {
    case 1: return launch_read_probe_depth<1>(buf, n16, n_workgroups, threads, lds, sink, stream);
    case 2: return launch_read_probe_depth<2>(buf, n16, n_workgroups, threads, lds, sink, stream);
    case 4: return launch_read_probe_depth<4>(buf, n16, n_workgroups, threads, lds, sink, stream);
    case 8: return launch_read_probe_depth<8>(buf, n16, n_workgroups, threads, lds, sink, stream);
    case 16: return launch_read_probe_depth<16>(buf, n16, n_workgroups, threads, lds, sink, stream);
    default: return (int)hipErrorInvalidValue;
    }
}

int launch_workspace_init(int32_t *ticket, int64_t n, murmur_stream_t stream) {
    const int64_t blocks = n / 256 + 1 < 1024 ? n / 256 + 1 : 1024;
    hipLaunchKernelGGL(workspace_init_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, ticket, n);
    return (int)hipGetLastError();
}

// Scratch of murmur_decode_step_static (tickets, then split partials, laid out
// as a workspace of MURMUR_STATIC_SCRATCH_BYTES): one copy per device, held
// until the process ends.  Host code never uses the array's name as an
// address: static_scratch() looks the device address up once per device.
static __device__ __align__(256) uint8_t scratch[MURMUR_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mutex;
static void *g_scratch_ptr[kMaxDevices];

int static_scratch(void **ptr, bool *fresh) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return (int)e;
    if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    *fresh = g_scratch_ptr[dev] == nullptr;
    if (*fresh) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return (int)e;
        if (p == nullptr || (uintptr_t)p % 256 != 0) return (int)hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return 0;
}

int read_and_clear_device_error(murmur_stream_t stream, int32_t *code) {
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e != hipSuccess) return (int)e;
    int32_t v = 0;
    e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_device_error), sizeof v, 0, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return (int)e;
    const int32_t zero = 0;
    e = hipMemcpyToSymbol(HIP_SYMBOL(g_device_error), &zero, sizeof zero, 0, hipMemcpyHostToDevice);
    if (e != hipSuccess) return (int)e;
    *code = v;
    return 0;
}

const char *hip_error_text(int err) { return hipGetErrorString((hipError_t)err); }

}  // namespace murmur
