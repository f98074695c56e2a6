// gfx950 (MI355X, CDNA4) kernels of libmurmur.
//
//   evict_compact_kernel  Section 3.2, Algorithms 1-2 and Equation 2: the
//                         retained set of every sequence as an ascending index
//                         list, a count and a six-piece range table.
//   decode_attn_kernel    Section 3.2, Equation 1: split-K grouped-query decode
//                         attention over the retained positions, fp32
//                         accumulation, with the log-sum-exp merge of the
//                         splits fused into the last workgroup of each
//                         (layer, sequence, KV head).
//
// Attention data flow per 64-wide wavefront and pass of 32 retained positions:
//   K rows  --global 16 B loads-->  MFMA A operands   S^T = K Q^T (16x16x32 bf16)
//   V rows  --global 16 B loads-->  8x8 bf16 transpose in registers
//           --ds_write_b128 (swizzled)--> LDS --ds_read_b64--> MFMA B operands
//   P = exp2(S - m) stays in registers: the S^T accumulator layout is already
//   the A-operand layout of O = P V, split into bf16 hi + lo parts so the
//   product keeps ~16 mantissa bits.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

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
__global__ __launch_bounds__(256) void evict_compact_kernel(const murmur_seg *__restrict__ seg,
                                                            const murmur_policy *__restrict__ pol,
                                                            int32_t pol_per_seq, int32_t max_keep,
                                                            int32_t *__restrict__ idx, int32_t *__restrict__ count,
                                                            int32_t *__restrict__ ranges) {
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
#pragma unroll
    for (int k = 0; k < kPieces; ++k) {
        const int n = pc.len[k] < max_keep - off ? pc.len[k] : max_keep - off;
        for (int t = tid; t < n; t += blockDim.x) row[off + t] = pc.start[k] + t;
        off += pc.len[k];
        if (off >= max_keep) break;
    }
    for (int r = pc.count + tid; r < max_keep; r += blockDim.x) row[r] = -1;
}

// ---------------------------------------------------------------------------
// decode_attn helpers
// ---------------------------------------------------------------------------
static __device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

static __device__ __forceinline__ u32x4 load16(const uint16_t *p) { return *reinterpret_cast<const u32x4 *>(p); }

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
static __device__ __forceinline__ uint32_t bf16_rne(float f) {
    const uint32_t u = __builtin_bit_cast(uint32_t, f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

static __device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __builtin_bit_cast(float, bits16 << 16); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two fp32 values -> packed bf16 pair (x in the low half), round to nearest
// even: one v_cvt_pk_bf16_f32 on gfx950.
static __device__ __forceinline__ uint32_t pack_bf16(float x, float y) {
    const bf16x2 v = {(__bf16)x, (__bf16)y};
    return __builtin_bit_cast(uint32_t, v);
}

// Rank r of the retained list -> global position, from the six-piece table.
static __device__ __forceinline__ int rank_to_pos(const int32_t (&rg)[2 * kPieces], int r) {
#pragma unroll
    for (int k = 0; k < kPieces; ++k) {
        if (r < rg[2 * k + 1]) return rg[2 * k] + r;
        r -= rg[2 * k + 1];
    }
    return -1;
}

// LDS tile of one wavefront: V^T for 128 head dims x 32 positions, in 16-byte
// units (one head dim, eight positions).  Unit (d, q) -- q = position octet --
// sits at q*128 + swz(d); the XOR swizzle and the half swap for odd d make both
// the transposing ds_write_b128 and the operand ds_read_b64 bank-conflict free
// for 32- and 64-bank LDS models.
static __device__ __forceinline__ int vt_unit(int d, int q) {
    const int dp = d ^ ((d >> 3) & 7) ^ (((d >> 6) & 1) << 3);
    return q * 128 + dp;
}

constexpr int kVtBytesPerWave = 4 * 128 * 16;  // 8 KiB
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

// K and V fragments of one pass of kWaveTile retained positions.
struct PassRegs {
    u32x4 kf[2][4];  // MFMA A operands: position 16*blk + n16, head dims kc*32 + 8*c4 .. +8
    u32x4 vf[8];     // position 8*c4 + t, head dims 8*n16 .. +8
};

// ---------------------------------------------------------------------------
// decode_attn: one workgroup per (split, KV head, sequence, layer).  Each of
// its four wavefronts takes passes of 32 retained positions, interleaved over
// the split.  kMultiPass: splits longer than one workgroup pass keep an online
// softmax across passes and have the next pass's loads in flight while the
// current one is computed; otherwise every wavefront makes at most one pass.
// ---------------------------------------------------------------------------
template <bool kMultiPass>
// The leading scalar arguments are the ones the first memory accesses need;
// the build preloads them into SGPRs so no kernel-argument load precedes the
// range-table load.
__global__ __launch_bounds__(256) void decode_attn_kernel(const int32_t *__restrict__ count,
                                                          const int32_t *__restrict__ ranges,
                                                          const int32_t *__restrict__ idx,
                                                          const uint16_t *__restrict__ q, int32_t max_keep,
                                                          int32_t B, const AttnLaunch a) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[kWavesPerWg * kVtBytesPerWave];
    __shared__ float ml_lds[kWavesPerWg][kMaxGroup][2];
    __shared__ int s_last;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int n16 = lane & 15;
    const int c4 = lane >> 4;

    // Grid: x = split, y = KV head, z = layer * B + sequence.
    const int split = blockIdx.x;
    const int g = blockIdx.y;
    const int lb = blockIdx.z;
    const int b = lb % B;
    const int layer = lb / B;
    const int grp = lb * a.Hkv + g;  // ((layer * B) + b) * Hkv + g
    const int G = a.G;

    int cnt = count[b];
    const bool bad_count = cnt < 1 || cnt > max_keep;
    if (bad_count) cnt = cnt < 0 ? 0 : (cnt > max_keep ? max_keep : cnt);
    int bad_pos = 0;
    const int r_begin = split * a.split_len;
    const int r_end = min(r_begin + a.split_len, cnt);

    int32_t rg[2 * kPieces];
    const bool use_ranges = ranges != nullptr;
#pragma unroll
    for (int k = 0; k < 2 * kPieces; ++k) rg[k] = use_ranges ? ranges[b * 2 * kPieces + k] : 0;
    const int32_t *idx_row = idx + (int64_t)b * max_keep;

    // Q^T as the MFMA B operand: lane (head n16, k-group c4) holds head dims
    // kc*32 + 8*c4 .. +8 for kc = 0..3.  Rows past the group are zero.
    u32x4 qf[4];
    {
        const int hq = n16 < G ? n16 : G - 1;  // keep the address inside q for padded rows
        const uint16_t *qrow = q + ((int64_t)lb * a.Hq + g * G + hq) * kHeadDim;
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) qf[kc] = n16 < G ? load16(qrow + kc * 32 + 8 * c4) : u32x4{0, 0, 0, 0};
    }
    const uint16_t *kbase = a.k + layer * a.s_layer + b * a.s_b + g * a.s_h;
    const uint16_t *vbase = a.v + layer * a.s_layer + b * a.s_b + g * a.s_h;

    uint8_t *vt = smem + wave * kVtBytesPerWave;

    float m_run = kNegInf;  // running max of head n16, log2 units
    float l_run = 0.f;      // running sum of exp2(s - m_run) of head n16
    f32x4 acc[8];           // O rows 4*c4 + i (heads), column 16*db + n16 (head dim)
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Positions of the pass starting at rank r0, then every K and V load of it.
    auto issue = [&](int r0, PassRegs &R) {
        const int myrank = r0 + (lane & 31);
        int mypos = -1;  // position of rank r0 + (lane & 31); -1 past the split or if invalid
        if (myrank < r_end) {
            const int p = use_ranges ? rank_to_pos(rg, myrank) : idx_row[myrank];
            if (p >= 0 && p < a.max_len)
                mypos = p;
            else
                bad_pos = 1;
        }
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            const int pos = __shfl(mypos, 16 * blk + n16);
            const uint16_t *row = kbase + (int64_t)(pos < 0 ? 0 : pos) * a.s_pos;
#pragma unroll
            for (int kc = 0; kc < 4; ++kc)
                R.kf[blk][kc] = pos >= 0 ? load16(row + kc * 32 + 8 * c4) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int pos = __shfl(mypos, 8 * c4 + t);
            const uint16_t *row = vbase + (int64_t)(pos < 0 ? 0 : pos) * a.s_pos;
            R.vf[t] = pos >= 0 ? load16(row + 8 * n16) : u32x4{0, 0, 0, 0};
        }
    };

    auto consume = [&](int r0, const PassRegs &R) {
        // S^T = K Q^T: lane (head n16, c4), register i of block blk holds the
        // logit of rank r0 + 16*blk + 4*c4 + i.
        f32x4 s[2];
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            s[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < 4; ++kc) s[blk] = mfma16x16x32(R.kf[blk][kc], qf[kc], s[blk]);
        }

        // Logits in log2 units; ranks past the split end are masked (only a
        // wavefront's last, partial pass has any).
        float x[2][4];
        const bool partial = r_end - r0 < kWaveTile;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[blk][i] = s[blk][i] * a.scale_log2;
                if (partial && 16 * blk + 4 * c4 + i >= r_end - r0) x[blk][i] = kNegInf;
            }
        float tmax = fmaxf(fmaxf(fmaxf(x[0][0], x[0][1]), fmaxf(x[0][2], x[0][3])),
                           fmaxf(fmaxf(x[1][0], x[1][1]), fmaxf(x[1][2], x[1][3])));
        tmax = max_over_c4(tmax);
        const float m_new = kMultiPass ? fmaxf(m_run, tmax) : tmax;  // finite: rank r0 is always valid
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
        if (kMultiPass) {
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // 0 on the first pass (m_run = -inf)
            l_run = l_run * alpha + psum;
            // Rescale O rows: row 4*c4 + i belongs to head 4*c4 + i.
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float ai = __shfl(alpha, 4 * c4 + i);
#pragma unroll
                for (int db = 0; db < 8; ++db) acc[db][i] *= ai;
            }
        } else {
            l_run = psum;
        }
        m_run = m_new;

        // P as the A operand of O = P V, k order (4*c4 + 0..3, 16 + 4*c4 + 0..3),
        // split into bf16 hi + lo so that hi + lo carries ~16 mantissa bits.
        u32x4 p_hi, p_lo;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const int blk = w >> 1, i0 = (w & 1) * 2;
            const float e0 = pr[blk][i0], e1 = pr[blk][i0 + 1];
            const uint32_t hi = pack_bf16(e0, e1);
            p_hi[w] = hi;
            p_lo[w] = pack_bf16(e0 - __builtin_bit_cast(float, hi << 16),
                                e1 - __builtin_bit_cast(float, hi & 0xffff0000u));
        }

        // V^T through LDS.  Lane (e = n16, octet c4) holds positions 8*c4 + t
        // (t = 0..7) of head dims 8e .. 8e+7; one v_perm_b32 per output word
        // gathers a head dim's values of two positions, then one 16-byte unit
        // per head dim is stored (halves swapped for odd head dims).
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int w = i >> 1;
            const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;  // high or low halves of both words
            uint32_t o[4];
#pragma unroll
            for (int pp = 0; pp < 4; ++pp) o[pp] = __builtin_amdgcn_perm(R.vf[2 * pp + 1][w], R.vf[2 * pp][w], sel);
            const u32x4 unit = (i & 1) ? u32x4{o[2], o[3], o[0], o[1]} : u32x4{o[0], o[1], o[2], o[3]};
            *reinterpret_cast<u32x4 *>(vt + vt_unit(8 * n16 + i, c4) * 16) = unit;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        // O += P V for each block of 16 head dims.  B operand lane (dim n16,
        // c4) needs positions 4*c4 .. +3 and 16 + 4*c4 .. +3 of head dim d.
#pragma unroll
        for (int db = 0; db < 8; ++db) {
            const int d = 16 * db + n16;
            const int hsw = ((c4 & 1) ^ (d & 1)) * 8;
            const u32x2 lo = *reinterpret_cast<const u32x2 *>(vt + vt_unit(d, c4 >> 1) * 16 + hsw);
            const u32x2 hi = *reinterpret_cast<const u32x2 *>(vt + vt_unit(d, 2 + (c4 >> 1)) * 16 + hsw);
            const u32x4 bv = u32x4{lo[0], lo[1], hi[0], hi[1]};
            acc[db] = mfma16x16x32(p_hi, bv, acc[db]);
            acc[db] = mfma16x16x32(p_lo, bv, acc[db]);
        }
        // The next pass overwrites this wave's tile only after these reads
        // have returned (their results feed the MFMAs above).
    };

    {
        int r0 = r_begin + wave * kWaveTile;
        PassRegs cur;
        if (r0 < r_end) issue(r0, cur);
        if (kMultiPass) {
            for (; r0 < r_end; r0 += kSplitUnit) {
                PassRegs nxt;
                const bool more = r0 + kSplitUnit < r_end;
                if (more) issue(r0 + kSplitUnit, nxt);
                consume(r0, cur);
                if (more) cur = nxt;
            }
        } else if (r0 < r_end) {
            consume(r0, cur);
        }
    }

    // ---- combine the four wavefronts of the workgroup -------------------
    __shared__ float mlf_lds[kMaxGroup][2];  // per head: workgroup max (log2 units), workgroup sum
    if (c4 == 0) {
        ml_lds[wave][n16][0] = m_run;
        ml_lds[wave][n16][1] = l_run;
    }
    const int wg_bad_pos = __syncthreads_or(bad_pos);
    const bool bad = wg_bad_pos || bad_count;
    float *o_lds = reinterpret_cast<float *>(smem);  // [wave][16][128], reuses the V tiles
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int h = 4 * c4 + i;
        if (h < G) {
            const float mx = fmaxf(fmaxf(ml_lds[0][h][0], ml_lds[1][h][0]), fmaxf(ml_lds[2][h][0], ml_lds[3][h][0]));
            const float mine = ml_lds[wave][h][0];
            const float f = mine == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mine - mx);
#pragma unroll
            for (int db = 0; db < 8; ++db) o_lds[(wave * kMaxGroup + h) * kHeadDim + 16 * db + n16] = acc[db][i] * f;
        }
    }
    if (tid < G) {
        const float mx = fmaxf(fmaxf(ml_lds[0][tid][0], ml_lds[1][tid][0]), fmaxf(ml_lds[2][tid][0], ml_lds[3][tid][0]));
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < kWavesPerWg; ++w) {
            const float mw = ml_lds[w][tid][0];
            L += ml_lds[w][tid][1] * (mw == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mw - mx));
        }
        mlf_lds[tid][0] = mx;
        mlf_lds[tid][1] = bad ? __builtin_nanf("") : L;
    }
    __syncthreads();

    // Each thread owns four consecutive head dims of one head.
    const int64_t row0 = (int64_t)lb * a.Hq + g * G;  // first output row of the group
    const float ln2 = 0.69314718055994530942f;
    for (int c = tid; c < G * (kHeadDim / 4); c += blockDim.x) {
        const int h = c / (kHeadDim / 4), d0 = (c % (kHeadDim / 4)) * 4;
        f32x4 O = *reinterpret_cast<const f32x4 *>(&o_lds[h * kHeadDim + d0]);
#pragma unroll
        for (int w = 1; w < kWavesPerWg; ++w) O += *reinterpret_cast<const f32x4 *>(&o_lds[(w * kMaxGroup + h) * kHeadDim + d0]);
        const float mx = mlf_lds[h][0], L = mlf_lds[h][1];
        if (a.n_split == 1) {
            const int64_t orow = (row0 + h) * kHeadDim + d0;
            const float inv = 1.f / L;
            if (a.out_f32)
                *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(a.out) + orow) = O * inv;
            else
                *reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(a.out) + orow) =
                    u32x2{pack_bf16(O[0] * inv, O[1] * inv), pack_bf16(O[2] * inv, O[3] * inv)};
            if (d0 == 0 && a.lse) a.lse[row0 + h] = (mx + __builtin_log2f(L)) * ln2;
        } else {
            const uint32_t prow = ((uint32_t)grp * a.n_split + split) * G + h;
            store_coherent4(raw_buffer(a.part_o, a.part_o_bytes), (prow * kHeadDim + d0) * 4, O);
            if (d0 == 0) {
                const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
                store_coherent1(rml, prow * 8, mx);
                store_coherent1(rml, prow * 8 + 4, L);
            }
        }
    }
    if (bad && tid == 0)
        raise_device_error((wg_bad_pos ? MURMUR_DEVERR_POSITION : 0) | (bad_count ? MURMUR_DEVERR_COUNT : 0));
    if (a.n_split == 1) return;

    // ---- cross-split log-sum-exp merge by the last workgroup of the group ----
    // Every partial store has completed before the ticket is taken, so the
    // workgroup that draws the last ticket sees all partials.
    wait_vmem();
    __syncthreads();
    if (tid == 0) {
        const int prev = __hip_atomic_fetch_add(&a.ticket[grp], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = prev == a.n_split - 1;
    }
    __syncthreads();
    if (!s_last) return;
    if (tid == 0) __hip_atomic_store(&a.ticket[grp], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    // Each thread owns four consecutive head dims of one head and folds the
    // splits in batches whose loads are all in flight together.
    const uint32_t pbase = (uint32_t)grp * a.n_split;
    const __amdgpu_buffer_rsrc_t ro = raw_buffer(a.part_o, a.part_o_bytes);
    const __amdgpu_buffer_rsrc_t rml = raw_buffer(a.part_ml, a.part_ml_bytes);
    for (int c = tid; c < G * (kHeadDim / 4); c += blockDim.x) {
        const int h = c / (kHeadDim / 4), d0 = (c % (kHeadDim / 4)) * 4;
        float M = kNegInf, L = 0.f;
        f32x4 O = {0.f, 0.f, 0.f, 0.f};
        for (int base = 0; base < a.n_split; base += kMergeBatch) {
            float mm[kMergeBatch], ll[kMergeBatch];
            f32x4 oo[kMergeBatch];
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                const uint32_t prow = (pbase + (base + k < a.n_split ? base + k : 0)) * G + h;
                mm[k] = load_coherent1(rml, prow * 8);
                ll[k] = load_coherent1(rml, prow * 8 + 4);
                oo[k] = load_coherent4(ro, (prow * kHeadDim + d0) * 4);
            }
            float bm = M;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k)
                if (base + k < a.n_split) bm = fmaxf(bm, mm[k]);
            const float sc = M == kNegInf ? 0.f : __builtin_amdgcn_exp2f(M - bm);
            L *= sc;
            O *= sc;
#pragma unroll
            for (int k = 0; k < kMergeBatch; ++k) {
                const float f = (base + k >= a.n_split || mm[k] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(mm[k] - bm);
                L += ll[k] * f;
                O += oo[k] * f;
            }
            M = bm;
        }
        const int64_t orow = (row0 + h) * kHeadDim + d0;
        const float inv = 1.f / L;
        if (a.out_f32)
            *reinterpret_cast<f32x4 *>(reinterpret_cast<float *>(a.out) + orow) =
                f32x4{O[0] * inv, O[1] * inv, O[2] * inv, O[3] * inv};
        else
            *reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(a.out) + orow) =
                u32x2{pack_bf16(O[0] * inv, O[1] * inv), pack_bf16(O[2] * inv, O[3] * inv)};
        if (d0 == 0 && a.lse) a.lse[row0 + h] = (M + __builtin_log2f(L)) * ln2;
    }
}

__global__ void workspace_init_kernel(int32_t *ticket, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        ticket[i] = 0;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
int launch_evict_compact(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B,
                         int32_t *idx, int32_t max_keep, int32_t *count, int32_t *ranges, murmur_stream_t stream) {
    hipLaunchKernelGGL(evict_compact_kernel, dim3(B), dim3(256), 0, (hipStream_t)stream, seg, pol, pol_per_seq,
                       max_keep, idx, count, ranges);
    return (int)hipGetLastError();
}

int launch_decode_attn(const AttnLaunch &a, murmur_stream_t stream) {
    const dim3 grid((unsigned)a.n_split, (unsigned)a.Hkv, (unsigned)(a.NL * a.B));
    // Splits of more than one pass per wavefront double-buffer their loads.
    if (a.split_len > kSplitUnit)
        hipLaunchKernelGGL(decode_attn_kernel<true>, grid, dim3(kWavesPerWg * 64), 0, (hipStream_t)stream, a.count,
                           a.ranges, a.idx, a.q, a.max_keep, a.B, a);
    else
        hipLaunchKernelGGL(decode_attn_kernel<false>, grid, dim3(kWavesPerWg * 64), 0, (hipStream_t)stream, a.count,
                           a.ranges, a.idx, a.q, a.max_keep, a.B, a);
    return (int)hipGetLastError();
}

int launch_workspace_init(int32_t *ticket, int64_t n, murmur_stream_t stream) {
    const int64_t blocks = n / 256 + 1 < 1024 ? n / 256 + 1 : 1024;
    hipLaunchKernelGGL(workspace_init_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, ticket, n);
    return (int)hipGetLastError();
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
