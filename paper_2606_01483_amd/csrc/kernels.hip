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

// ---------------------------------------------------------------------------
// decode_attn: one workgroup per (split, KV head, sequence, layer).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void decode_attn_kernel(const AttnLaunch a) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[kWavesPerWg * kVtBytesPerWave];
    __shared__ float ml_lds[kWavesPerWg][kMaxGroup][2];
    __shared__ int s_last;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int n16 = lane & 15;
    const int c4 = lane >> 4;

    const int split = blockIdx.x % a.n_split;
    const int grp = blockIdx.x / a.n_split;  // ((layer * B) + b) * Hkv + g
    const int g = grp % a.Hkv;
    const int lb = grp / a.Hkv;
    const int b = lb % a.B;
    const int layer = lb / a.B;
    const int G = a.G;

    int cnt = a.count[b];
    const bool bad_count = cnt < 1 || cnt > a.max_keep;
    if (bad_count) cnt = cnt < 0 ? 0 : (cnt > a.max_keep ? a.max_keep : cnt);
    int bad_pos = 0;
    const int r_begin = split * a.split_len;
    const int r_end = min(r_begin + a.split_len, cnt);

    int32_t rg[2 * kPieces];
    const bool use_ranges = a.ranges != nullptr;
#pragma unroll
    for (int k = 0; k < 2 * kPieces; ++k) rg[k] = use_ranges ? a.ranges[b * 2 * kPieces + k] : 0;
    const int32_t *idx_row = a.idx + (int64_t)b * a.max_keep;

    // Q^T as the MFMA B operand: lane (head n16, k-group c4) holds head dims
    // kc*32 + 8*c4 .. +8 for kc = 0..3.  Rows past the group are zero.
    u32x4 qf[4];
    {
        const int hq = n16 < G ? n16 : G - 1;  // keep the address inside q for padded rows
        const uint16_t *qrow = a.q + ((int64_t)(layer * a.B + b) * a.Hq + g * G + hq) * kHeadDim;
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

    for (int r0 = r_begin + wave * kWaveTile; r0 < r_end; r0 += kSplitUnit) {
        // Position of rank r0 + (lane & 31); -1 past the split or if invalid.
        const int myrank = r0 + (lane & 31);
        int mypos = -1;
        if (myrank < r_end) {
            const int p = use_ranges ? rank_to_pos(rg, myrank) : idx_row[myrank];
            if (p >= 0 && p < a.max_len)
                mypos = p;
            else
                bad_pos = 1;
        }
        int kpos[2], vpos[8];
        kpos[0] = __shfl(mypos, n16);
        kpos[1] = __shfl(mypos, 16 + n16);
#pragma unroll
        for (int t = 0; t < 8; ++t) vpos[t] = __shfl(mypos, 8 * c4 + t);

        // Issue every K and V load of the pass before any use.
        u32x4 kf[2][4], vf[8];
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            const uint16_t *row = kbase + (int64_t)(kpos[blk] < 0 ? 0 : kpos[blk]) * a.s_pos;
#pragma unroll
            for (int kc = 0; kc < 4; ++kc)
                kf[blk][kc] = kpos[blk] >= 0 ? load16(row + kc * 32 + 8 * c4) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint16_t *row = vbase + (int64_t)(vpos[t] < 0 ? 0 : vpos[t]) * a.s_pos;
            vf[t] = vpos[t] >= 0 ? load16(row + 8 * n16) : u32x4{0, 0, 0, 0};
        }

        // S^T = K Q^T: lane (head n16, c4), register i of block blk holds the
        // logit of rank r0 + 16*blk + 4*c4 + i.
        f32x4 s[2];
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            s[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < 4; ++kc) s[blk] = mfma16x16x32(kf[blk][kc], qf[kc], s[blk]);
        }

        float x[2][4];
        float tmax = kNegInf;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rank = r0 + 16 * blk + 4 * c4 + i;
                x[blk][i] = rank < r_end ? s[blk][i] * a.scale_log2 : kNegInf;
                tmax = fmaxf(tmax, x[blk][i]);
            }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float m_new = fmaxf(m_run, tmax);  // finite: rank r0 is always valid
        const float alpha = exp2f(m_run - m_new);
        float psum = 0.f;
        float pr[2][4];
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                pr[blk][i] = exp2f(x[blk][i] - m_new);
                psum += pr[blk][i];
            }
        psum += __shfl_xor(psum, 16);
        psum += __shfl_xor(psum, 32);
        l_run = l_run * alpha + psum;
        m_run = m_new;

        // Rescale O rows: row 4*c4 + i belongs to head 4*c4 + i.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float ai = __shfl(alpha, 4 * c4 + i);
#pragma unroll
            for (int db = 0; db < 8; ++db) acc[db][i] *= ai;
        }

        // P as the A operand of O = P V: k order (4*c4 + 0..3, 16 + 4*c4 + 0..3).
        u32x4 p_hi, p_lo;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const int blk = w >> 1, i0 = (w & 1) * 2;
            const uint32_t h0 = bf16_rne(pr[blk][i0]), h1 = bf16_rne(pr[blk][i0 + 1]);
            const uint32_t l0 = bf16_rne(pr[blk][i0] - bf16_to_f32(h0));
            const uint32_t l1 = bf16_rne(pr[blk][i0 + 1] - bf16_to_f32(h1));
            p_hi[w] = h0 | (h1 << 16);
            p_lo[w] = l0 | (l1 << 16);
        }

        // V^T through LDS.  Lane (e = n16, octet c4) holds positions 8*c4 + t
        // (t = 0..7) of head dims 8e .. 8e+7; transpose to one 16-byte unit per
        // head dim and store it (halves swapped for odd head dims).
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int w = i >> 1;
            uint32_t o[4];
#pragma unroll
            for (int pp = 0; pp < 4; ++pp) {
                const uint32_t lo = vf[2 * pp][w], hi = vf[2 * pp + 1][w];
                o[pp] = (i & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
            }
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
    }

    // ---- combine the four wavefronts of the workgroup -------------------
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
            float mx = kNegInf;
#pragma unroll
            for (int w = 0; w < kWavesPerWg; ++w) mx = fmaxf(mx, ml_lds[w][h][0]);
            const float mine = ml_lds[wave][h][0];
            const float f = mine == kNegInf ? 0.f : exp2f(mine - mx);
#pragma unroll
            for (int db = 0; db < 8; ++db) o_lds[(wave * kMaxGroup + h) * kHeadDim + 16 * db + n16] = acc[db][i] * f;
        }
    }
    __syncthreads();

    const int64_t row0 = (int64_t)(layer * a.B + b) * a.Hq + g * G;  // first output row of the group
    const float qnan = __builtin_nanf("");
    const float ln2 = 0.69314718055994530942f;
    for (int e = tid; e < G * kHeadDim; e += blockDim.x) {
        const int h = e >> 7, d = e & 127;
        float mx = kNegInf;
#pragma unroll
        for (int w = 0; w < kWavesPerWg; ++w) mx = fmaxf(mx, ml_lds[w][h][0]);
        float L = 0.f, O = 0.f;
#pragma unroll
        for (int w = 0; w < kWavesPerWg; ++w) {
            const float mw = ml_lds[w][h][0];
            const float f = mw == kNegInf ? 0.f : exp2f(mw - mx);
            L += ml_lds[w][h][1] * f;
            O += o_lds[(w * kMaxGroup + h) * kHeadDim + d];
        }
        if (bad) L = qnan;
        if (a.n_split == 1) {
            const float y = O / L;
            if (a.out_f32)
                reinterpret_cast<float *>(a.out)[(row0 + h) * kHeadDim + d] = y;
            else
                reinterpret_cast<uint16_t *>(a.out)[(row0 + h) * kHeadDim + d] = (uint16_t)bf16_rne(y);
            if (d == 0 && a.lse) a.lse[row0 + h] = (mx + log2f(L)) * ln2;
        } else {
            const int64_t prow = ((int64_t)grp * a.n_split + split) * G + h;
            a.part_o[prow * kHeadDim + d] = O;
            if (d == 0) {
                a.part_ml[prow * 2 + 0] = mx;
                a.part_ml[prow * 2 + 1] = L;
            }
        }
    }
    if (bad && tid == 0)
        raise_device_error((wg_bad_pos ? MURMUR_DEVERR_POSITION : 0) | (bad_count ? MURMUR_DEVERR_COUNT : 0));
    if (a.n_split == 1) return;

    // ---- cross-split log-sum-exp merge by the last workgroup of the group ----
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const int prev = atomicAdd(&a.ticket[grp], 1);
        s_last = prev == a.n_split - 1;
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (tid == 0) atomicExch(&a.ticket[grp], 0);  // ready for the next call

    const int64_t pbase = (int64_t)grp * a.n_split;
    for (int e = tid; e < G * kHeadDim; e += blockDim.x) {
        const int h = e >> 7, d = e & 127;
        float mx = kNegInf;
        for (int sp = 0; sp < a.n_split; ++sp) mx = fmaxf(mx, a.part_ml[((pbase + sp) * G + h) * 2]);
        float L = 0.f, O = 0.f;
        for (int sp = 0; sp < a.n_split; ++sp) {
            const int64_t prow = (pbase + sp) * G + h;
            const float ms = a.part_ml[prow * 2];
            const float f = ms == kNegInf ? 0.f : exp2f(ms - mx);
            L += a.part_ml[prow * 2 + 1] * f;
            O += a.part_o[prow * kHeadDim + d] * f;
        }
        const float y = O / L;
        if (a.out_f32)
            reinterpret_cast<float *>(a.out)[(row0 + h) * kHeadDim + d] = y;
        else
            reinterpret_cast<uint16_t *>(a.out)[(row0 + h) * kHeadDim + d] = (uint16_t)bf16_rne(y);
        if (d == 0 && a.lse) a.lse[row0 + h] = (mx + log2f(L)) * ln2;
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
    const int64_t groups = (int64_t)a.NL * a.B * a.Hkv;
    const int64_t grid = groups * a.n_split;
    hipLaunchKernelGGL(decode_attn_kernel, dim3((unsigned)grid), dim3(kWavesPerWg * 64), 0, (hipStream_t)stream, a);
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
