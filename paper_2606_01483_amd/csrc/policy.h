// Closed form of Murmur's retained KV set (Section 3.2), shared by the host
// sizing call and the device kernels of libmurmur.
//
// For one sequence with layout [prompt_pre][speech][prompt_mid][output] at
// output step j (1-based, counting the current token) the kept positions are:
//   * both system prompts, always;
//   * speech (Algorithm 2 with Equation 2's sinks): the first n_sink speech
//     tokens and a window of w speech tokens starting at
//     l_j = max(0, j - max(d,1) + 1), clamped to speech_len - w;
//     the window count is w (Algorithm 2), not w + 1;
//   * output (Algorithm 1, applied to the output region): 1-based output
//     tokens 1..n_sink and max(1, j-w+1)..j.
// A window of -1 (or one at least as long as its region) keeps the region.
//
// The set is returned as six non-overlapping pieces in ascending position
// order: prompt_pre, speech sinks, speech window, prompt_mid, output sinks,
// output window.  Adjacent or overlapping parts are merged into the earlier
// piece, so every piece but a merged-away one is maximal and empty pieces
// start where the previous one ends.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define MURMUR_HD __host__ __device__
#else
#define MURMUR_HD
#endif

namespace murmur {

constexpr int kPieces = 6;

// Row of position p (>= 0) of one sequence in a paged pool: block table row
// bt_row of max_blocks physical block numbers, blocks of 1 << log2_bs rows
// (log2_bs <= 20), row = bt_row[p >> log2_bs] * block size + p mod block size.
// -1 when p lies past the table, in a block whose entry is negative (a freed
// block), or in a row beyond 2^31 - 1.  The table is read inside its bounds only.
MURMUR_HD inline int32_t paged_pool_row(const int32_t *bt_row, int32_t max_blocks, int32_t log2_bs, int32_t p) {
    const int32_t blk = p >> log2_bs;
    const int32_t entry = bt_row[blk < max_blocks ? blk : 0];
    const int32_t phys = blk < max_blocks ? entry : -1;
    if (phys < 0) return -1;
    const int64_t row = ((int64_t)phys << log2_bs) | (int64_t)(p & ((1 << log2_bs) - 1));
    return row > (int64_t)0x7fffffff ? -1 : (int32_t)row;
}

struct Pieces {
    int32_t start[kPieces];
    int32_t len[kPieces];
    int32_t count;
};

// Whether a layout and policy are valid: no negative length, j >= 1, windows
// -1 or >= 1, no negative delay or sink count, and a sequence of at most
// 2^31 - 1 positions.
MURMUR_HD inline bool layout_valid(int32_t p_pre, int32_t l_s, int32_t p_mid, int32_t j, int32_t w_s, int32_t d,
                                   int32_t n_ss, int32_t w_o, int32_t n_so) {
    if (p_pre < 0 || l_s < 0 || p_mid < 0 || j < 1) return false;
    if (!(w_s == -1 || w_s >= 1) || d < 0 || n_ss < 0) return false;
    if (!(w_o == -1 || w_o >= 1) || n_so < 0) return false;
    return (int64_t)p_pre + l_s + p_mid + j <= 0x7fffffffLL;
}

// 32-bit sums and differences that wrap instead of overflowing: for a valid
// layout every intermediate value fits, so they are exact there.
MURMUR_HD inline int32_t wrap_add(int32_t a, int32_t b) { return (int32_t)((uint32_t)a + (uint32_t)b); }
MURMUR_HD inline int32_t wrap_sub(int32_t a, int32_t b) { return (int32_t)((uint32_t)a - (uint32_t)b); }

// The pieces of the retained set without the validity test: for a valid layout
// and policy the same as retained_pieces; for an invalid one some well-defined
// but meaningless table (a caller that uses it must bound every position it
// reads and discard the result once layout_valid says no).
MURMUR_HD inline void retained_pieces_unchecked(int32_t p_pre, int32_t l_s, int32_t p_mid, int32_t j, int32_t w_s,
                                                int32_t d, int32_t n_ss, int32_t w_o, int32_t n_so, Pieces *out) {
    const int32_t speech0 = p_pre, mid0 = wrap_add(p_pre, l_s), out0 = wrap_add(mid0, p_mid);

    out->start[0] = 0;
    out->len[0] = p_pre;

    // Speech: sinks [0, ns) united with the window [l, l + w).
    if (w_s == -1 || w_s >= l_s) {
        out->start[1] = speech0;
        out->len[1] = l_s;
        out->start[2] = mid0;
        out->len[2] = 0;
    } else {
        const int32_t first_move = d > 1 ? d : 1;
        int32_t l = j >= first_move ? wrap_add(wrap_sub(j, first_move), 1) : 0;
        const int32_t room = wrap_sub(l_s, w_s);
        if (l > room) l = room;
        const int32_t ns = n_ss < l_s ? n_ss : l_s;
        const int32_t win_end = wrap_add(l, w_s);
        if (l <= ns) {  // the window touches or overlaps the sinks: one piece
            const int32_t end = ns > win_end ? ns : win_end;
            out->start[1] = speech0;
            out->len[1] = end;
            out->start[2] = wrap_add(speech0, end);
            out->len[2] = 0;
        } else {
            out->start[1] = speech0;
            out->len[1] = ns;
            out->start[2] = wrap_add(speech0, l);
            out->len[2] = w_s;
        }
    }

    out->start[3] = mid0;
    out->len[3] = p_mid;

    // Output: 0-based sinks [0, so) united with the window [j - w, j).
    const int32_t w0 = wrap_sub(j, w_o);
    const int32_t so = n_so < j ? n_so : j;
    if (w_o == -1 || w_o >= j || w0 <= so) {
        out->start[4] = out0;
        out->len[4] = j;
        out->start[5] = wrap_add(out0, j);
        out->len[5] = 0;
    } else {
        out->start[4] = out0;
        out->len[4] = so;
        out->start[5] = wrap_add(out0, w0);
        out->len[5] = w_o;
    }
    int32_t c = 0;
    for (int k = 0; k < kPieces; ++k) c = wrap_add(c, out->len[k]);
    out->count = c;
}

// Returns 0 and fills *out, or -1 if the layout or policy is invalid (see
// layout_valid).
MURMUR_HD inline int retained_pieces(int32_t p_pre, int32_t l_s, int32_t p_mid, int32_t j, int32_t w_s, int32_t d,
                                     int32_t n_ss, int32_t w_o, int32_t n_so, Pieces *out) {
    if (!layout_valid(p_pre, l_s, p_mid, j, w_s, d, n_ss, w_o, n_so)) return -1;
    retained_pieces_unchecked(p_pre, l_s, p_mid, j, w_s, d, n_ss, w_o, n_so, out);
    return 0;
}

// Physical eviction storage: the output region of a sequence holds its
// n_sink output sinks at slots 0 .. n_sink-1, followed by a ring of `cap`
// slots; 0-based output token i >= n_sink lives at slot
// n_sink + (i - n_sink) mod cap.  A token whose slot is reused by a later
// one is exactly a token Algorithm 1 has evicted, as long as the window fits
// the ring (cap >= w) or, with output eviction off, as long as no slot has
// been reused yet (j - n_sink <= cap).  Prompt and speech positions are
// unchanged, so the storage of a sequence spans
// prompt_pre + speech_len + prompt_mid + n_sink + cap rows.
//
// Rewrites the pieces of retained_pieces (same count) into storage
// positions and gives the slot of the current token j.  The output part
// stays within two pieces: when the window wraps around the ring, its newer
// part starts at ring slot 0, right after the sinks, and joins them in
// piece 4; the older part is piece 5.  Pieces are then in storage order of
// rows, not in order of position.  Returns 0, -1 for an invalid layout or
// policy (as retained_pieces), or -2 when the ring cannot hold the retained
// outputs (cap < 1, cap < w, or output eviction off and j - n_sink > cap).
MURMUR_HD inline int ring_pieces(int32_t p_pre, int32_t l_s, int32_t p_mid, int32_t j, int32_t w_s, int32_t d,
                                 int32_t n_ss, int32_t w_o, int32_t n_so, int32_t cap, Pieces *out, int32_t *cur) {
    if (retained_pieces(p_pre, l_s, p_mid, j, w_s, d, n_ss, w_o, n_so, out) != 0) return -1;
    if (cap < 1 || (w_o >= 1 && cap < w_o)) return -2;
    const int64_t rows = (int64_t)p_pre + l_s + p_mid + n_so + cap;
    if (rows > 0x7fffffffLL) return -1;
    const int32_t out0 = p_pre + l_s + p_mid;
    const int32_t last = j - 1;  // 0-based output index of the current token
    *cur = out0 + (last < n_so ? last : n_so + (last - n_so) % cap);
    if (out->len[5] == 0) {
        // Every output token 0 .. j-1 is kept (one piece from the region's
        // start): the ring must not have wrapped yet.
        if (j > n_so && j - n_so > cap) return -2;
        return 0;
    }
    // Window [w0, j) of w_o tokens, all past the sinks (w0 > n_so).
    const int32_t w0 = j - w_o;
    const int32_t a = (w0 - n_so) % cap;
    const int32_t ring0 = out0 + n_so;
    if (a + w_o <= cap) {
        out->start[5] = ring0 + a;
    } else {
        out->len[4] = n_so + (a + w_o - cap);  // sinks, then ring slots 0 .. a + w_o - cap - 1
        out->start[5] = ring0 + a;
        out->len[5] = cap - a;
    }
    return 0;
}

// Positions that no step from j on retains again, so their K/V can be freed
// (Section 3.2: an evicted entry leaves the cache for good).  The speech
// window's start l_j never decreases with j and the output window
// [j - w, j) only moves forward, so these are, in global positions,
//   speech:  [prompt_pre + min(n_sink, l_s), prompt_pre + l_j), the tokens
//            behind the window that are not sinks (empty with speech
//            eviction off);
//   output:  [out0 + n_sink, out0 + j - w), the output tokens older than the
//            window that are not sinks (empty with output eviction off).
// Everything else -- prompts, sinks, the windows, speech ahead of the window
// -- is retained now or at a later step.  Returns 0 and fills
// {start, length} of both, or -1 for an invalid layout or policy (as
// retained_pieces).
MURMUR_HD inline int evicted_ranges(int32_t p_pre, int32_t l_s, int32_t p_mid, int32_t j, int32_t w_s, int32_t d,
                                    int32_t n_ss, int32_t w_o, int32_t n_so, int32_t speech[2], int32_t output[2]) {
    Pieces pc;
    if (retained_pieces(p_pre, l_s, p_mid, j, w_s, d, n_ss, w_o, n_so, &pc) != 0) return -1;
    speech[0] = p_pre;
    speech[1] = 0;
    if (w_s != -1 && w_s < l_s) {
        const int32_t first_move = d > 1 ? d : 1;
        int32_t l = j >= first_move ? j - first_move + 1 : 0;
        if (l > l_s - w_s) l = l_s - w_s;
        const int32_t ns = n_ss < l_s ? n_ss : l_s;
        if (l > ns) {
            speech[0] = p_pre + ns;
            speech[1] = l - ns;
        }
    }
    const int32_t out0 = p_pre + l_s + p_mid;
    output[0] = out0;
    output[1] = 0;
    if (w_o != -1 && j - w_o > n_so) {
        output[0] = out0 + n_so;
        output[1] = j - w_o - n_so;
    }
    return 0;
}

}  // namespace murmur
