"""Chunked inference (Section 3.1) and Equation 4's timestamp offsets: the oracle's pins, and the
library's host planner (murmur_plan_chunks, murmur_chunk_timestamps) against the oracle.  CPU only."""
import functools
import math

import numpy as np
import pytest

from oracle import chunks as C
from paper_2606_01483_amd import murmur as M


def random_segments(rng, n, max_seg=40.0, max_gap=20.0, long_every=0):
    segs, t = [], float(rng.uniform(0, max_gap))
    for i in range(n):
        d = float(rng.uniform(0.5, max_seg))
        if long_every and i % long_every == long_every - 1:
            d = float(rng.uniform(300, 800))  # longer than a chunk
        segs.append((t, t + d))
        t += d + float(rng.uniform(0.0, max_gap))
    return segs, t + float(rng.uniform(0, max_gap))


def check_tiling(chunks, segs, audio_len, c):
    assert chunks[0][0] == 0.0
    for (s0, l0), (s1, _) in zip(chunks, chunks[1:]):
        assert math.isclose(s0 + l0, s1, rel_tol=0, abs_tol=1e-9)
    for s, ln in chunks:
        assert 0 < ln <= c + 1e-9
    end = chunks[-1][0] + chunks[-1][1]
    assert end <= audio_len + 1e-9
    assert all(e <= end + 1e-9 for _, e in segs)  # every segment's speech is covered


# ---- oracle pins -------------------------------------------------------------------------------------

def test_an_hour_of_speech_is_twelve_chunks_of_2250_speech_tokens():
    """An hour of continuous speech in 300 s chunks: 12 chunks (the batch of the 12 x 300 s workloads),
    each 300 s, i.e. the paper's L_s = 2,250 speech tokens at 7.5 tokens per second (Section 3.2)."""
    segs = [(10.0 * i, 10.0 * (i + 1)) for i in range(360)]
    chunks = C.plan(segs, 3600.0, 300.0)
    assert chunks == [(300.0 * i, 300.0) for i in range(12)]
    assert all(round(ln * 7.5) == 2250 for _, ln in chunks)


def test_chunks_tile_the_recording_and_respect_the_limit():
    rng = np.random.default_rng(1)
    for long_every in (0, 7):
        for _ in range(100):
            segs, audio_len = random_segments(rng, int(rng.integers(1, 60)), long_every=long_every)
            check_tiling(C.plan(segs, audio_len, 300.0), segs, audio_len, 300.0)


def test_only_segments_longer_than_a_chunk_are_cut():
    rng = np.random.default_rng(2)
    for _ in range(100):
        segs, audio_len = random_segments(rng, int(rng.integers(1, 60)), long_every=9)
        chunks = C.plan(segs, audio_len, 300.0)
        bounds = [s for s, _ in chunks[1:]]
        for s, e in segs:
            cuts = [b for b in bounds if s < b < e]
            if e - s <= 300.0:
                assert not cuts, (s, e, cuts)
            else:
                assert len(cuts) >= math.ceil((e - s) / 300.0) - 1


def test_equation_4_offsets_are_the_chunk_starts():
    """Equation 4's offset (the summed lengths of the earlier chunks) is the chunk's start time."""
    rng = np.random.default_rng(3)
    segs, audio_len = random_segments(rng, 80, long_every=11)
    chunks = C.plan(segs, audio_len, 300.0)
    lens = [ln for _, ln in chunks]
    idx = list(range(len(chunks)))
    t_local = [float(rng.uniform(0, ln)) for ln in lens]
    for t, (s, _), tl in zip(C.timestamps(t_local, idx, lens), chunks, t_local):
        assert math.isclose(t, s + tl, rel_tol=0, abs_tol=1e-9)


def test_greedy_uses_the_fewest_chunks():
    """With every segment shorter than a chunk, the greedy merge needs as few chunks as any tiling from 0
    that keeps segments whole and chunks within c (brute force over the admissible chunk ends: segment
    starts and ends and t + c, never inside a segment)."""
    rng = np.random.default_rng(4)
    c = 60.0
    for _ in range(300):
        n = int(rng.integers(1, 8))
        segs, t = [], float(rng.uniform(0, 10))
        for _ in range(n):
            d = float(rng.uniform(1, 30))
            segs.append((t, t + d))
            t += d + float(rng.uniform(0, 40))
        points = sorted({p for s in segs for p in s})

        @functools.lru_cache(maxsize=None)
        def fewest(t0):  # chunks needed for the speech after t0, the next chunk starting at t0
            if all(e <= t0 for _, e in segs):
                return 0
            if all(e <= t0 + c for _, e in segs):
                return 1
            ends = [p for p in points if t0 < p <= t0 + c] + [t0 + c]
            ends = [e for e in ends if not any(s < e < f for s, f in segs)]
            return min((1 + fewest(e) for e in ends), default=math.inf)

        assert len(C.plan(segs, t, c)) == fewest(0.0)


# ---- the library's host planner against the oracle ---------------------------------------------------

@pytest.mark.parametrize("long_every", [0, 5])
def test_plan_chunks_matches_oracle(long_every):
    rng = np.random.default_rng(10 + long_every)
    for _ in range(150):
        segs, audio_len = random_segments(rng, int(rng.integers(0, 70)), max_gap=float(rng.choice([20.0, 400.0])),
                                          long_every=long_every)
        want = C.plan(segs, audio_len, 300.0)
        s0 = [s for s, _ in segs]
        s1 = [e for _, e in segs]
        cs, cl, tok, of = M.murmur_plan_chunks(s0, s1, audio_len, 300.0, 7.5)
        assert len(cs) == len(want)
        for (ws, wl), gs, gl, gt in zip(want, cs, cl, tok):
            assert gs == ws and math.isclose(gl, wl, rel_tol=0, abs_tol=1e-9)
            assert gt == round(gl * 7.5)
        for i, (s, _) in enumerate(segs):
            c = int(of[i])
            assert cs[c] <= s and (c == len(cs) - 1 or s < cs[c + 1])


def test_plan_chunks_an_hour():
    cs, cl, tok, of = M.murmur_plan_chunks([10.0 * i for i in range(360)], [10.0 * (i + 1) for i in range(360)],
                                           3600.0, 300.0, 7.5)
    assert np.array_equal(cs, 300.0 * np.arange(12)) and np.all(cl == 300.0) and np.all(tok == 2250)
    assert np.array_equal(of, np.arange(360) // 30)


def test_chunk_timestamps_match_oracle():
    rng = np.random.default_rng(7)
    lens = [float(x) for x in rng.uniform(1, 300, 40)]
    chunk = [int(x) for x in rng.integers(0, 40, 500)]
    t_local = [float(rng.uniform(0, lens[i])) for i in chunk]
    got = M.murmur_chunk_timestamps(t_local, chunk, lens)
    assert np.allclose(got, C.timestamps(t_local, chunk, lens), rtol=0, atol=1e-9)


def test_plan_chunks_rejects_bad_input():
    with pytest.raises(M.MurmurError):
        M.murmur_plan_chunks([10.0, 5.0], [12.0, 8.0], 100.0)      # unsorted
    with pytest.raises(M.MurmurError):
        M.murmur_plan_chunks([0.0, 5.0], [6.0, 8.0], 100.0)        # overlapping
    with pytest.raises(M.MurmurError):
        M.murmur_plan_chunks([0.0], [120.0], 100.0)                # past the end
    with pytest.raises(M.MurmurError):
        M.murmur_plan_chunks([0.0], [10.0], 100.0, max_chunk=0.0)
    with pytest.raises(M.MurmurError):
        M.murmur_chunk_timestamps([1.0], [3], [10.0, 10.0])        # no chunk 3
    with pytest.raises(M.MurmurError):
        M.murmur_plan_chunks([0.0], [10.0], 1e9, max_chunk=1.0)  # more than 2^24 chunks
    cs, cl, tok, of = M.murmur_plan_chunks([], [], 100.0)
    assert len(cs) == 0
