"""Pins for the oracle's retained set (paper Section 3.2: Algorithm 1, Algorithm 2, Equation 2, Equation 3).

The oracle runs the eviction procedures as loops over a boolean mask.  These
tests hold it to things fixed independently of that code: the ratios the paper
prints for Equation 3, a hand-worked example, closed forms for the set sizes,
the prose description of the speech window's motion, and structural invariants.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
OFF = -1


def ranges_of(idx_row, count):
    """Compress an ascending position list into [start, end) runs."""
    runs = []
    for p in idx_row[:count]:
        p = int(p)
        if runs and runs[-1][1] == p:
            runs[-1][1] = p + 1
        else:
            runs.append([p, p + 1])
    return [tuple(r) for r in runs]


def one(seg, pol):
    idx, cnt = oracle.retained(np.array([seg]), np.array(pol))
    return idx[0], int(cnt[0])


# ---- Equation 3: the paper's printed speed-up ratios -------------------------------------------

def test_eq3_printed_ratios():
    """Summing the oracle's per-step attention-set sizes over T steps reproduces rho = 1.51 and 1.06.

    Equation 3 charges L_s + j tokens per step without eviction and n_sink + w + j with it.  The
    oracle is run with a speech window of n_sink + w tokens (sinks disjoint from the window carry the
    same count), outputs un-evicted, no prompts, over j = 1..T.
    """
    g = json.load(open(os.path.join(GOLDEN, "eq3_speedup.json")))
    l_s, T = g["speech_tokens"], g["decode_steps"]
    j = np.arange(1, T + 1)
    seg = np.stack([np.zeros(T), np.full(T, l_s), np.zeros(T), j], axis=1).astype(np.int32)
    _, dense = oracle.retained(seg, np.array([OFF, 0, 0, OFF, 0]))
    assert np.array_equal(dense, l_s + j)
    for case in g["cases"]:
        kept = case["n_sink"] + case["window"]
        _, evict = oracle.retained(seg, np.array([kept, 0, 0, OFF, 0]))
        assert np.array_equal(evict, kept + j)
        rho = dense.astype(np.float64).sum() / evict.astype(np.float64).sum()
        assert round(rho, case["decimals"]) == case["rho_printed"], (case, rho)


def test_eq3_with_real_sinks_rounds_to_printed():
    """With the 4 sinks held separately from a 1024 window the ratio still rounds to the printed 1.51
    (the sinks overlap the window only during the first few steps)."""
    l_s, T = 2250, 2700
    j = np.arange(1, T + 1)
    seg = np.stack([np.zeros(T), np.full(T, l_s), np.zeros(T), j], axis=1).astype(np.int32)
    _, dense = oracle.retained(seg, np.array([OFF, 0, 0, OFF, 0]))
    _, evict = oracle.retained(seg, np.array([1024, 0, 4, OFF, 0]))
    assert round(dense.sum() / evict.sum(), 2) == 1.51


# ---- a hand-worked example (the Tiny workload) -----------------------------------------------

@pytest.mark.parametrize("j,expected", [
    # prompt [0,32); speech [32,482); output starts at 482.  Speech window w=128, delay d=72,
    # output window 32.  j=65 < d: window start l=0 -> speech [32,160), contiguous with the
    # prompt; output keeps 1-based 34..65 -> [482+33, 482+65).
    (65, [(0, 160), (515, 547)]),
    # j = d: Algorithm 2 increments l once before forming the set -> speech [33,161).
    (72, [(0, 32), (33, 161), (522, 554)]),
    # j = 80: l = 80-72+1 = 9 -> speech [41,169); output 49..80 -> [530,562).
    (80, [(0, 32), (41, 169), (530, 562)]),
])
def test_tiny_worked_example(j, expected):
    idx, cnt = one([32, 450, 0, j], [128, 72, 0, 32, 0])
    assert cnt == 192
    assert ranges_of(idx, cnt) == expected
    assert np.all(idx[cnt:] == -1)


# ---- closed forms -------------------------------------------------------------------------------

def window_start_from_prose(j, d):
    """Equation 2's prose: l = 0 for the steps before d, then one further every step (from j = d on,
    as Algorithm 2 increments before forming the set)."""
    first_move = max(d, 1)
    return 0 if j < first_move else j - first_move + 1


def closed_form_count(seg, pol):
    p_pre, l_s, p_mid, j = seg
    w_s, d, n_ss, w_o, n_so = pol
    if w_s == OFF or w_s >= l_s:
        speech = l_s
    else:
        l = min(window_start_from_prose(j, d), l_s - w_s)
        sinks = min(n_ss, l_s)
        speech = w_s + sinks - max(0, min(sinks, l + w_s) - l)  # |[0,sinks) U [l,l+w)|
    if w_o == OFF or w_o >= j:
        out = j
    else:
        out = min(j, min(n_so, j) + w_o)  # Algorithm 1: sinks 1..n plus the last w tokens
    return p_pre + p_mid + speech + out


layouts = st.tuples(st.integers(0, 6), st.integers(0, 40), st.integers(0, 5), st.integers(1, 60))
policies = st.tuples(st.one_of(st.just(OFF), st.integers(1, 45)), st.integers(0, 30), st.integers(0, 8),
                     st.one_of(st.just(OFF), st.integers(1, 70)), st.integers(0, 8))


@settings(max_examples=400, deadline=None)
@given(layouts, policies)
def test_count_closed_form(seg, pol):
    idx, cnt = one(list(seg), list(pol))
    assert cnt == closed_form_count(seg, pol)


@settings(max_examples=300, deadline=None)
@given(layouts, policies)
def test_structure(seg, pol):
    """Ascending, unique, in range; prompts and the current token always kept; speech kept set is
    sinks plus one contiguous window; output kept set is sinks plus the most recent tokens."""
    p_pre, l_s, p_mid, j = seg
    w_s, d, n_ss, w_o, n_so = pol
    idx, cnt = one(list(seg), list(pol))
    r = idx[:cnt]
    total = p_pre + l_s + p_mid + j
    assert np.all(np.diff(r) > 0) and (cnt == 0 or (r[0] >= 0 and r[-1] < total))
    kept = set(r.tolist())
    assert set(range(p_pre)) <= kept
    assert set(range(p_pre + l_s, p_pre + l_s + p_mid)) <= kept
    assert total - 1 in kept
    speech = sorted(p - p_pre for p in kept if p_pre <= p < p_pre + l_s)
    if w_s == OFF or w_s >= l_s:
        assert speech == list(range(l_s))
    else:
        assert set(range(min(n_ss, l_s))) <= set(speech)
        rest = [s for s in speech if s >= min(n_ss, l_s)]
        assert rest == list(range(rest[0], rest[0] + len(rest))) if rest else True
        assert len(speech) >= w_s
        assert max(speech) <= l_s - 1
    out0 = p_pre + l_s + p_mid
    out = sorted(p - out0 + 1 for p in kept if p >= out0)  # 1-based
    if w_o != OFF and w_o < j:
        recent = set(range(j - w_o + 1, j + 1))
        assert recent <= set(out)
        assert set(out) - recent == set(range(1, min(n_so, j) + 1)) - recent


def test_window_motion_matches_prose():
    """Speech window start read off the oracle's lists: 0 before the delay, then +1 per step
    (Equation 2's description), until it reaches the end of speech (clamp reading)."""
    p_pre, l_s, w, d = 4, 60, 16, 10
    starts = []
    for j in range(1, 80):
        idx, cnt = one([p_pre, l_s, 0, j], [w, d, 0, OFF, 0])
        speech = [p - p_pre for p in idx[:cnt] if p_pre <= p < p_pre + l_s]
        assert len(speech) == w
        starts.append(speech[0])
    for j, l in enumerate(starts, start=1):
        assert l == min(window_start_from_prose(j, d), l_s - w)
    assert starts[:d - 1] == [0] * (d - 1)
    assert starts[d - 1] == 1
    assert all(b - a in (0, 1) for a, b in zip(starts, starts[1:]))
    assert starts[-1] == l_s - w  # clamped: the window ends at the last speech token


def test_window_at_least_length_keeps_everything():
    for seg in ([3, 20, 2, 9], [0, 5, 0, 1], [7, 0, 3, 4]):
        total = sum(seg)
        for pol in ([seg[1], 0, 0, seg[3], 0], [seg[1] + 5, 3, 2, seg[3] + 1, 1], [OFF, 0, 0, OFF, 0]):
            if pol[0] == 0:
                continue
            idx, cnt = one(seg, pol)
            assert cnt == total and np.array_equal(idx[:cnt], np.arange(total))


def test_speech_count_independent_of_delay():
    counts = set()
    for d in (0, 1, 5, 17, 40):
        for j in (1, 8, 30):
            _, cnt = one([2, 50, 1, j], [12, d, 0, OFF, 0])
            counts.add(cnt - 2 - 1 - j)
    assert counts == {12}


def test_output_sinks_and_window():
    # Algorithm 1 with n_sink = 2, w = 3 at j = 10: 1-based {1,2} U {8,9,10}.
    idx, cnt = one([1, 0, 0, 10], [OFF, 0, 0, 3, 2])
    assert idx[:cnt].tolist() == [0, 1, 2, 8, 9, 10]


def test_invalid_inputs_rejected():
    for seg, pol in (([0, 5, 0, 0], [OFF, 0, 0, OFF, 0]),    # j < 1
                     ([0, 5, 0, 3], [0, 0, 0, OFF, 0]),       # speech window 0
                     ([0, 5, 0, 3], [OFF, 0, 0, 0, 0]),       # output window 0
                     ([0, 5, 0, 3], [2, -1, 0, OFF, 0]),      # negative delay
                     ([-1, 5, 0, 3], [OFF, 0, 0, OFF, 0])):   # negative length
        with pytest.raises(ValueError):
            one(seg, pol)


def test_max_keep_too_small_rejected():
    with pytest.raises(ValueError):
        oracle.retained(np.array([[4, 10, 0, 3]]), np.array([OFF, 0, 0, OFF, 0]), max_keep=5)


def test_per_sequence_policy():
    seg = np.array([[2, 30, 0, 20], [2, 30, 0, 20]])
    pol = np.array([[8, 0, 0, OFF, 0], [OFF, 0, 0, 4, 1]])
    idx, cnt = oracle.retained(seg, pol)
    assert cnt.tolist() == [2 + 8 + 20, 2 + 30 + 5]
