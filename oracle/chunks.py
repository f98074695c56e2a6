"""Chunked inference of a long recording -- TEST INFRASTRUCTURE (oracle side).

Only ``tests/`` may import this module; it imports nothing from the GPU package.

Section 3.1 merges the speech segments a voice-activity detector finds, greedily, into chunks of at most
c seconds, and Equation 4 turns chunk-relative timestamps into absolute ones by adding the chunk's
offset, the sum of the lengths of the chunks before it, which the paper calls the chunk's start time in
the recording.  For that to hold the chunks must tile the recording from 0.  The reading implemented
here (the paper gives no finer rule): a chunk keeps taking whole segments while the next one ends within
c of the chunk's start; it then ends where that next segment begins, or c after its start if that comes
first, and the next chunk starts there (also when the chunk then holds only silence: a segment that fits
a chunk is never cut).  A segment longer than c is cut every c seconds.  The last chunk
ends at the recording's end or c after its start.

  * ``plan``        -- the chunks [(start, length)], stated per chunk: from a start t, find the last
                       segment that can join, then the end;
  * ``timestamps``  -- Equation 4 with the offsets summed by math.fsum.
"""
from __future__ import annotations

import math


def plan(segments: list[tuple[float, float]], audio_len: float, c: float) -> list[tuple[float, float]]:
    """Chunks (start, length) for sorted, non-overlapping segments [(start, end)] of a recording."""
    chunks = []
    t = 0.0
    k = 0  # first segment that does not end by t
    while k < len(segments):
        # segments k .. m end within c of the chunk start t
        m = k - 1
        while m + 1 < len(segments) and segments[m + 1][1] - t <= c:
            m += 1
        if m < k:  # the first pending segment does not end within c of t
            s, e = segments[k]
            # keep it whole if it fits a chunk of its own: the chunk ends where it begins (t < s then)
            end = s if (e - s <= c and s < t + c) else t + c
        elif m + 1 < len(segments):  # stop where the first segment that did not fit begins
            end = min(segments[m + 1][0], t + c)
        else:  # every segment is placed: the last chunk
            end = min(audio_len, t + c)
            chunks.append((t, end - t))
            return chunks
        chunks.append((t, end - t))
        t = end
        while k < len(segments) and segments[k][1] <= t:
            k += 1
    return chunks


def timestamps(t_local: list[float], chunk: list[int], lengths: list[float]) -> list[float]:
    """Equation 4: t = t_local + sum of the lengths of the chunks before the timestamp's chunk."""
    return [tl + math.fsum(lengths[:i]) for tl, i in zip(t_local, chunk)]
