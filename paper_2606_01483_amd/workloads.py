"""Seeded synthetic decode workloads shaped like the paper's (Section 4.1, Section 3.2).

This module only draws inputs.  It holds none of the method's arithmetic: no
retained-set rule and no attention.  The same arrays feed both the GPU path and
the fp64 oracle, which never regenerates them.

Shapes follow the paper's workloads: 300 s chunks at about 7.5 speech tokens/s
(2250 speech tokens, Equation 3's worked example), roughly 2700 output tokens
per 300 s chunk, recordings up to 60 min, a batch of chunks decoded together
(Section 3.1).  The decoder is GQA with 28 query heads, 4 KV heads and head_dim
128, in bf16.  The paper's audio and model weights are not used: K and V are
N(0,1) and queries N(0,1)/sqrt(128); on the eviction workloads about 5 % of the
speech keys are planted to align with their group's queries (+3 sigma logits)
to mimic the sparse speech attention the paper profiles (Section 2.3).

Every generator is numpy PCG64, seeded with 1000 + workload number, with one
independent stream per purpose so that e.g. drawing fewer steps does not change
the caches.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import math
import os

import numpy as np

HQ, HKV, HEAD_DIM = 28, 4, 128
PLANT_RHO = 0.8        # query/planted-direction correlation
PLANT_SHIFT = 3.0      # expected logit lift of a planted key, in units of the logit std
PLANT_FRACTION = 0.05  # share of speech positions planted per (layer, sequence, kv head)

# Stream identifiers (second SeedSequence word).
_S_LAYOUT, _S_K, _S_V, _S_PLANT, _S_Q = 1, 2, 3, 4, 5

BF16_NAN = np.uint16(0x7FC0)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); returns uint16 bit patterns."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    odd = (u >> np.uint32(16)) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += odd
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, *extra])))


@dataclasses.dataclass
class Workload:
    """One synthetic decode job.

    seg0:   int32 [B, 4] (prompt_pre, speech_len, prompt_mid, out_len) before step 0;
            at step s the current token is output number out_len0 + s + 1.
    policy: int32 [B, 5] (speech_window, speech_delay, speech_sink, out_window, out_sink),
            or [NL, B, 5] for a policy per layer.
    k, v:   uint16 bf16 bits [NL, B, Hkv, max_len, D]; positions past a sequence's
            last step hold bf16 NaN, so reading them cannot go unnoticed.
    """
    name: str
    seed: int
    n_layers: int
    batch: int
    hq: int
    hkv: int
    head_dim: int
    steps: int
    seg0: np.ndarray
    policy: np.ndarray
    k: np.ndarray
    v: np.ndarray
    planted: bool
    scale: float = 1.0
    q_scale: float = 1.0 / math.sqrt(HEAD_DIM)
    plant_dir: np.ndarray | None = None   # float32 [NL, B, Hkv, D] unit directions (planted workloads)

    @property
    def max_len(self) -> int:
        return int(self.k.shape[3])

    def seg(self, step: int) -> np.ndarray:
        """Layout at decode step `step` (0-based): out_len = out_len0 + step + 1."""
        s = self.seg0.copy()
        s[:, 3] += step + 1
        return s

    def q(self, step: int) -> np.ndarray:
        """Queries of decode step `step`: uint16 bf16 bits [NL, B, Hq, D]."""
        rng = _rng(self.seed, _S_Q, step)
        x = rng.standard_normal((self.n_layers, self.batch, self.hq, self.head_dim), dtype=np.float32)
        if self.planted:
            group = self.hq // self.hkv
            m = np.repeat(self.plant_dir, group, axis=2) * np.float32(math.sqrt(self.head_dim))
            x = np.float32(math.sqrt(1.0 - PLANT_RHO ** 2)) * x + np.float32(PLANT_RHO) * m
        return f32_to_bf16_bits(x * np.float32(self.q_scale))


def _draw_cache(seed: int, stream: int, shape: tuple[int, ...]) -> np.ndarray:
    """N(0,1) bf16 bits.  Each (layer, sequence) slab has its own stream, so the result does not depend
    on how many threads draw it (numpy releases the GIL while filling and converting)."""
    out = np.empty(shape, dtype=np.uint16)

    def fill(lb: tuple[int, int]) -> None:
        layer, b = lb
        rng = _rng(seed, stream, layer, b)
        out[layer, b] = f32_to_bf16_bits(rng.standard_normal(shape[2:], dtype=np.float32))

    jobs = [(layer, b) for layer in range(shape[0]) for b in range(shape[1])]
    workers = max(1, min(16, len(os.sched_getaffinity(0)), len(jobs)))
    with concurrent.futures.ThreadPoolExecutor(workers) as pool:
        list(pool.map(fill, jobs))
    return out


def build(name: str, seed: int, n_layers: int, seg0: np.ndarray, policy: np.ndarray, steps: int,
          planted: bool, hq: int = HQ, hkv: int = HKV, head_dim: int = HEAD_DIM,
          scale: float = 1.0, q_scale: float | None = None) -> Workload:
    """Draw caches for an explicit layout.  seg0 [B,4], policy [5] or [B,5]."""
    seg0 = np.ascontiguousarray(seg0, dtype=np.int32).reshape(-1, 4)
    B = seg0.shape[0]
    policy = np.ascontiguousarray(policy, dtype=np.int32)
    if policy.ndim == 1:
        policy = np.repeat(policy.reshape(1, 5), B, axis=0)
    if policy.ndim == 3 and policy.shape != (n_layers, B, 5):
        raise ValueError("a per-layer policy is [n_layers, B, 5]")
    final_len = seg0[:, 0].astype(np.int64) + seg0[:, 1] + seg0[:, 2] + seg0[:, 3] + steps
    max_len = int(final_len.max())
    max_len = (max_len + 7) // 8 * 8
    shape = (n_layers, B, hkv, max_len, head_dim)
    k = _draw_cache(seed, _S_K, shape)
    v = _draw_cache(seed, _S_V, shape)
    plant_dir = None
    if planted:
        rng = _rng(seed, _S_PLANT)
        m = rng.standard_normal((n_layers, B, hkv, head_dim), dtype=np.float32)
        plant_dir = (m / np.linalg.norm(m, axis=-1, keepdims=True)).astype(np.float32)
        lift = np.float32(PLANT_SHIFT / PLANT_RHO)
        for layer in range(n_layers):
            for b in range(B):
                p_pre, l_s = int(seg0[b, 0]), int(seg0[b, 1])
                n_plant = int(round(PLANT_FRACTION * l_s))
                for g in range(hkv):
                    pos = p_pre + rng.choice(l_s, size=n_plant, replace=False)
                    z = bf16_bits_to_f32(k[layer, b, g, pos])
                    k[layer, b, g, pos] = f32_to_bf16_bits(z + lift * plant_dir[layer, b, g])
    for b in range(B):  # poison the tail past the last step of each sequence
        k[:, b, :, final_len[b]:, :] = BF16_NAN
        v[:, b, :, final_len[b]:, :] = BF16_NAN
    return Workload(name=name, seed=seed, n_layers=n_layers, batch=B, hq=hq, hkv=hkv, head_dim=head_dim,
                    steps=steps, seg0=seg0, policy=policy, k=k, v=v, planted=planted, scale=scale,
                    q_scale=(1.0 / math.sqrt(head_dim)) if q_scale is None else q_scale, plant_dir=plant_dir)


OFF = -1  # window value that disables eviction for a region


@dataclasses.dataclass
class Layout:
    """Sizes and policy of a workload without its caches (enough for the retained sets)."""
    name: str
    seed: int
    n_layers: int
    steps: int
    seg0: np.ndarray
    policy: np.ndarray
    planted: bool

    def seg(self, step: int) -> np.ndarray:
        s = self.seg0.copy()
        s[:, 3] += step + 1
        return s


def make(config: str, steps: int | None = None) -> Workload:
    """The five workloads of the evaluation, with caches drawn (see layout())."""
    lay = layout(config, steps)
    return build(lay.name, lay.seed, lay.n_layers, lay.seg0, lay.policy, lay.steps, planted=lay.planted)


def layout(config: str, steps: int | None = None) -> Layout:
    """The five workloads of the evaluation.

    c1        Tiny: 1 layer, batch 1, 32 prompt + 450 speech (60 s) + 64 output tokens,
              16 steps, speech window 128 (delay 72), output window 32.
    c2        12 x 300 s chunks, 1 layer: 32 prompt + 2250 speech + U{600..1200} output
              tokens, 64 steps, no eviction (dense decode baseline).
    c3        c2 with eviction: speech window 562 (25 % of 2250) with delay 512,
              output window 256; ~5 % planted speech keys.
    c4_dense  single-pass hour, 1 layer, batch 1: 32 + 27000 speech + 8000 output, 128 steps, dense.
    c4_evict  the same with speech window 2048 (delay 512) and output window 512.
    c5        28 layers x 12 chunks: speech U{1800..2250}, output U{300..1200}, speech window
              floor(L_s/4) (delay 512), output window 256, planted keys, 256 steps.
    c5_layers c5 with its first 4 layers dense (no eviction) and the c5 policy on the other 24.
    """
    if config == "c1":
        seed = 1001
        seg0 = np.array([[32, 450, 0, 64]], dtype=np.int32)
        pol = np.array([128, 72, 0, 32, 0], dtype=np.int32)
        return _layout("c1", seed, 1, seg0, pol, steps or 16, planted=False)
    if config in ("c2", "c3"):
        seed = 1002 if config == "c2" else 1003
        rng = _rng(seed, _S_LAYOUT)
        out0 = rng.integers(600, 1200, size=12, endpoint=True)
        seg0 = np.stack([np.full(12, 32), np.full(12, 2250), np.zeros(12), out0], axis=1).astype(np.int32)
        if config == "c2":
            pol = np.array([OFF, 0, 0, OFF, 0], dtype=np.int32)
            return _layout("c2", seed, 1, seg0, pol, steps or 64, planted=False)
        pol = np.array([2250 // 4, 512, 0, 256, 0], dtype=np.int32)
        return _layout("c3", seed, 1, seg0, pol, steps or 64, planted=True)
    if config in ("c4_dense", "c4_evict"):
        seed = 1004
        seg0 = np.array([[32, 27000, 0, 8000]], dtype=np.int32)
        if config == "c4_dense":
            pol = np.array([OFF, 0, 0, OFF, 0], dtype=np.int32)
        else:
            pol = np.array([2048, 512, 0, 512, 0], dtype=np.int32)
        return _layout(config, seed, 1, seg0, pol, steps or 128, planted=False)
    if config == "c5":
        seed = 1005
        rng = _rng(seed, _S_LAYOUT)
        l_s = rng.integers(1800, 2250, size=12, endpoint=True)
        out0 = rng.integers(300, 1200, size=12, endpoint=True)
        seg0 = np.stack([np.full(12, 32), l_s, np.zeros(12), out0], axis=1).astype(np.int32)
        pol = np.stack([l_s // 4, np.full(12, 512), np.zeros(12), np.full(12, 256), np.zeros(12)],
                       axis=1).astype(np.int32)
        return _layout("c5", seed, 28, seg0, pol, steps or 256, planted=True)
    if config == "c5_layers":
        # c5 with the first DENSE_LAYERS layers dense: the paper finds the speech sparsity on 24 of the
        # 28 layers (Section 1, Section 2.3), strongest in the deeper ones.
        base = layout("c5", steps)
        pol = np.repeat(base.policy[None], base.n_layers, axis=0)
        pol[:DENSE_LAYERS] = np.array([OFF, 0, 0, OFF, 0], dtype=np.int32)
        return Layout(name="c5_layers", seed=base.seed, n_layers=base.n_layers, steps=base.steps, seg0=base.seg0,
                      policy=pol, planted=True)
    raise KeyError(f"unknown workload {config!r}")


def _layout(name, seed, n_layers, seg0, pol, steps, planted) -> Layout:
    seg0 = np.ascontiguousarray(seg0, dtype=np.int32)
    pol = np.ascontiguousarray(pol, dtype=np.int32)
    if pol.ndim == 1:
        pol = np.repeat(pol.reshape(1, 5), seg0.shape[0], axis=0)
    return Layout(name=name, seed=seed, n_layers=n_layers, steps=steps, seg0=seg0, policy=pol, planted=planted)


CONFIGS = ("c1", "c2", "c3", "c4_dense", "c4_evict", "c5")
DENSE_LAYERS = 4
EXTRA_CONFIGS = ("c5_layers",)  # per-layer policies: fused steps only

# Eviction policies of the paper's ablations, all on 300 s chunks decoded in a batch of 16 (Section 4,
# Tables 2-4): (speech_window, speech_delay, speech_sink, out_window, out_sink).  Table 3 varies
# Algorithm 1's sinks / window; Table 4 Algorithm 2's delay / window (its "S / W" columns); Table 2
# combines output s4 w1024 with speech d512 w1024.
ABLATION_PRESETS = {
    "full": (OFF, 0, 0, OFF, 0),
    "out s4 w1024": (OFF, 0, 0, 1024, 4),
    "out s4 w512": (OFF, 0, 0, 512, 4),
    "out s4 w256": (OFF, 0, 0, 256, 4),
    "out s8 w1024": (OFF, 0, 0, 1024, 8),
    "out s8 w512": (OFF, 0, 0, 512, 8),
    "out s8 w256": (OFF, 0, 0, 256, 8),
    "speech d256 w1024": (1024, 256, 0, OFF, 0),
    "speech d256 w1538": (1538, 256, 0, OFF, 0),
    "speech d512 w1024": (1024, 512, 0, OFF, 0),
    "speech d512 w1538": (1538, 512, 0, OFF, 0),
    "both: out s4 w1024 + speech d512 w1024": (1024, 512, 0, 1024, 4),
}
ABLATION_BATCH = 16
ABLATION_OUTPUTS = 2700  # output tokens per 300 s chunk (Equation 3's example)


def ablation_workload(preset: str = "full", n_outputs: int = ABLATION_OUTPUTS) -> Workload:
    """A batch of 16 chunks of 300 s (32 prompt + 2250 speech tokens) decoded from the first output token
    to n_outputs under one of ABLATION_PRESETS; step s generates output token s + 1.  The caches do not
    depend on the preset (same seed), so presets can share one draw via with_policy()."""
    seg0 = np.tile(np.array([[32, 2250, 0, 0]], dtype=np.int32), (ABLATION_BATCH, 1))
    return build("ablation", 1006, 1, seg0, np.array(ABLATION_PRESETS[preset], dtype=np.int32), n_outputs,
                 planted=False)


def with_policy(wl: Workload, policy) -> Workload:
    """The same workload (same arrays) under another policy, [5] or [B, 5]."""
    pol = np.ascontiguousarray(policy, dtype=np.int32)
    if pol.ndim == 1:
        pol = np.repeat(pol.reshape(1, 5), wl.batch, axis=0)
    return dataclasses.replace(wl, policy=pol)


def large_cache(n_positions: int, seed: int, hkv: int = HKV, device: str = "cuda"):
    """K and V of one sequence of n_positions (a long-context stand-in far beyond the paper's hour-long
    recording, for tests at the largest sizes): N(0,1) rounded to bf16, drawn on the device from a seeded
    torch generator one KV head at a time, since a host draw of this size takes minutes.  Returns torch bf16
    tensors [1, 1, hkv, n_positions, 128]."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    k = torch.empty((1, 1, hkv, n_positions, HEAD_DIM), dtype=torch.bfloat16, device=device)
    v = torch.empty_like(k)
    for h in range(hkv):
        for t in (k, v):
            t[0, 0, h].copy_(torch.randn((n_positions, HEAD_DIM), generator=gen, device=device, dtype=torch.float32))
    return k, v
