"""Device-resident decode batch: uploads a workload once and runs the two C-ABI calls per step.

Memory plumbing only (torch allocates, the HIP kernels compute):
  * K/V caches [R][NL][B][Hkv][max_len][D] bf16, R identical replicas so that
    consecutive timed steps can read different addresses (cold caches);
  * per-step layouts [steps][B][4] and queries [steps][NL][B][Hq][D];
  * retained lists, counts, range tables, outputs and the split workspace.
A step is murmur_evict_compact followed by murmur_decode_attn, or the single
murmur_decode_step launch, enqueued on the current torch stream with no host
synchronisation.
"""
from __future__ import annotations

import numpy as np
import torch

from . import murmur as M
from .workloads import Workload


def pol_mode(policy: np.ndarray) -> int:
    """MURMUR_POL_* bits of a workload's policy array: [B, 5] per sequence, [NL, B, 5] per layer too."""
    return M.MURMUR_POL_PER_SEQ | (M.MURMUR_POL_PER_LAYER if np.ndim(policy) == 3 else 0)


def layer_policies(wl: Workload) -> list[np.ndarray]:
    """The [B, 5] policy of every layer."""
    if np.ndim(wl.policy) == 3:
        return [wl.policy[layer] for layer in range(wl.n_layers)]
    return [wl.policy] * wl.n_layers


def retained_counts(wl: Workload, step: int) -> np.ndarray:
    """Retained counts [NL, B] at a step, from the host closed form (murmur_retained_count_host)."""
    seg = wl.seg(step)
    return np.stack([M.murmur_retained_count_host(seg, pol, 1)[0] for pol in layer_policies(wl)])


class DecodeBatch:
    def __init__(self, wl: Workload, device: str = "cuda", replicas: int = 1, out_dtype: int = M.MURMUR_DTYPE_BF16,
                 split_len: int = 0, use_ranges: bool = True, steps: list[int] | None = None,
                 max_keep: int | None = None):
        self.wl = wl
        self.device = torch.device(device)
        self.steps = list(range(wl.steps)) if steps is None else list(steps)
        self.out_dtype = out_dtype
        self.split_len = split_len
        self.use_ranges = use_ranges
        B, NL, Hq, Hkv, D = wl.batch, wl.n_layers, wl.hq, wl.hkv, wl.head_dim
        self.B, self.NL, self.Hq, self.Hkv, self.D = B, NL, Hq, Hkv, D

        # Sizing from the host closed form over every step this batch will run.
        self.pol_mode = pol_mode(wl.policy)
        self.per_layer = bool(self.pol_mode & M.MURMUR_POL_PER_LAYER)
        counts = [int(retained_counts(wl, s).max()) for s in self.steps]
        self.max_keep = int(max(counts)) if max_keep is None else int(max_keep)

        dev = self.device
        k = torch.from_numpy(wl.k).view(torch.bfloat16)
        v = torch.from_numpy(wl.v).view(torch.bfloat16)
        self.replicas = replicas
        self.k = torch.empty((replicas,) + tuple(k.shape), dtype=torch.bfloat16, device=dev)
        self.v = torch.empty_like(self.k)
        self.k[0].copy_(k)
        self.v[0].copy_(v)
        for r in range(1, replicas):
            self.k[r].copy_(self.k[0])
            self.v[r].copy_(self.v[0])
        self.kv = [M.kv_from_tensors(self.k[r], self.v[r]) for r in range(replicas)]

        self.seg = torch.from_numpy(np.stack([wl.seg(s) for s in self.steps]).astype(np.int32)).to(dev)
        self.pol = torch.from_numpy(np.ascontiguousarray(wl.policy, dtype=np.int32)).to(dev)
        self.q = torch.from_numpy(np.stack([wl.q(s) for s in self.steps])).view(torch.bfloat16).to(dev)

        # Two sets of retained-set buffers, so that the eviction of the next step can run while the
        # attention of the current one still reads its set.
        # (with per-layer policies the fused step writes one set per layer: [NL][B] rows)
        rows = NL * B if self.per_layer else B
        self.sets = [(torch.full((rows, self.max_keep), -1, dtype=torch.int32, device=dev),
                      torch.zeros(rows, dtype=torch.int32, device=dev),
                      torch.zeros((rows, M.N_PIECES, 2), dtype=torch.int32, device=dev)) for _ in range(2)]
        self.idx, self.count, self.ranges = self.sets[0]
        odt = torch.bfloat16 if out_dtype == M.MURMUR_DTYPE_BF16 else torch.float32
        self.out = torch.zeros((NL, B, Hq, D), dtype=odt, device=dev)
        self.lse = torch.zeros((NL, B, Hq), dtype=torch.float32, device=dev)
        self.ws_bytes = M.murmur_decode_attn_workspace(NL, B, Hq, Hkv, self.max_keep, split_len)
        self.ws = torch.zeros(max(self.ws_bytes, 256) // 4 + 64, dtype=torch.int32, device=dev)

    def evict(self, i: int, stream=None, buf: int = 0) -> None:
        """murmur_evict_compact for the i-th step of this batch into retained-set buffer `buf`."""
        if self.per_layer:
            raise ValueError("per-layer policies run on the fused step only")
        idx, count, ranges = self.sets[buf]
        M.murmur_evict_compact(self.seg[i], self.pol, 1, self.B, idx, self.max_keep, count, ranges, stream)

    def attend(self, i: int, replica: int = 0, stream=None, buf: int = 0) -> None:
        """murmur_decode_attn for the i-th step, reading K/V replica `replica` and retained-set buffer `buf`."""
        idx, count, ranges = self.sets[buf]
        M.murmur_decode_attn(self.q[i], self.kv[replica], idx, ranges if self.use_ranges else None, count,
                             self.max_keep, self.B, self.Hq, self.Hkv, self.D, self.wl.scale, self.split_len,
                             self.out, self.out_dtype, self.lse, self.ws, self.ws_bytes, stream)

    def step(self, i: int, replica: int = 0, stream=None) -> None:
        self.evict(i, stream)
        self.attend(i, replica, stream)

    def step_fused(self, i: int, replica: int = 0, stream=None, buf: int = 0, outputs: bool = True) -> None:
        """murmur_decode_step for the i-th step: eviction and attention in one launch, the retained-set
        outputs (index list, count, range table) written into buffer set `buf` when `outputs`."""
        idx, count, ranges = self.sets[buf] if outputs else (None, None, None)
        M.murmur_decode_step(self.seg[i], self.pol, self.pol_mode, self.q[i], self.kv[replica], idx, count, ranges,
                             self.max_keep, self.B, self.Hq, self.Hkv, self.D, self.wl.scale, self.split_len,
                             self.out, self.out_dtype, self.lse, self.ws, self.ws_bytes, stream)

    def pipelined_steps(self, steps: list[int], replicas: list[int], attn_stream, evict_stream) -> None:
        """Enqueue the given steps with the eviction of step k+1 overlapping the attention of step k.

        The retained set is a function of the layout alone, so the next step's set can be built while
        the current step attends; the two buffer sets alternate.  attention(k) waits for eviction(k);
        eviction(k+1) reuses the buffer attention(k-1) read and waits for it.  Both streams keep the
        default priority.  Ends with attn_stream waiting for evict_stream."""
        import torch
        n = len(steps)
        ev_evict = [torch.cuda.Event() for _ in range(n)]
        ev_attn = [torch.cuda.Event() for _ in range(n)]
        evict_stream.wait_stream(attn_stream)
        with torch.cuda.stream(evict_stream):
            self.evict(steps[0], buf=0)
            ev_evict[0].record(evict_stream)
        for k in range(n):
            attn_stream.wait_event(ev_evict[k])
            with torch.cuda.stream(attn_stream):
                self.attend(steps[k], replicas[k], buf=k % 2)
                ev_attn[k].record(attn_stream)
            if k + 1 < n:
                if k >= 1:
                    evict_stream.wait_event(ev_attn[k - 1])
                with torch.cuda.stream(evict_stream):
                    self.evict(steps[k + 1], buf=(k + 1) % 2)
                    ev_evict[k + 1].record(evict_stream)
        attn_stream.wait_stream(evict_stream)

    def kv_bytes_read(self, i: int) -> int:
        """Algorithmic K/V bytes of step i: retained positions of every layer x KV heads x (K + V) x D x 2 B."""
        return int(retained_counts(self.wl, self.steps[i]).sum()) * self.Hkv * 2 * self.D * 2

    def io_bytes(self) -> int:
        """Algorithmic bytes besides K/V: queries, outputs, lse, count and range table (or index list)."""
        out_b = 4 if self.out_dtype == M.MURMUR_DTYPE_F32 else 2
        n = self.NL * self.B * self.Hq
        if self.per_layer:  # the fused step reads layouts and per-layer policies
            return n * self.D * 2 + n * self.D * out_b + n * 4 + self.B * 16 + self.NL * self.B * 20
        sel = self.B * M.N_PIECES * 2 * 4 if self.use_ranges else self.B * self.max_keep * 4
        return n * self.D * 2 + n * self.D * out_b + n * 4 + self.B * 4 + sel


def ring_rows(seg_row, n_sink: int, cap: int) -> int:
    """Rows of ring storage one sequence needs: prompts, speech, output sinks and `cap` ring rows."""
    p_pre, l_s, p_mid, _ = (int(x) for x in seg_row)
    return p_pre + l_s + p_mid + int(n_sink) + int(cap)


def ring_prefill(cache: np.ndarray, seg: np.ndarray, n_sink: np.ndarray, cap: int, rows: int) -> np.ndarray:
    """Places a sequence-ordered cache [NL, B, Hkv, L, D] into ring storage [NL, B, Hkv, rows, D] as it
    stands after output tokens 0 .. out_len-1 have been appended (the layout of include/murmur.h's
    murmur_ring): prompts and speech in place, output sinks after them, and each of the last `cap`
    later tokens at its ring row.  Rows that hold no token are zero."""
    seg = np.asarray(seg).reshape(-1, 4)
    NL, B, Hkv, _, D = cache.shape
    st = np.zeros((NL, B, Hkv, rows, D), dtype=cache.dtype)
    for b in range(B):
        p_pre, l_s, p_mid, j = (int(x) for x in seg[b])
        out0, ns = p_pre + l_s + p_mid, int(n_sink[b])
        st[:, b, :, :out0] = cache[:, b, :, :out0]
        ks = min(ns, j)
        st[:, b, :, out0:out0 + ks] = cache[:, b, :, out0:out0 + ks]
        tok = np.arange(max(ns, j - cap), j)  # the ring tokens still in storage
        st[:, b, :, out0 + ns + (tok - ns) % cap] = cache[:, b, :, out0 + tok]
    return st


class RingBatch:
    """Decode steps on ring storage (murmur_decode_step_ring): eviction, attention and the append of the
    current token in one launch per step.

    Memory plumbing only: the ring storage [R][NL][B][Hkv][rows][D] (R replicas for cold reads), per-step
    layouts, queries and current-token K/V [steps][NL][B][Hkv][D], outputs and workspace.  `storage`
    (optional, uint16 bf16 bits [NL, B, Hkv, rows, D]) replaces the prefill of the first step's state."""

    def __init__(self, wl: Workload, cap: int, device: str = "cuda", replicas: int = 1,
                 out_dtype: int = M.MURMUR_DTYPE_BF16, split_len: int = 0, steps: list[int] | None = None,
                 storage: tuple[np.ndarray, np.ndarray] | None = None):
        self.wl = wl
        self.cap = int(cap)
        self.device = torch.device(device)
        self.steps = list(range(wl.steps)) if steps is None else list(steps)
        self.out_dtype = out_dtype
        self.split_len = split_len
        B, NL, Hq, Hkv, D = wl.batch, wl.n_layers, wl.hq, wl.hkv, wl.head_dim
        self.B, self.NL, self.Hq, self.Hkv, self.D = B, NL, Hq, Hkv, D
        self.pol_mode = pol_mode(wl.policy)
        n_sink = layer_policies(wl)[0][:, 4]  # the output sinks precede the ring: one count per sequence
        if any(not np.array_equal(p[:, 4], n_sink) for p in layer_policies(wl)):
            raise ValueError("ring storage needs the same output sink count in every layer")
        counts = [int(retained_counts(wl, s).max()) for s in self.steps]
        self.max_keep = int(max(counts))
        seg_before = wl.seg(self.steps[0])
        seg_before[:, 3] -= 1  # the state before the first step: its token is not appended yet
        self.rows = max(ring_rows(seg_before[b], n_sink[b], cap) for b in range(B))
        self.rows = (self.rows + 7) // 8 * 8
        if storage is None:
            storage = (ring_prefill(wl.k, seg_before, n_sink, cap, self.rows),
                       ring_prefill(wl.v, seg_before, n_sink, cap, self.rows))
        dev = self.device
        self.replicas = replicas
        k0 = torch.from_numpy(np.ascontiguousarray(storage[0])).view(torch.bfloat16)
        v0 = torch.from_numpy(np.ascontiguousarray(storage[1])).view(torch.bfloat16)
        self.k = torch.empty((replicas,) + tuple(k0.shape), dtype=torch.bfloat16, device=dev)
        self.v = torch.empty_like(self.k)
        for r in range(replicas):
            self.k[r].copy_(k0)
            self.v[r].copy_(v0)
        self.kv = [M.kv_from_tensors(self.k[r], self.v[r]) for r in range(replicas)]

        self.seg = torch.from_numpy(np.stack([wl.seg(s) for s in self.steps]).astype(np.int32)).to(dev)
        self.pol = torch.from_numpy(np.ascontiguousarray(wl.policy, dtype=np.int32)).to(dev)
        self.q = torch.from_numpy(np.stack([wl.q(s) for s in self.steps])).view(torch.bfloat16).to(dev)
        # The current token's K/V of every step, taken from the sequence-ordered cache.
        knew = np.empty((len(self.steps), NL, B, Hkv, D), dtype=np.uint16)
        vnew = np.empty_like(knew)
        for i, s in enumerate(self.steps):
            seg = wl.seg(s)
            for b in range(B):
                p = int(seg[b, 0] + seg[b, 1] + seg[b, 2] + seg[b, 3]) - 1
                knew[i, :, b] = wl.k[:, b, :, p]
                vnew[i, :, b] = wl.v[:, b, :, p]
        self.k_new = torch.from_numpy(knew).view(torch.bfloat16).to(dev)
        self.v_new = torch.from_numpy(vnew).view(torch.bfloat16).to(dev)
        self.ring = [M.make_ring(cap, self.k_new[i], self.v_new[i]) for i in range(len(self.steps))]

        rows = NL * B if self.pol_mode & M.MURMUR_POL_PER_LAYER else B
        self.idx = torch.full((rows, self.max_keep), -1, dtype=torch.int32, device=dev)
        self.count = torch.zeros(rows, dtype=torch.int32, device=dev)
        self.ranges = torch.zeros((rows, M.N_PIECES, 2), dtype=torch.int32, device=dev)
        odt = torch.bfloat16 if out_dtype == M.MURMUR_DTYPE_BF16 else torch.float32
        self.out = torch.zeros((NL, B, Hq, D), dtype=odt, device=dev)
        self.lse = torch.zeros((NL, B, Hq), dtype=torch.float32, device=dev)
        self.ws_bytes = M.murmur_decode_attn_workspace(NL, B, Hq, Hkv, self.max_keep, split_len)
        self.ws = torch.zeros(max(self.ws_bytes, 256) // 4 + 64, dtype=torch.int32, device=dev)

    def step(self, i: int, replica: int = 0, stream=None, outputs: bool = True) -> None:
        """murmur_decode_step_ring for the i-th step of this batch on storage replica `replica`."""
        idx, count, ranges = (self.idx, self.count, self.ranges) if outputs else (None, None, None)
        M.murmur_decode_step_ring(self.seg[i], self.pol, self.pol_mode, self.ring[i], self.q[i], self.kv[replica],
                                  idx, count,
                                  ranges, self.max_keep, self.B, self.Hq, self.Hkv, self.D, self.wl.scale,
                                  self.split_len, self.out, self.out_dtype, self.lse, self.ws, self.ws_bytes,
                                  stream)

    def resident_bytes(self) -> int:
        """Bytes of one replica of the ring storage (K and V)."""
        return 2 * self.k[0].numel() * 2


class PagedBatch:
    """Decode steps on a paged KV cache: one shared pool of blocks of `block_size` rows and a block table per
    sequence (a random placement of its blocks, seeded).  A step is murmur_evict_compact_paged (the retained
    set as pool rows) followed by murmur_decode_attn in index-list mode over the pool.

    Memory plumbing only: the pool [R][NL][rows][Hkv][D] ("flash": block, slot, head) or [R][NL][Hkv][rows][D]
    ("head"), R replicas for cold reads, the block table [B][max_blocks], per-step layouts and queries,
    outputs and workspace."""

    def __init__(self, wl: Workload, block_size: int = 16, layout: str = "flash", device: str = "cuda",
                 replicas: int = 1, out_dtype: int = M.MURMUR_DTYPE_BF16, split_len: int = 0,
                 steps: list[int] | None = None, seed: int = 0, spare_blocks: int = 7):
        if np.ndim(wl.policy) == 3:
            raise ValueError("paged steps take per-sequence policies")
        self.wl = wl
        self.bs = int(block_size)
        self.layout = layout
        self.device = torch.device(device)
        self.steps = list(range(wl.steps)) if steps is None else list(steps)
        self.out_dtype = out_dtype
        self.split_len = split_len
        B, NL, Hq, Hkv, D = wl.batch, wl.n_layers, wl.hq, wl.hkv, wl.head_dim
        self.B, self.NL, self.Hq, self.Hkv, self.D = B, NL, Hq, Hkv, D
        self.max_keep = int(max(int(retained_counts(wl, s).max()) for s in self.steps))
        last = wl.seg(self.steps[-1])
        self.lengths = last.sum(axis=1).astype(np.int64)  # positions each sequence fills by the last step
        per_seq = -(-self.lengths // self.bs)
        self.max_blocks = int(per_seq.max())
        self.n_blocks = int(per_seq.sum()) + spare_blocks
        rng = np.random.default_rng(seed)
        perm = rng.permutation(self.n_blocks)
        self.block_table = np.zeros((B, self.max_blocks), dtype=np.int32)
        o = 0
        for b in range(B):
            self.block_table[b, :per_seq[b]] = perm[o:o + per_seq[b]]
            o += int(per_seq[b])
        self.rows = self.n_blocks * self.bs
        dev = self.device
        self.replicas = replicas
        k0 = torch.from_numpy(self.pool(wl.k)).view(torch.bfloat16)
        v0 = torch.from_numpy(self.pool(wl.v)).view(torch.bfloat16)
        self.k = torch.empty((replicas,) + tuple(k0.shape), dtype=torch.bfloat16, device=dev)
        self.v = torch.empty_like(self.k)
        for r in range(replicas):
            self.k[r].copy_(k0)
            self.v[r].copy_(v0)
        if layout == "flash":
            strides = (self.rows * Hkv * D, 0, D, Hkv * D)
        else:
            strides = (Hkv * self.rows * D, 0, self.rows * D, D)
        self.kv = [M.make_kv(self.k[r], self.v[r], NL, self.rows, strides) for r in range(replicas)]
        self.bt = torch.from_numpy(self.block_table).to(dev)
        self.seg = torch.from_numpy(np.stack([wl.seg(s) for s in self.steps]).astype(np.int32)).to(dev)
        self.pol = torch.from_numpy(np.ascontiguousarray(wl.policy, dtype=np.int32)).to(dev)
        self.q = torch.from_numpy(np.stack([wl.q(s) for s in self.steps])).view(torch.bfloat16).to(dev)
        self.idx = torch.full((B, self.max_keep), -1, dtype=torch.int32, device=dev)
        self.count = torch.zeros(B, dtype=torch.int32, device=dev)
        odt = torch.bfloat16 if out_dtype == M.MURMUR_DTYPE_BF16 else torch.float32
        self.out = torch.zeros((NL, B, Hq, D), dtype=odt, device=dev)
        self.lse = torch.zeros((NL, B, Hq), dtype=torch.float32, device=dev)
        self.ws_bytes = M.murmur_decode_attn_workspace(NL, B, Hq, Hkv, self.max_keep, split_len)
        self.ws = torch.zeros(max(self.ws_bytes, 256) // 4 + 64, dtype=torch.int32, device=dev)

    def pool(self, cache: np.ndarray) -> np.ndarray:
        """The pool of a sequence-ordered cache [NL, B, Hkv, L, D] (positions up to each sequence's length)."""
        NL, B, Hkv, _, D = cache.shape
        flash = np.zeros((NL, self.rows, Hkv, D), dtype=cache.dtype)
        for b in range(B):
            n = int(self.lengths[b])
            for i in range(-(-n // self.bs)):
                lo, hi = i * self.bs, min((i + 1) * self.bs, n)
                r0 = int(self.block_table[b, i]) * self.bs
                flash[:, r0:r0 + hi - lo] = cache[:, b, :, lo:hi].transpose(0, 2, 1, 3)
        return flash if self.layout == "flash" else np.ascontiguousarray(flash.transpose(0, 2, 1, 3))

    def evict(self, i: int, stream=None) -> None:
        M.murmur_evict_compact_paged(self.seg[i], self.pol, 1, self.B, self.bt, self.max_blocks, self.bs, self.idx,
                                     self.max_keep, self.count, None, stream)

    def attend(self, i: int, replica: int = 0, stream=None) -> None:
        M.murmur_decode_attn(self.q[i], self.kv[replica], self.idx, None, self.count, self.max_keep, self.B,
                             self.Hq, self.Hkv, self.D, self.wl.scale, self.split_len, self.out, self.out_dtype,
                             self.lse, self.ws, self.ws_bytes, stream)

    def step(self, i: int, replica: int = 0, stream=None) -> None:
        self.evict(i, stream)
        self.attend(i, replica, stream)


class RecyclingPagedBatch:
    """Consecutive decode steps on a paged cache whose blocks are recycled: before each step the blocks that
    no later step retains (murmur_freeable_blocks_host) go back to a free list, and the blocks new positions
    need are taken from it, so the pool holds O(prompt + speech + output window) rows per sequence however
    long the decode runs.  A step is then murmur_evict_compact_paged + murmur_decode_attn (index list).

    Host-side block manager and memory plumbing only: the pool [NL][n_blocks * block_size][Hkv][D] ("flash"
    layout), the block table [B][max_blocks] (-1 = no block), the free list (a stack).  A block's rows are
    written from the workload's cache when the block is taken, and overwritten with bf16 NaN when it is
    freed (`poison`), so that a read of a freed block would show in the outputs."""

    BF16_NAN = 0x7FC0

    def __init__(self, wl: Workload, block_size: int, n_blocks: int, device: str = "cuda",
                 out_dtype: int = M.MURMUR_DTYPE_F32, split_len: int = 0, poison: bool = True):
        if np.ndim(wl.policy) == 3:
            raise ValueError("paged steps take per-sequence policies")
        self.wl = wl
        self.bs = int(block_size)
        self.n_blocks = int(n_blocks)
        self.rows = self.n_blocks * self.bs
        self.poison = poison
        self.out_dtype = out_dtype
        self.split_len = split_len
        B, NL, Hq, Hkv, D = wl.batch, wl.n_layers, wl.hq, wl.hkv, wl.head_dim
        self.B, self.NL, self.Hq, self.Hkv, self.D = B, NL, Hq, Hkv, D
        self.pol_np = np.ascontiguousarray(wl.policy, dtype=np.int32)
        final = wl.seg(wl.steps - 1)
        self.max_blocks = int((-(-final.sum(axis=1) // self.bs)).max())
        self.max_keep = int(max(int(retained_counts(wl, s).max()) for s in range(wl.steps)))
        self.table = np.full((B, self.max_blocks), -1, dtype=np.int32)
        self.free = list(range(self.n_blocks - 1, -1, -1))
        self.freed = np.zeros((B, self.max_blocks), dtype=bool)  # logical blocks already returned
        self.peak_in_use = 0
        dev = torch.device(device)
        self.k = torch.zeros((NL, self.rows, Hkv, D), dtype=torch.bfloat16, device=dev)
        self.v = torch.zeros_like(self.k)
        self.kv = M.make_kv(self.k, self.v, NL, self.rows, (self.rows * Hkv * D, 0, D, Hkv * D))
        self.bt = torch.from_numpy(self.table).to(dev)
        self.pol = torch.from_numpy(self.pol_np).to(dev)
        self.seg_dev = torch.zeros((B, 4), dtype=torch.int32, device=dev)
        self.q = torch.zeros((NL, B, Hq, D), dtype=torch.bfloat16, device=dev)
        self.idx = torch.full((B, self.max_keep), -1, dtype=torch.int32, device=dev)
        self.count = torch.zeros(B, dtype=torch.int32, device=dev)
        odt = torch.bfloat16 if out_dtype == M.MURMUR_DTYPE_BF16 else torch.float32
        self.out = torch.zeros((NL, B, Hq, D), dtype=odt, device=dev)
        self.lse = torch.zeros((NL, B, Hq), dtype=torch.float32, device=dev)
        self.ws_bytes = M.murmur_decode_attn_workspace(NL, B, Hq, Hkv, self.max_keep, split_len)
        self.ws = torch.zeros(max(self.ws_bytes, 256) // 4 + 64, dtype=torch.int32, device=dev)

    def in_use(self) -> int:
        return self.n_blocks - len(self.free)

    def _fill(self, b: int, blk: int, phys: int) -> None:
        lo = blk * self.bs
        hi = min(lo + self.bs, self.wl.max_len)
        r0 = phys * self.bs
        for dst, src in ((self.k, self.wl.k), (self.v, self.wl.v)):
            rows = np.ascontiguousarray(src[:, b, :, lo:hi].transpose(0, 2, 1, 3))
            dst[:, r0:r0 + hi - lo].copy_(torch.from_numpy(rows).view(torch.bfloat16))

    def _release(self, b: int, blk: int) -> None:
        phys = int(self.table[b, blk])
        self.table[b, blk] = -1
        self.freed[b, blk] = True
        if phys < 0:  # freeable before it was ever needed: never allocated
            return
        if self.poison:
            r0 = phys * self.bs
            self.k[:, r0:r0 + self.bs].view(torch.int16).fill_(self.BF16_NAN)
            self.v[:, r0:r0 + self.bs].view(torch.int16).fill_(self.BF16_NAN)
        self.free.append(phys)

    def prepare(self, step: int) -> np.ndarray:
        """Frees what `step` and later steps never read, then takes blocks for every position up to the
        current token.  Returns the freeable block ranges [B, 2, 2] of this step."""
        seg = self.wl.seg(step)
        blocks = M.murmur_freeable_blocks_host(seg, self.pol_np, self.bs, 1)
        for b in range(self.B):
            for first, n in blocks[b]:
                for blk in range(int(first), int(first) + int(n)):
                    if not self.freed[b, blk]:
                        self._release(b, blk)
        for b in range(self.B):
            n_blk = -(-int(seg[b].sum()) // self.bs)
            for blk in range(n_blk):
                if self.table[b, blk] < 0 and not self.freed[b, blk]:
                    if not self.free:
                        raise MemoryError(f"block pool of {self.n_blocks} blocks exhausted at step {step}")
                    phys = self.free.pop()
                    self.table[b, blk] = phys
                    self._fill(b, blk, phys)
        self.peak_in_use = max(self.peak_in_use, self.in_use())
        self.bt.copy_(torch.from_numpy(self.table))
        self.seg_dev.copy_(torch.from_numpy(seg))
        self.q.copy_(torch.from_numpy(self.wl.q(step)).view(torch.bfloat16))
        return blocks

    def step(self, step: int, stream=None) -> None:
        M.murmur_evict_compact_paged(self.seg_dev, self.pol, 1, self.B, self.bt, self.max_blocks, self.bs, self.idx,
                                     self.max_keep, self.count, None, stream)
        M.murmur_decode_attn(self.q, self.kv, self.idx, None, self.count, self.max_keep, self.B, self.Hq, self.Hkv,
                             self.D, self.wl.scale, self.split_len, self.out, self.out_dtype, self.lse, self.ws,
                             self.ws_bytes, stream)


class DevicePagedBatch:
    """Consecutive decode steps on a paged cache whose block manager runs on the device: per step,
    murmur_paged_step (free the blocks no later step reads, take a block for the current token, write its
    K/V), murmur_evict_compact_paged and murmur_decode_attn -- three launches and no host work, so a run of
    steps can be captured into one HIP graph.

    Memory plumbing only: the pool [NL][n_blocks * block_size][Hkv][D] ("flash" layout), the block table
    [B][max_blocks], the free stack [n_blocks] and its top, per-step layouts, queries and current-token K/V
    [steps][NL][B][Hkv][D].  The host prefill gives every position before step 0's current token a block
    (taken from the top of the stack, as the device takes them) and writes its rows."""

    def __init__(self, wl: Workload, block_size: int, n_blocks: int, device: str = "cuda",
                 out_dtype: int = M.MURMUR_DTYPE_F32, split_len: int = 0):
        if np.ndim(wl.policy) == 3:
            raise ValueError("paged steps take per-sequence policies")
        self.wl = wl
        self.bs = int(block_size)
        self.n_blocks = int(n_blocks)
        self.rows = self.n_blocks * self.bs
        self.out_dtype = out_dtype
        self.split_len = split_len
        B, NL, Hq, Hkv, D = wl.batch, wl.n_layers, wl.hq, wl.hkv, wl.head_dim
        self.B, self.NL, self.Hq, self.Hkv, self.D = B, NL, Hq, Hkv, D
        final = wl.seg(wl.steps - 1)
        self.max_blocks = int((-(-final.sum(axis=1) // self.bs)).max())
        self.max_keep = int(max(int(retained_counts(wl, s).max()) for s in range(wl.steps)))
        dev = torch.device(device)
        # host prefill: positions [0, len - 1) of step 0, blocks popped from the top of the stack
        table = np.full((B, self.max_blocks), -1, dtype=np.int32)
        stack = list(range(self.n_blocks))
        k = np.zeros((NL, self.rows, Hkv, D), dtype=np.uint16)
        v = np.zeros_like(k)
        seg0 = wl.seg(0)
        for b in range(B):
            n = int(seg0[b].sum()) - 1
            for blk in range(-(-n // self.bs)):
                if not stack:
                    raise MemoryError("the pool cannot hold the prefill")
                phys = stack.pop()
                table[b, blk] = phys
                lo, hi = blk * self.bs, min((blk + 1) * self.bs, n)
                r0 = phys * self.bs
                k[:, r0:r0 + hi - lo] = wl.k[:, b, :, lo:hi].transpose(0, 2, 1, 3)
                v[:, r0:r0 + hi - lo] = wl.v[:, b, :, lo:hi].transpose(0, 2, 1, 3)
        self.k = torch.from_numpy(k).view(torch.bfloat16).to(dev)
        self.v = torch.from_numpy(v).view(torch.bfloat16).to(dev)
        self.kv = M.make_kv(self.k, self.v, NL, self.rows, (self.rows * Hkv * D, 0, D, Hkv * D))
        self.bt = torch.from_numpy(table).to(dev)
        self.stack = torch.zeros(self.n_blocks, dtype=torch.int32, device=dev)
        self.stack[:len(stack)] = torch.tensor(stack, dtype=torch.int32, device=dev)
        self.top = torch.tensor([len(stack)], dtype=torch.int32, device=dev)
        self.pol = torch.from_numpy(np.ascontiguousarray(wl.policy, dtype=np.int32)).to(dev)
        self.seg = torch.from_numpy(np.stack([wl.seg(s) for s in range(wl.steps)]).astype(np.int32)).to(dev)
        self.q = torch.from_numpy(np.stack([wl.q(s) for s in range(wl.steps)])).view(torch.bfloat16).to(dev)
        cur = []  # current token's K/V of every step: [steps][NL][B][Hkv][D]
        for s in range(wl.steps):
            p = wl.seg(s).sum(axis=1) - 1
            cur.append((np.stack([wl.k[:, b, :, p[b]] for b in range(B)], axis=1),
                        np.stack([wl.v[:, b, :, p[b]] for b in range(B)], axis=1)))
        self.k_new = torch.from_numpy(np.stack([c[0] for c in cur])).view(torch.bfloat16).to(dev)
        self.v_new = torch.from_numpy(np.stack([c[1] for c in cur])).view(torch.bfloat16).to(dev)
        self.idx = torch.full((B, self.max_keep), -1, dtype=torch.int32, device=dev)
        self.count = torch.zeros(B, dtype=torch.int32, device=dev)
        odt = torch.bfloat16 if out_dtype == M.MURMUR_DTYPE_BF16 else torch.float32
        self.out = torch.zeros((NL, B, Hq, D), dtype=odt, device=dev)
        self.lse = torch.zeros((NL, B, Hq), dtype=torch.float32, device=dev)
        self.ws_bytes = M.murmur_decode_attn_workspace(NL, B, Hq, Hkv, self.max_keep, split_len)
        self.ws = torch.zeros(max(self.ws_bytes, 256) // 4 + 64, dtype=torch.int32, device=dev)

    def state(self) -> tuple:
        """Copies of everything a step changes (pool, table, stack, top)."""
        return tuple(t.clone() for t in (self.k, self.v, self.bt, self.stack, self.top))

    def restore(self, st: tuple) -> None:
        for t, s in zip((self.k, self.v, self.bt, self.stack, self.top), st):
            t.copy_(s)

    def manage(self, i: int, stream=None) -> None:
        """murmur_paged_step of step i (a full scan at the first step, after the host prefill)."""
        M.murmur_paged_step(self.seg[i], self.pol, 1, self.B, self.bt, self.max_blocks, self.bs, self.stack, self.top,
                            self.n_blocks, i == 0, self.kv, self.Hkv, self.k_new[i], self.v_new[i], stream)

    def step(self, i: int, stream=None) -> None:
        self.manage(i, stream)
        M.murmur_evict_compact_paged(self.seg[i], self.pol, 1, self.B, self.bt, self.max_blocks, self.bs, self.idx,
                                     self.max_keep, self.count, None, stream)
        M.murmur_decode_attn(self.q[i], self.kv, self.idx, None, self.count, self.max_keep, self.B, self.Hq, self.Hkv,
                             self.D, self.wl.scale, self.split_len, self.out, self.out_dtype, self.lse, self.ws,
                             self.ws_bytes, stream)
