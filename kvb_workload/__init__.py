"""Seeded synthetic workloads for the stitched-prefill path.

This module only *draws* inputs: random numbers with the shapes, value
distributions and structure of the five workloads (Qwen2.5-3B attention shape,
128-token chunks, KIVI int8/int4 pools, chunk re-placement, planted
deviation).  It holds none of the method's arithmetic: no RoPE, no
quantisation, no dequantisation, no deviation, no selection, no attention.
Each side that consumes these draws (the CPU oracle under ``oracle/`` and the
HIP library) turns them into rotated / quantised tensors with its own code.

Everything is produced with ``numpy.random.default_rng``:

* structure (chunk map, hit/miss choice, original offsets):
  ``default_rng([seed, 10**6])``
* layer ``l`` values: ``default_rng([seed, l])``, so one layer can be drawn on
  its own and a full 36-layer stack never has to sit in host memory at once.

Draws are taken in float64 and stored as float32.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import numpy as np

STRUCT_STREAM = 10**6


@dataclass(frozen=True)
class Workload:
    """One workload: model shape, cache format and prompt structure."""

    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    bits: int              # KIVI code width, 8 or 4
    k_group: int           # Gk: tokens per key-statistic group (keys are per channel)
    v_group: int           # Gv: channels per value-statistic group (values are per token)
    n_prompts: int
    chunks_per_prompt: int
    placement: str         # "permuted" | "identity" | "half_hits" | "prefix_hits" | "ramp_hits"
    n_sinks: int = 0
    seam_left: int = 0     # rows before each chunk boundary forced into the recompute set
    seam_right: int = 0    # rows after each chunk boundary forced into the recompute set
    rho_num: int = 15      # recompute fraction rho = rho_num / rho_den
    rho_den: int = 100
    per_layer: bool = True  # deviation and selection per layer (else one set for all layers)
    channel_scales: bool = True  # per-channel log-uniform scale in [0.1, 10]
    noise_num: int = 20    # fraction of candidate rows that carry planted deviation
    noise_den: int = 100
    noise_std: float = 0.1
    max_src_pos: int = 32768
    seed: int = 0
    chunk_len: int = 128
    hit_chunks: int = 0    # "prefix_hits": the first hit_chunks chunks of each prompt are cached
    # threshold-activated probe: a prompt whose cached fraction of rows is below
    # probe_min_num / probe_min_den skips the deviation pass (its top-k is empty)
    probe_min_num: int = 0
    probe_min_den: int = 100

    @property
    def prompt_len(self) -> int:
        return self.n_sinks + self.chunks_per_prompt * self.chunk_len

    @property
    def t_total(self) -> int:
        return self.n_prompts * self.prompt_len

    @property
    def group_size(self) -> int:
        return self.n_q_heads // self.n_kv_heads


# The five workloads.  Some details are choices made here, not given by the
# paper: the statistic group sizes, the seeds of the second and fourth
# workload, and the batched workload's hit placement (half of each prompt's
# chunks, cached at multiples of 128).
WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(
        name="tiny", n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64,
        rope_theta=1e4, bits=8, k_group=128, v_group=64, n_prompts=1,
        chunks_per_prompt=4, placement="permuted", channel_scales=False,
        max_src_pos=1, seed=0),
    "qwen_1l": Workload(
        name="qwen_1l", n_layers=1, n_q_heads=16, n_kv_heads=2, head_dim=128,
        rope_theta=1e6, bits=8, k_group=128, v_group=128, n_prompts=1,
        chunks_per_prompt=32, placement="identity", seam_left=16, seam_right=16,
        seed=3),
    "qwen_36l_8k": Workload(
        name="qwen_36l_8k", n_layers=36, n_q_heads=16, n_kv_heads=2, head_dim=128,
        rope_theta=1e6, bits=4, k_group=32, v_group=32, n_prompts=1,
        chunks_per_prompt=64, placement="identity", seed=1),
    "batched_mixed": Workload(
        name="batched_mixed", n_layers=1, n_q_heads=16, n_kv_heads=2, head_dim=128,
        rope_theta=1e6, bits=8, k_group=128, v_group=128, n_prompts=16,
        chunks_per_prompt=16, placement="half_hits", seed=4),
    "long_32k": Workload(
        name="long_32k", n_layers=36, n_q_heads=16, n_kv_heads=2, head_dim=128,
        rope_theta=1e6, bits=4, k_group=32, v_group=32, n_prompts=1,
        chunks_per_prompt=256, placement="identity", n_sinks=4, seam_left=16,
        seam_right=16, seed=2),
}
ORDER = ["tiny", "qwen_1l", "qwen_36l_8k", "batched_mixed", "long_32k"]


def scaled(w: Workload, **changes) -> Workload:
    """A copy of ``w`` with some fields replaced (smaller parity cases)."""
    d = dict(w.__dict__)
    d.update(changes)
    return Workload(**d)


@dataclass
class Structure:
    """Prompt layout and chunk map of a workload (identical for every layer).

    Rows are absolute indices into the ragged batch; prompt ``b`` owns rows
    ``cu_seqlens[b] .. cu_seqlens[b+1]-1`` and a row's position is its offset
    from ``cu_seqlens[b]``.

    Cached (hit) chunks are listed in pool order: pool slot ``i`` is placed at
    ``dst_row[i]`` (position ``dst_pos[i]``) and was cached at original
    position ``src_pos[i]``.  Rows of miss chunks and sink rows are live.
    """

    cu_seqlens: np.ndarray          # int32 [B+1]
    chunk_starts: List[np.ndarray]  # per prompt: in-prompt start positions of every chunk
    src_pos: np.ndarray             # int32 [P]
    dst_row: np.ndarray             # int32 [P]
    dst_pos: np.ndarray             # int32 [P]
    hit_row: np.ndarray             # bool [T]: row belongs to a cached chunk
    noise_rows: np.ndarray = field(default=None)  # filled per layer

    @property
    def n_pool(self) -> int:
        return int(self.src_pos.shape[0])

    def positions(self) -> np.ndarray:
        """Position of every row inside its own prompt (int32 [T])."""
        t = int(self.cu_seqlens[-1])
        pos = np.empty(t, dtype=np.int32)
        for b in range(len(self.cu_seqlens) - 1):
            lo, hi = int(self.cu_seqlens[b]), int(self.cu_seqlens[b + 1])
            pos[lo:hi] = np.arange(hi - lo, dtype=np.int32)
        return pos


def structure(w: Workload) -> Structure:
    rng = np.random.default_rng([w.seed, STRUCT_STREAM])
    C = w.chunk_len
    T_b = w.prompt_len
    cu = np.arange(w.n_prompts + 1, dtype=np.int64) * T_b
    src, dst_row, dst_pos = [], [], []
    hit = np.zeros(w.t_total, dtype=bool)
    starts = []
    for b in range(w.n_prompts):
        base = int(cu[b])
        chunk_pos = w.n_sinks + C * np.arange(w.chunks_per_prompt)
        starts.append(chunk_pos.astype(np.int32))
        if w.placement == "permuted":
            # pool slot i goes to chunk position perm[i]; every chunk was
            # cached at offset 0
            perm = rng.permutation(w.chunks_per_prompt)
            for i in range(w.chunks_per_prompt):
                p = int(chunk_pos[perm[i]])
                src.append(0)
                dst_pos.append(p)
                dst_row.append(base + p)
        elif w.placement == "identity":
            offs = rng.integers(0, w.max_src_pos, size=w.chunks_per_prompt)
            for i in range(w.chunks_per_prompt):
                p = int(chunk_pos[i])
                src.append(int(offs[i]))
                dst_pos.append(p)
                dst_row.append(base + p)
        elif w.placement in ("prefix_hits", "ramp_hits"):
            # a reused context: its leading chunks were cached at random offsets
            # ("ramp_hits": prompt b has floor(b * chunks / n_prompts) of them)
            if w.placement == "prefix_hits":
                n_hit = min(w.hit_chunks, w.chunks_per_prompt)
            else:
                n_hit = b * w.chunks_per_prompt // w.n_prompts
            offs = rng.integers(0, w.max_src_pos, size=n_hit)
            for i in range(n_hit):
                p = int(chunk_pos[i])
                src.append(int(offs[i]))
                dst_pos.append(p)
                dst_row.append(base + p)
        elif w.placement == "half_hits":
            order = rng.permutation(w.chunks_per_prompt)
            hits = np.sort(order[: w.chunks_per_prompt // 2])
            shifts = C * rng.integers(0, 256, size=hits.shape[0])
            for i, c in enumerate(hits):
                p = int(chunk_pos[c])
                src.append(int(shifts[i]))
                dst_pos.append(p)
                dst_row.append(base + p)
        else:
            raise ValueError(w.placement)
    src = np.asarray(src, dtype=np.int32)
    dst_row = np.asarray(dst_row, dtype=np.int32)
    dst_pos = np.asarray(dst_pos, dtype=np.int32)
    for r in dst_row:
        hit[int(r): int(r) + C] = True
    return Structure(cu_seqlens=cu.astype(np.int32), chunk_starts=starts,
                     src_pos=src, dst_row=dst_row, dst_pos=dst_pos, hit_row=hit)


@dataclass
class LayerDraws:
    """Raw (un-rotated, un-quantised) values of one layer, float32.

    ``k_pool_raw`` / ``v_pool_raw`` [P][Hkv][C][d]: content of each cached
    chunk before RoPE, i.e. the same underlying draw as the rows the chunk is
    placed on, without the planted deviation.  ``k_raw`` / ``v_raw``
    [Hkv][T][d] and ``q_raw`` [T][Hq][d]: the fresh (probe-pass) values before
    RoPE; rows in ``noise_rows`` carry ``noise_std * N(0,1)`` extra before the
    channel scale is applied.
    """

    k_pool_raw: np.ndarray
    v_pool_raw: np.ndarray
    k_raw: np.ndarray
    v_raw: np.ndarray
    q_raw: np.ndarray
    noise_rows: np.ndarray  # bool [T]


def _channel_scale(rng, shape):
    return np.exp(rng.uniform(np.log(0.1), np.log(10.0), size=shape))


def layer_draws(w: Workload, s: Structure, layer: int, with_q: bool = True) -> LayerDraws:
    rng = np.random.default_rng([w.seed, layer])
    H, Hq, d, T, C = w.n_kv_heads, w.n_q_heads, w.head_dim, w.t_total, w.chunk_len
    if w.channel_scales:
        sk = _channel_scale(rng, (H, 1, d))
        sv = _channel_scale(rng, (H, 1, d))
        sq = _channel_scale(rng, (1, Hq, d))
    else:
        sk = np.ones((H, 1, d))
        sv = np.ones((H, 1, d))
        sq = np.ones((1, Hq, d))
    zk = rng.standard_normal((H, T, d))
    zv = rng.standard_normal((H, T, d))
    # planted deviation: floor(noise_frac * n_b) candidate rows per prompt
    noise = np.zeros(T, dtype=bool)
    for b in range(w.n_prompts):
        lo, hi = int(s.cu_seqlens[b]), int(s.cu_seqlens[b + 1])
        cand = np.nonzero(s.hit_row[lo:hi])[0] + lo
        n = (w.noise_num * cand.shape[0]) // w.noise_den
        pick = rng.permutation(cand.shape[0])[:n]
        noise[cand[pick]] = True
    rows = np.nonzero(noise)[0]
    ek = w.noise_std * rng.standard_normal((H, rows.shape[0], d))
    ev = w.noise_std * rng.standard_normal((H, rows.shape[0], d))
    pool_idx = np.concatenate([np.arange(r, r + C) for r in s.dst_row]) if s.n_pool else np.zeros(0, np.int64)
    k_pool = (zk[:, pool_idx, :] * sk).reshape(H, s.n_pool, C, d).transpose(1, 0, 2, 3)
    v_pool = (zv[:, pool_idx, :] * sv).reshape(H, s.n_pool, C, d).transpose(1, 0, 2, 3)
    zk[:, rows, :] += ek
    zv[:, rows, :] += ev
    k_raw = zk * sk
    v_raw = zv * sv
    if with_q:
        q_raw = (rng.standard_normal((T, Hq, d)) * sq).astype(np.float32)
    else:
        q_raw = None
    return LayerDraws(
        k_pool_raw=np.ascontiguousarray(k_pool, dtype=np.float32),
        v_pool_raw=np.ascontiguousarray(v_pool, dtype=np.float32),
        k_raw=k_raw.astype(np.float32), v_raw=v_raw.astype(np.float32),
        q_raw=q_raw, noise_rows=noise)


def row_subset(w: Workload, s: Structure, n: int, seed: int) -> np.ndarray:
    """A sorted random subset of ``n`` rows (int32), for attention-only cases."""
    rng = np.random.default_rng([seed, 7])
    return np.sort(rng.choice(w.t_total, size=min(n, w.t_total), replace=False)).astype(np.int32)


def deviation_draw(n_sets: int, t_total: int, seed: int, n_levels: int = 0) -> np.ndarray:
    """Random per-row scores for exercising selection on its own.

    With ``n_levels > 0`` the scores are drawn from that many distinct values,
    so many rows tie exactly; some rows get ``-0.0`` and ``+0.0`` so both signs
    of zero are present.
    """
    rng = np.random.default_rng([seed, 11])
    if n_levels:
        levels = rng.uniform(0.0, 2.0, size=n_levels)
        out = levels[rng.integers(0, n_levels, size=(n_sets, t_total))]
    else:
        out = rng.uniform(0.0, 2.0, size=(n_sets, t_total))
    z = rng.random((n_sets, t_total)) < 0.02
    out[z] = 0.0
    neg = z & (rng.random((n_sets, t_total)) < 0.5)
    out = out.astype(np.float32)
    out[neg] = np.float32(-0.0)
    return out
