"""Seeded synthetic decode workloads for SPLA (inputs only).

This module produces the query, key and value tensors that both the fp64
oracle and the HIP library consume. It holds none of the method's arithmetic:
only random draws, the structure planted into the keys (block offsets,
heavy-tailed block norms, planted relevant blocks, drifting block means) and
the rounding of the draws to the storage dtype (bfloat16, round to nearest
even), which fixes the exact input values both sides see.

Every token's key and value depend only on (seed, workload, sequence, KV
head, token position): tokens are drawn in independently seeded chunks of
CHUNK positions, so any slicing of a sequence (bulk append, per-step append,
sampled check) sees the same values.

RNG streams (numpy default_rng seeded with a list of ints):
  [seed, code, 0, b, step]      queries of sequence b at decode step `step`
  [seed, code, 1, b, h, c]      key noise, chunk c
  [seed, code, 2, b, h, c]      value noise, chunk c
  [seed, code, 3, b, h]         per-block key offsets
  [seed, code, 4, b, h]         planted block positions
  [seed, code, 5, b, h]         per-block value offsets
  [seed, code, 6]               per-sequence lengths
  [seed, code, 7]               RMSNorm weight
"""

from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace
from functools import lru_cache
from typing import Optional

import numpy as np

CHUNK = 4096

@dataclass(frozen=True)
class Workload:
    """Shape, structure and seed of one synthetic decode workload.

    lengths[b] is the number of cached tokens sequence b holds when it is
    decoded (for workloads that append one token per step, that count
    includes the token appended by the first step). capacity is the
    per-sequence cache size.
    """

    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    block_size: int
    top_k: int
    capacity: int
    lengths: tuple
    dtype: str  # "f32" or "bf16"
    kind: str
    code: int
    seed: int = 0
    n_sink: int = 1
    n_local: int = 4
    n_planted: int = 0
    plant_scale: float = 2.0
    pareto_alpha: float = 1.5
    pareto_xm: float = 0.25
    offset_std: float = 0.5
    drift_std: float = 0.05
    appends_per_step: int = 0

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def n_blocks(self, b: int) -> int:
        return -(-int(self.lengths[b]) // self.block_size)

    @property
    def max_blocks(self) -> int:
        return -(-self.capacity // self.block_size)

    def prefill_length(self, b: int) -> int:
        """Tokens appended in bulk before the first decode step."""
        return int(self.lengths[b]) - self.appends_per_step


def _lengths_uniform(seed: int, code: int, batch: int, lo: int, hi: int) -> tuple:
    rng = np.random.default_rng([seed, code, 6])
    return tuple(int(x) for x in rng.integers(lo, hi + 1, size=batch))


def config(i, seed: int = 0, **overrides) -> Workload:
    """The five decode workloads (and "g5", the paper's own G = 5 shape).

    1: fp32, b=1, 1 q / 1 kv head, d=64, L=4096, B=64, k=8; i.i.d. N(0,1)
       with two planted blocks (keys + 2 q/|q|).
    2: bf16, b=8, 32 q / 8 kv, d=128, L=32768, B=64, k=16; N(0,1) plus
       per-block offsets N(0, 0.5^2) for keys and (independently) values.
    3: bf16, b=4, 32/8, d=128, L=131072, B=64, k=32; keys N(0,1) plus a
       per-block offset r_i u_i (u_i uniform on the sphere, r_i Pareto with
       alpha 1.5 and scale 0.25) and 8 planted blocks per (b, kv head)
       shifted by 2 * (normalised group-mean query).
    4: bf16, b=64, 32/8, d=128, capacity 65536, lengths U{16384..65024},
       B=128, k=16; N(0,1); one token appended per decode step.
    5: bf16, b=1, 64/8, d=128, L=2^20, B=64, k=64; keys N(0,1) plus block
       means following a random walk with N(0, 0.05^2) steps.
    g5: as 3 with 40 q heads over 8 kv heads (G = 5), i.i.d. keys.
    """
    key = str(i)
    if key == "1":
        w = Workload("cfg1_tiny_fp32", 1, 1, 1, 64, 64, 8, 4096, (4096,), "f32", "planted_iid", 11,
                     seed=seed, n_planted=2)
    elif key == "2":
        w = Workload("cfg2_gqa_32k", 8, 32, 8, 128, 64, 16, 32768, (32768,) * 8, "bf16",
                     "block_offsets", 12, seed=seed)
    elif key == "3":
        w = Workload("cfg3_long_128k", 4, 32, 8, 128, 64, 32, 131072, (131072,) * 4, "bf16",
                     "pareto_planted", 13, seed=seed, n_planted=8)
    elif key == "4":
        lens = _lengths_uniform(seed, 14, 64, 16384, 65536 - 512)
        w = Workload("cfg4_batch64_var", 64, 32, 8, 128, 128, 16, 65536, lens, "bf16", "iid", 14,
                     seed=seed, appends_per_step=1)
    elif key == "5":
        w = Workload("cfg5_1m_single", 1, 64, 8, 128, 64, 64, 1 << 20, (1 << 20,), "bf16",
                     "drift", 15, seed=seed)
    elif key == "g5":
        w = Workload("g5_paper_model_128k", 1, 40, 8, 128, 64, 32, 131072, (131072,), "bf16", "iid",
                     16, seed=seed)
    else:
        raise ValueError(f"unknown workload {i!r}")
    return replace(w, **overrides) if overrides else w


def custom(name: str, batch: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
           block_size: int, top_k: int, lengths, dtype: str = "bf16", kind: str = "iid",
           capacity: Optional[int] = None, seed: int = 0, code: int = 99, **kw) -> Workload:
    """A workload of any shape (used by the tests for ragged and edge cases)."""
    lengths = tuple(int(x) for x in lengths)
    if capacity is None:
        capacity = max(max(lengths), 1)
        capacity = -(-capacity // block_size) * block_size
    return Workload(name, batch, n_q_heads, n_kv_heads, head_dim, block_size, top_k, capacity,
                    lengths, dtype, kind, code, seed=seed, **kw)


# --------------------------------------------------------------- rounding
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); the
    result is float32 holding bfloat16-representable values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def _store(w: Workload, x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    return round_bf16(x) if w.dtype == "bf16" else x


# ---------------------------------------------------------------- queries
def gen_q(w: Workload, b: int, step: int = 0) -> np.ndarray:
    """Query heads of sequence b at decode step `step`: [Hq, d], N(0, 1)."""
    rng = np.random.default_rng([w.seed, w.code, 0, b, step])
    return _store(w, rng.standard_normal((w.n_q_heads, w.head_dim), dtype=np.float32))


def gen_q_batch(w: Workload, step: int = 0) -> np.ndarray:
    return np.stack([gen_q(w, b, step) for b in range(w.batch)])


def gen_gamma(w: Workload, seed: int = 0, ones: bool = False) -> np.ndarray:
    """RMSNorm weight [Hq, d] (fp32): ones, or 1 + N(0, 0.1^2)."""
    if ones:
        return np.ones((w.n_q_heads, w.head_dim), dtype=np.float32)
    rng = np.random.default_rng([seed, w.code, 7])
    return (1.0 + 0.1 * rng.standard_normal((w.n_q_heads, w.head_dim))).astype(np.float32)


# -------------------------------------------------------------- structure
@lru_cache(maxsize=64)
def _key_offsets(w: Workload, b: int, h: int) -> Optional[np.ndarray]:
    nbc = w.max_blocks
    d = w.head_dim
    rng = np.random.default_rng([w.seed, w.code, 3, b, h])
    if w.kind == "block_offsets":
        return (w.offset_std * rng.standard_normal((nbc, d))).astype(np.float32)
    if w.kind == "pareto_planted":
        u = rng.standard_normal((nbc, d))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        r = w.pareto_xm * (1.0 + rng.pareto(w.pareto_alpha, size=nbc))
        return (r[:, None] * u).astype(np.float32)
    if w.kind == "drift":
        steps = w.drift_std * rng.standard_normal((nbc, d))
        steps[0] = 0.0
        return np.cumsum(steps, axis=0).astype(np.float32)
    return None


@lru_cache(maxsize=64)
def _value_offsets(w: Workload, b: int, h: int) -> Optional[np.ndarray]:
    if w.kind != "block_offsets":
        return None
    rng = np.random.default_rng([w.seed, w.code, 5, b, h])
    return (w.offset_std * rng.standard_normal((w.max_blocks, w.head_dim))).astype(np.float32)


def planted_blocks(w: Workload, b: int, h: int) -> np.ndarray:
    """Block ids that receive the planted shift: distinct, drawn from
    [n_sink, nb - n_local) so that they are never forced blocks."""
    if w.n_planted == 0:
        return np.zeros(0, dtype=np.int64)
    nb = w.n_blocks(b)
    lo, hi = w.n_sink, nb - w.n_local
    rng = np.random.default_rng([w.seed, w.code, 4, b, h])
    return np.sort(rng.choice(np.arange(lo, hi), size=w.n_planted, replace=False))


def plant_direction(w: Workload, b: int, h: int) -> np.ndarray:
    """Unit vector along the mean of the group's query heads (decode step 0)."""
    q = gen_q(w, b, 0)[h * w.group:(h + 1) * w.group].astype(np.float64).mean(axis=0)
    return (q / np.linalg.norm(q)).astype(np.float32)


# ---------------------------------------------------------------- K and V
def _chunk_kv(w: Workload, b: int, h: int, c: int):
    d = w.head_dim
    k = np.random.default_rng([w.seed, w.code, 1, b, h, c]).standard_normal((CHUNK, d),
                                                                           dtype=np.float32)
    v = np.random.default_rng([w.seed, w.code, 2, b, h, c]).standard_normal((CHUNK, d),
                                                                           dtype=np.float32)
    pos = np.arange(c * CHUNK, (c + 1) * CHUNK)
    blk = pos // w.block_size
    valid = blk < w.max_blocks
    ko = _key_offsets(w, b, h)
    if ko is not None:
        k[valid] += ko[blk[valid]]
    vo = _value_offsets(w, b, h)
    if vo is not None:
        v[valid] += vo[blk[valid]]
    planted = planted_blocks(w, b, h)
    if len(planted):
        shift = (w.plant_scale * plant_direction(w, b, h)).astype(np.float32)
        k[np.isin(blk, planted)] += shift
    return _store(w, k), _store(w, v)


def gen_kv(w: Workload, b: int, h: int, t0: int, t1: int, threads: int = 1):
    """Keys and values of tokens [t0, t1) of (sequence b, KV head h):
    two float32 arrays [t1 - t0, d] (bfloat16 values for bf16 workloads)."""
    d = w.head_dim
    if t1 <= t0:
        return np.zeros((0, d), np.float32), np.zeros((0, d), np.float32)
    c0, c1 = t0 // CHUNK, (t1 - 1) // CHUNK
    chunks = list(range(c0, c1 + 1))
    if threads > 1 and len(chunks) > 1:
        with ThreadPoolExecutor(threads) as ex:
            parts = list(ex.map(lambda c: _chunk_kv(w, b, h, c), chunks))
    else:
        parts = [_chunk_kv(w, b, h, c) for c in chunks]
    K = np.concatenate([p[0] for p in parts])
    V = np.concatenate([p[1] for p in parts])
    off = t0 - c0 * CHUNK
    return K[off:off + (t1 - t0)], V[off:off + (t1 - t0)]


def gen_kv_slab(w: Workload, t0: int, t1: int, lengths=None, threads: int = 8):
    """Keys and values of positions [t0, t1) for every (b, h):
    arrays [batch, Hkv, t1 - t0, d] (zeros past each sequence's `lengths`),
    and n_new[b] = number of valid positions of sequence b in the slab."""
    if lengths is None:
        lengths = w.lengths
    T = t1 - t0
    K = np.zeros((w.batch, w.n_kv_heads, T, w.head_dim), np.float32)
    V = np.zeros_like(K)
    n_new = np.array([max(0, min(T, int(lengths[b]) - t0)) for b in range(w.batch)], np.int32)
    jobs = [(b, h) for b in range(w.batch) for h in range(w.n_kv_heads) if n_new[b] > 0]

    # fewer (sequence, KV head) jobs than threads: each job splits its chunks
    inner = max(1, threads // max(1, len(jobs)))

    def run(job):
        b, h = job
        kk, vv = gen_kv(w, b, h, t0, t0 + int(n_new[b]), threads=inner)
        K[b, h, :n_new[b]] = kk
        V[b, h, :n_new[b]] = vv

    if threads > 1 and len(jobs) > 1:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(run, jobs))
    else:
        for j in jobs:
            run(j)
    return K, V, n_new


def algorithmic_bytes(w: Workload, sel_counts=None) -> dict:
    """Bytes the decode step must move (not part of the method): queries and
    outputs, every block's statistics (fp32 mean and M2), the selected key and
    value rows, and the fp32 global state; an appending step also writes the
    state back and touches one key/value row and one block's statistics.
    sel_counts[b][h] = tokens in the selected blocks (defaults to the
    expected count: k full blocks, or the whole sequence when nb <= k)."""
    e = 4 if w.dtype == "f32" else 2
    d, B = w.head_dim, w.block_size
    qo = 2 * w.batch * w.n_q_heads * d * e
    stats = sum(w.n_blocks(b) * 2 * d * 4 for b in range(w.batch)) * w.n_kv_heads
    sel = 0
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            if sel_counts is not None:
                n = int(sel_counts[b][h])
            else:
                n = min(w.top_k * B, int(w.lengths[b]))
            sel += n * d * 2 * e
    state = w.batch * w.n_kv_heads * d * d * 4
    extra = 0
    if w.appends_per_step:
        extra = w.batch * w.n_kv_heads * (d * d * 4 + 2 * d * e + 2 * 2 * d * 4 + 2 * d * 4)
    return {"q_out": qo, "stats": stats, "selected_kv": sel, "state": state, "append": extra,
            "total": qo + stats + sel + state + extra}


__all__ = ["CHUNK", "Workload", "config", "custom", "round_bf16", "gen_q", "gen_q_batch",
           "gen_gamma", "planted_blocks", "plant_direction", "gen_kv", "gen_kv_slab",
           "algorithmic_bytes"]
