"""Helpers of the GPU parity tests: fill a cache through the C ABI, run the
oracle on the same seeded inputs, compare (not collected by pytest)."""

from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle as O
import spla_inputs as si
from paper_2601_22379_amd import spla

TIE_REL = 1e-6     # selection ties allowed within this relative distance of the cutoff
TOL = {"bf16": 2e-2, "f32": 1e-4}


def log(msg):
    sys.stderr.write(f"[{time.strftime('%H:%M:%S')}] {msg}\n")
    sys.stderr.flush()


def params_of(w: si.Workload, **kw) -> O.SplaParams:
    return O.SplaParams(block_size=w.block_size, top_k=w.top_k, n_sink=w.n_sink,
                        n_local=w.n_local, **kw)


def config_of(w: si.Workload, flags=0, rms_eps=1e-6, softmax_scale=0.0, sel_window=0,
              sel_stride=0):
    return spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                            w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local,
                            softmax_scale=softmax_scale, rms_eps=rms_eps, flags=flags,
                            sel_window=sel_window, sel_stride=sel_stride)


def to_dev(x: np.ndarray, w: si.Workload, device):
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    return torch.from_numpy(np.ascontiguousarray(x)).to(dt).to(device)


def slab_tokens(w: si.Workload, budget_bytes=1 << 29) -> int:
    per_tok = w.batch * w.n_kv_heads * w.head_dim * 8
    t = max(256, budget_bytes // per_tok)
    return int(min(w.capacity, 1 << int(np.log2(t))))


def fill_cache(w: si.Workload, cache: spla.SplaCache, lengths=None, slab=None, device="cuda"):
    """Append tokens [0, lengths[b]) of every sequence through spla_append."""
    if lengths is None:
        lengths = [w.prefill_length(b) for b in range(w.batch)]
    T = slab or slab_tokens(w)
    top = max(lengths) if len(lengths) else 0
    for t0 in range(0, top, T):
        t1 = min(t0 + T, top)
        K, V, n = si.gen_kv_slab(w, t0, t1, lengths=lengths, threads=16)
        cache.append(to_dev(K, w, device), to_dev(V, w, device),
                     torch.from_numpy(n).to(device))
    torch.cuda.synchronize()


def oracle_kv_head(w: si.Workload, b: int, h: int, gamma: np.ndarray, q: np.ndarray,
                   p: O.SplaParams, L=None, force=None, state=None):
    L = int(w.lengths[b]) if L is None else L
    K, V = si.gen_kv(w, b, h, 0, L, threads=16)
    if state is None:
        state = O.build_state(K, V, L, w.block_size, p.window, p.stride)
    G = w.group
    res = O.decode_kv_head(q[h * G:(h + 1) * G], state, K, V, gamma[h * G:(h + 1) * G], p, force)
    return res, state, K, V


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over rows of max_j |got - ref| / max_j |ref|."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-30)
    return float((np.abs(got - ref).max(axis=-1) / den).max())


def check_kv_head(w, b, h, out_gpu, sel_gpu, q, gamma, p, L=None, state=None, tol=None):
    """Compare one (sequence, KV head) of the GPU result with the oracle.
    Returns a dict of measured errors; raises AssertionError on a mismatch."""
    tol = TOL[w.dtype] if tol is None else tol
    res, state, K, V = oracle_kv_head(w, b, h, gamma, q, p, L=L, state=state)
    G = w.group
    nsel = len(res.sel)
    gsel = [int(x) for x in sel_gpu[:nsel]]
    assert all(x == -1 for x in sel_gpu[nsel:]), (b, h, "padding", sel_gpu)
    info = {"b": b, "h": h, "n_swapped": 0}
    if gsel != [int(x) for x in res.sel]:
        c = O.cutoff_score(res.score, res.sel, p.top_k, p.n_sink, p.n_local)
        assert c is not None, (b, h, gsel, res.sel)
        diff = set(gsel) ^ set(int(x) for x in res.sel)
        for i in diff:
            assert 0 <= i < len(res.score), (b, h, i)
            rel = abs(res.score[i] - c) / c
            assert rel <= TIE_REL, (b, h, "selection differs beyond the tie window", i, rel)
        assert len(set(gsel)) == len(gsel) == nsel and gsel == sorted(gsel)
        info["n_swapped"] = len(diff) // 2
        res = O.decode_kv_head(q[h * G:(h + 1) * G], state, K, V, gamma[h * G:(h + 1) * G], p,
                               gsel)
    err = row_rel_err(out_gpu[h * G:(h + 1) * G], res.out)
    info["rel_err"] = err
    assert err <= tol, (b, h, "output error", err, tol)
    return info
