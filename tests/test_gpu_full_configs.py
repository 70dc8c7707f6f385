"""GPU parity at the five workloads' full sizes (and the paper's G = 5 shape).

The cache is filled through spla_append and decoded with the same library
call the benchmark times. The oracle recomputes a seeded sample of
(sequence, KV head) units from scratch in fp64; every unit is also checked
for properties that hold at any size (ascending ids, forced blocks present,
finite outputs).
"""

import numpy as np
import pytest
import torch

import gpu_harness as H
import spla_inputs as si
from paper_2601_22379_amd import spla

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

SAMPLES = {"1": 1, "2": 32, "3": 32, "4": 32, "5": 8, "g5": 8}


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spla.lib()
    return torch.device("cuda:0")


def sample_pairs(w, n, seed):
    rng = np.random.default_rng([seed, w.code, 77])
    allp = [(b, h) for b in range(w.batch) for h in range(w.n_kv_heads)]
    idx = rng.choice(len(allp), size=min(n, len(allp)), replace=False)
    return [allp[i] for i in sorted(idx)]


def check_properties(w, sel, out, lengths):
    assert np.all(np.isfinite(out))
    for b in range(w.batch):
        nb = -(-int(lengths[b]) // w.block_size)
        for h in range(w.n_kv_heads):
            s = sel[b, h]
            if nb <= w.top_k:
                assert list(s[:nb]) == list(range(nb)) and np.all(s[nb:] == -1)
                continue
            assert np.all(np.diff(s) > 0) and s[0] >= 0 and s[-1] < nb
            forced = set(range(w.n_sink)) | set(range(nb - w.n_local, nb))
            assert forced <= set(s.tolist())


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cfg_id", ["1", "2", "3", "5", "g5"])
def test_full_size_decode(dev, cfg_id):
    w = si.config(cfg_id)
    H.log(f"full config {cfg_id} ({w.name}): filling cache")
    cache = spla.SplaCache(H.config_of(w), dev)
    H.fill_cache(w, cache, device=dev)
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    out = out.float().cpu().numpy()
    sel = sel.cpu().numpy()
    check_properties(w, sel, out, w.lengths)
    p = H.params_of(w)
    pairs = sample_pairs(w, SAMPLES[cfg_id], 0)
    H.log(f"config {cfg_id}: oracle on {pairs}")
    infos = [H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p) for b, h in pairs]
    H.log(f"config {cfg_id}: worst rel err {max(i['rel_err'] for i in infos):.3e}, "
          f"swaps {sum(i['n_swapped'] for i in infos)}")
    if w.n_planted:
        for b, h in pairs:
            assert set(si.planted_blocks(w, b, h).tolist()) <= set(sel[b, h].tolist())


@pytest.mark.timeout(1200)
def test_full_size_config4_steps(dev):
    """Config 4: 64 sequences of 16K-64K tokens, each decode step appends one
    token per (sequence, KV head) first (spla_step)."""
    w = si.config(4)
    H.log("config 4: filling cache")
    cache = spla.SplaCache(H.config_of(w), dev)
    H.fill_cache(w, cache, device=dev)
    gamma = si.gen_gamma(w)
    p = H.params_of(w)
    pairs = sample_pairs(w, SAMPLES["4"], 0)
    for step in range(2):
        lens = [w.lengths[b] + step for b in range(w.batch)]
        kn = np.zeros((w.batch, w.n_kv_heads, w.head_dim), np.float32)
        vn = np.zeros_like(kn)
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                k1, v1 = si.gen_kv(w, b, h, lens[b] - 1, lens[b])
                kn[b, h], vn[b, h] = k1[0], v1[0]
        q = si.gen_q_batch(w, step)
        out, sel = cache.step(H.to_dev(kn, w, dev), H.to_dev(vn, w, dev), H.to_dev(q, w, dev),
                              torch.from_numpy(gamma).to(dev))
        torch.cuda.synchronize()
        assert cache.seq_lens.cpu().tolist() == lens
        out = out.float().cpu().numpy()
        sel = sel.cpu().numpy()
        check_properties(w, sel, out, lens)
        H.log(f"config 4 step {step}: oracle on {pairs}")
        infos = [H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p, L=lens[b])
                 for b, h in pairs]
        H.log(f"config 4 step {step}: worst rel err {max(i['rel_err'] for i in infos):.3e}, "
              f"swaps {sum(i['n_swapped'] for i in infos)}")


@pytest.mark.timeout(900)
def test_full_size_strided_selection(dev):
    """The 128K workload with the paper's strided selection windows (C = 32,
    s = 16, max-pooled into B = 64 blocks): 8192 windows per sequence."""
    w = si.config("3")
    C, s = 32, 16
    cache = spla.SplaCache(H.config_of(w, sel_window=C, sel_stride=s), dev)
    H.fill_cache(w, cache, device=dev)
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    out = out.float().cpu().numpy()
    sel = sel.cpu().numpy()
    check_properties(w, sel, out, w.lengths)
    p = H.params_of(w, window=C, stride=s)
    pairs = sample_pairs(w, 8, 1)
    H.log(f"strided config 3: oracle on {pairs}")
    infos = [H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p) for b, h in pairs]
    H.log(f"strided config 3: worst rel err {max(i['rel_err'] for i in infos):.3e}, "
          f"swaps {sum(i['n_swapped'] for i in infos)}")


@pytest.mark.timeout(900)
def test_full_size_paged_cache(dev):
    """The 128K workload in a paged pool behind a shuffled block table: the
    same selection and bit-identical outputs as the per-sequence cache, and
    sampled units against the oracle."""
    w = si.config("3")
    nb = w.capacity // w.block_size
    pages = w.batch * nb + 64
    rng = np.random.default_rng([3, w.code])
    tab = rng.permutation(pages)[:w.batch * nb].reshape(w.batch, nb).astype(np.int32)
    cfg = spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                           w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local,
                           kv_pages=pages)
    paged = spla.SplaCache(cfg, dev, block_table=torch.from_numpy(tab).to(dev))
    H.fill_cache(w, paged, device=dev)
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    qd, gd = H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev)
    out_p, sel_p = paged.decode(qd, gd)
    torch.cuda.synchronize()
    del paged
    flat = spla.SplaCache(H.config_of(w, flags=spla.FLAG_SEPARATE_KERNELS), dev)
    H.fill_cache(w, flat, device=dev)
    out_f, sel_f = flat.decode(qd, gd)
    torch.cuda.synchronize()
    assert torch.equal(sel_f, sel_p) and torch.equal(out_f, out_p)
    out = out_p.float().cpu().numpy()
    sel = sel_p.cpu().numpy()
    check_properties(w, sel, out, w.lengths)
    p = H.params_of(w)
    pairs = sample_pairs(w, 8, 2)
    infos = [H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p) for b, h in pairs]
    H.log(f"paged config 3: worst rel err {max(i['rel_err'] for i in infos):.3e}")
