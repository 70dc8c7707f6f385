"""GPU parity of the causal prefill (spla_prefill) against the oracle.

T tokens per sequence are prefilled; the query at position L_b + t must
match the oracle's decode over the first L_b + t + 1 tokens (the oracle
prefill). bf16 shapes with G <= 8 run the chunked kernels (chunks of up to
32 positions); the fp32 case runs position by position. The cases cross
block and window boundaries, span several chunks, start from an empty
cache, run into the capacity, use a paged pool and every variant flag.
"""

import numpy as np
import pytest
import torch

import gpu_harness as H
import oracle as O
import spla_inputs as si
from paper_2601_22379_amd import spla

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spla.lib()
    return torch.device("cuda:0")


CASES = {
    # one chunk, crossing a block boundary in sequence 1
    "bf16_g4_B64": (dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                         top_k=6, lengths=[1000, 60], capacity=1088, kind="block_offsets"),
                    {}, 9),
    # fp32: position by position (VALU pass)
    "f32_g2_B32": (dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, block_size=32,
                        top_k=5, lengths=[700, 29], capacity=768, dtype="f32", kind="drift"),
                   {}, 6),
    # strided selection windows, one chunk crossing windows and a block
    "bf16_strided": (dict(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                          top_k=8, lengths=[2040], capacity=2112, kind="iid"),
                     dict(sel_window=32, sel_stride=16), 12),
    # three chunks (32 + 32 + 6), G = 8, B = 32: chunks cross several blocks
    "bf16_g8_B32_chunks": (dict(batch=2, n_q_heads=16, n_kv_heads=2, head_dim=128, block_size=32,
                                top_k=10, lengths=[300, 1500], capacity=1600,
                                kind="pareto_planted", n_planted=3), {}, 70),
    # d = 64, B = 128, G = 2, from an empty cache and from 600 tokens
    "bf16_d64_B128_empty": (dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, block_size=128,
                                 top_k=3, lengths=[0, 600], capacity=1024, kind="drift",
                                 n_sink=1, n_local=1), {}, 40),
    # strided windows over two chunks, G = 6
    "bf16_g6_strided_chunks": (dict(batch=2, n_q_heads=12, n_kv_heads=2, head_dim=128,
                                    block_size=64, top_k=8, lengths=[1500, 777], capacity=2048,
                                    kind="block_offsets"),
                               dict(sel_window=32, sel_stride=16), 45),
}


def chunk_inputs(w, T, lengths):
    kn = np.zeros((T, w.batch, w.n_kv_heads, w.head_dim), np.float32)
    vn = np.zeros_like(kn)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            K, V = si.gen_kv(w, b, h, lengths[b], lengths[b] + T)
            kn[:, b, h], vn[:, b, h] = K, V
    q = np.stack([si.gen_q_batch(w, t) for t in range(T)])
    return kn, vn, q


def check_positions(w, out, sel, q, gamma, p, lengths, T, cap=None):
    worst = 0.0
    for t in range(T):
        for b in range(w.batch):
            L = lengths[b] + t + 1
            if cap is not None:
                L = min(L, cap)
            for h in range(w.n_kv_heads):
                info = H.check_kv_head(w, b, h, out[t, b], sel[t, b, h], q[t, b], gamma, p, L=L)
                worst = max(worst, info["rel_err"])
    return worst


def run_prefill(w, cache, T, dev, lengths=None):
    lengths = list(w.lengths) if lengths is None else lengths
    kn, vn, q = chunk_inputs(w, T, lengths)
    gamma = si.gen_gamma(w)
    out, sel = cache.prefill(H.to_dev(kn, w, dev), H.to_dev(vn, w, dev), H.to_dev(q, w, dev),
                             torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), sel.cpu().numpy(), q, gamma


@pytest.mark.parametrize("name", list(CASES))
def test_prefill_matches_oracle_at_every_position(dev, name):
    spec, kw, T = CASES[name]
    w = si.custom(name, code=180 + list(CASES).index(name), **spec)
    H.log(f"case {name} T={T}")
    cache = spla.SplaCache(H.config_of(w, **kw), dev)
    H.fill_cache(w, cache, lengths=list(w.lengths), device=dev)
    out, sel, q, gamma = run_prefill(w, cache, T, dev)
    assert cache.seq_lens.cpu().tolist() == [L + T for L in w.lengths]
    assert cache.device_errors() == 0
    p = H.params_of(w, window=kw.get("sel_window"), stride=kw.get("sel_stride"))
    worst = check_positions(w, out, sel, q, gamma, p, list(w.lengths), T)
    H.log(f"{name}: worst row rel err {worst:.3e}")


@pytest.mark.parametrize("flags,kw", [
    (spla.FLAG_NO_RLA, dict(no_rla=True)),
    (spla.FLAG_FIRST_ORDER, dict(first_order=True)),
    (spla.FLAG_RLA_NORMALIZE, dict(rla_normalize=True)),
])
def test_prefill_variant_flags(dev, flags, kw):
    w = si.custom("pflags", 2, 8, 2, 128, 64, 6, [900, 2000], kind="block_offsets", code=190,
                  capacity=2112)
    cache = spla.SplaCache(H.config_of(w, flags=flags), dev)
    H.fill_cache(w, cache, device=dev)
    out, sel, q, gamma = run_prefill(w, cache, 20, dev)
    check_positions(w, out, sel, q, gamma, H.params_of(w, **kw), list(w.lengths), 20)


def test_prefill_into_the_capacity(dev):
    """Sequence 0 has room for 24 of the 40 positions: the rest are dropped
    (flagged) and their queries decode over the full cache, as spla_step
    does at capacity."""
    w = si.custom("pcap", 2, 8, 2, 128, 64, 6, [1000, 500], kind="iid", code=191, capacity=1024)
    cache = spla.SplaCache(H.config_of(w), dev)
    H.fill_cache(w, cache, device=dev)
    T = 40
    out, sel, q, gamma = run_prefill(w, cache, T, dev)
    assert cache.seq_lens.cpu().tolist() == [1024, 540]
    assert cache.device_errors() & spla.DEVERR_CAPACITY
    check_positions(w, out, sel, q, gamma, H.params_of(w), list(w.lengths), T, cap=1024)


def test_prefill_paged_equals_contiguous(dev):
    """The same prefill into a paged pool behind a shuffled table: identical
    outputs and selections, and the decode after it agrees too."""
    w = si.custom("ppaged", 2, 8, 2, 128, 64, 8, [1200, 300], kind="block_offsets", code=192,
                  capacity=2048)
    nb = w.capacity // w.block_size
    pages = w.batch * nb + 17
    rng = np.random.default_rng(192)
    tab = rng.permutation(pages)[:w.batch * nb].reshape(w.batch, nb).astype(np.int32)
    cfg_p = spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                             w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local,
                             kv_pages=pages)
    paged = spla.SplaCache(cfg_p, dev, block_table=torch.from_numpy(tab).to(dev))
    flat = spla.SplaCache(H.config_of(w), dev)
    for c in (paged, flat):
        H.fill_cache(w, c, device=dev)
    T = 37
    a = run_prefill(w, paged, T, dev)
    b = run_prefill(w, flat, T, dev)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert paged.device_errors() == 0
    check_positions(w, a[0], a[1], a[2], a[3], H.params_of(w), list(w.lengths), T)
    qd = si.gen_q_batch(w, 99)
    g = torch.from_numpy(a[3]).to(dev)
    o1, s1 = paged.decode(H.to_dev(qd, w, dev), g)
    o2, s2 = flat.decode(H.to_dev(qd, w, dev), g)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(s1, s2)


def test_prefill_then_decode_and_state(dev):
    """After a chunked prefill the cache holds what appending the same tokens
    would give: statistics and S_bar agree with the oracle's, and a decode
    step after it matches the oracle."""
    w = si.custom("pstate", 2, 8, 2, 128, 64, 8, [700, 1999], kind="drift", code=193,
                  capacity=2112)
    cache = spla.SplaCache(H.config_of(w), dev)
    H.fill_cache(w, cache, device=dev)
    T = 50
    run_prefill(w, cache, T, dev)
    mean, m2 = (x.cpu().numpy() for x in cache.stats_logical())
    S, z = (x.cpu().numpy() for x in cache.state_logical())
    for b in range(w.batch):
        L = w.lengths[b] + T
        for h in range(w.n_kv_heads):
            K, V = si.gen_kv(w, b, h, 0, L)
            st = O.build_state(K, V, L, w.block_size)
            nb = len(st.counts)
            np.testing.assert_allclose(mean[b, h, :nb], st.mean, rtol=0, atol=2e-6)
            np.testing.assert_allclose(m2[b, h, :nb] / st.counts[:, None], st.var, rtol=2e-5,
                                       atol=1e-6)
            np.testing.assert_allclose(S[b, h], st.s_bar, rtol=2e-4, atol=2e-4)
            np.testing.assert_allclose(z[b, h], st.z_bar, rtol=2e-5, atol=1e-5)
    qd = si.gen_q_batch(w, 77)
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(qd, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    out = out.float().cpu().numpy()
    sel = sel.cpu().numpy()
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], qd[b], gamma, H.params_of(w),
                            L=w.lengths[b] + T)
