"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Every case fills a cache with spla_append from the seeded generators, runs
spla_decode / spla_step, and compares with the oracle on the same inputs:
selected block ids must match exactly except for blocks whose oracle score
lies within 1e-6 (relative) of the top-k cutoff, and outputs must match to
a max row-relative error of 2e-2 (bf16) or 1e-4 (fp32).
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


def run_decode(w, dev, flags=0, rms_eps=1e-6, lengths=None, slab=None):
    cfg = H.config_of(w, flags=flags, rms_eps=rms_eps)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, lengths=lengths if lengths is not None else list(w.lengths),
                 slab=slab, device=dev)
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    return cache, q, gamma, out.float().cpu().numpy(), sel.cpu().numpy()


def check_all(w, q, gamma, out, sel, p, pairs=None):
    infos = []
    if pairs is None:
        pairs = [(b, h) for b in range(w.batch) for h in range(w.n_kv_heads)]
    for b, h in pairs:
        infos.append(H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p))
    worst = max(i["rel_err"] for i in infos)
    swaps = sum(i["n_swapped"] for i in infos)
    H.log(f"{w.name}: {len(infos)} kv heads, worst row rel err {worst:.3e}, tie swaps {swaps}")
    return infos


SMALL = {
    "f32_g2_d64_B32": dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, block_size=32,
                           top_k=6, lengths=[1000, 3071], dtype="f32", kind="block_offsets"),
    "bf16_g5_d128_B64": dict(batch=2, n_q_heads=10, n_kv_heads=2, head_dim=128, block_size=64,
                             top_k=8, lengths=[4097, 2500], kind="block_offsets"),
    "bf16_ragged_edges": dict(batch=7, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                              top_k=8, lengths=[1, 63, 64, 65, 512, 513, 9000], kind="iid"),
    "f32_g1_B128": dict(batch=1, n_q_heads=3, n_kv_heads=3, head_dim=128, block_size=128,
                        top_k=5, lengths=[5000], dtype="f32", kind="drift"),
    "bf16_g16_d64_k40": dict(batch=1, n_q_heads=16, n_kv_heads=1, head_dim=64, block_size=32,
                             top_k=40, lengths=[20000], kind="pareto_planted", n_planted=8),
    "bf16_empty_and_short": dict(batch=3, n_q_heads=4, n_kv_heads=1, head_dim=128,
                                 block_size=32, top_k=6, lengths=[0, 300, 31], kind="iid"),
    # library limits: k = SPLA_MAX_TOP_K with G = SPLA_MAX_GROUP (VALU pass) and on
    # the single-launch kernel; SPLA_MAX_BLOCKS blocks per sequence
    "bf16_k256_g16": dict(batch=1, n_q_heads=16, n_kv_heads=1, head_dim=64, block_size=32,
                          top_k=256, lengths=[20000], kind="iid"),
    "bf16_k256_single_launch": dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128,
                                    block_size=64, top_k=256, lengths=[40000, 17000],
                                    kind="block_offsets"),
    "bf16_32768_blocks": dict(batch=1, n_q_heads=4, n_kv_heads=1, head_dim=64, block_size=32,
                              top_k=32, lengths=[32768 * 32 - 7], capacity=32768 * 32,
                              kind="iid"),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_shapes_match_oracle(dev, name):
    spec = dict(SMALL[name])
    w = si.custom(name, code=100 + list(SMALL).index(name), **spec)
    H.log(f"case {name}")
    cache, q, gamma, out, sel = run_decode(w, dev)
    check_all(w, q, gamma, out, sel, H.params_of(w))


@pytest.mark.parametrize("flags,kw", [
    (spla.FLAG_NO_RLA, dict(no_rla=True)),
    (spla.FLAG_FIRST_ORDER, dict(first_order=True)),
    (spla.FLAG_RLA_NORMALIZE, dict(rla_normalize=True)),
    (spla.FLAG_NO_RLA | spla.FLAG_FIRST_ORDER, dict(no_rla=True, first_order=True)),
])
def test_variant_flags_match_oracle(dev, flags, kw):
    w = si.custom("flags", 2, 8, 2, 128, 64, 8, [3000, 4100], kind="block_offsets", code=120)
    H.log(f"flags {flags}")
    cache, q, gamma, out, sel = run_decode(w, dev, flags=flags)
    check_all(w, q, gamma, out, sel, H.params_of(w, **kw))


def test_no_forced_blocks(dev):
    w = si.custom("noforce", 2, 4, 1, 128, 64, 5, [3000, 700], kind="iid", code=121, n_sink=0,
                  n_local=0)
    cache, q, gamma, out, sel = run_decode(w, dev)
    check_all(w, q, gamma, out, sel, H.params_of(w))


def test_config1_full(dev):
    w = si.config(1)
    cache, q, gamma, out, sel = run_decode(w, dev)
    infos = check_all(w, q, gamma, out, sel, H.params_of(w))
    planted = set(si.planted_blocks(w, 0, 0).tolist())
    assert planted <= set(sel[0, 0].tolist())
    assert infos[0]["rel_err"] < 1e-4


def test_append_statistics_and_state(dev):
    """Block mean / M2 and S_bar, z_bar after appends in uneven slabs equal
    the oracle's (fp64 definitions) to fp32 accuracy."""
    w = si.custom("stats", 2, 4, 2, 128, 64, 8, [5000, 2345], kind="drift", code=122)
    cache, q, gamma, out, sel = run_decode(w, dev, slab=777)
    mean, m2 = (x.cpu().numpy() for x in cache.stats_logical())
    S, z = (x.cpu().numpy() for x in cache.state_logical())
    lens = cache.seq_lens.cpu().numpy()
    assert list(lens) == list(w.lengths)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            L = w.lengths[b]
            K, V = si.gen_kv(w, b, h, 0, L)
            st = O.build_state(K, V, L, w.block_size)
            nb = len(st.counts)
            np.testing.assert_allclose(mean[b, h, :nb], st.mean, rtol=0, atol=2e-6)
            np.testing.assert_allclose(m2[b, h, :nb] / st.counts[:, None], st.var, rtol=2e-5,
                                       atol=1e-6)
            np.testing.assert_allclose(S[b, h], st.s_bar, rtol=2e-5, atol=2e-5)
            np.testing.assert_allclose(z[b, h], st.z_bar, rtol=2e-5, atol=1e-5)
            kl = cache.k_logical()[b, h, :L].float().cpu().numpy()
            vl = cache.v_logical()[b, h, :L].float().cpu().numpy()
            assert np.array_equal(kl, K) and np.array_equal(vl, V)


@pytest.mark.parametrize("B,slab", [(32, 1000), (128, 1500)])
def test_one_pass_append_block_sizes(dev, B, slab):
    """The bulk append's one pass (bf16, d = 128) at one and four 32-token
    steps per block: uneven slabs start mid-block, and the shorter sequence
    receives nothing in the last calls; block mean / M2, S_bar, z_bar and the
    K/V rows equal the oracle's."""
    w = si.custom(f"onepass_B{B}", 2, 4, 2, 128, B, 8, [4321, 1234], kind="drift",
                  code=180 + B // 32)
    cache, q, gamma, out, sel = run_decode(w, dev, slab=slab)
    mean, m2 = (x.cpu().numpy() for x in cache.stats_logical())
    S, z = (x.cpu().numpy() for x in cache.state_logical())
    assert list(cache.seq_lens.cpu().numpy()) == list(w.lengths)
    assert cache.err.item() == 0
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            L = w.lengths[b]
            K, V = si.gen_kv(w, b, h, 0, L)
            st = O.build_state(K, V, L, w.block_size)
            nb = len(st.counts)
            np.testing.assert_allclose(mean[b, h, :nb], st.mean, rtol=0, atol=2e-6)
            np.testing.assert_allclose(m2[b, h, :nb] / st.counts[:, None], st.var, rtol=2e-5,
                                       atol=1e-6)
            np.testing.assert_allclose(S[b, h], st.s_bar, rtol=2e-5, atol=2e-5)
            np.testing.assert_allclose(z[b, h], st.z_bar, rtol=2e-5, atol=1e-5)
            kl = cache.k_logical()[b, h, :L].float().cpu().numpy()
            vl = cache.v_logical()[b, h, :L].float().cpu().numpy()
            assert np.array_equal(kl, K) and np.array_equal(vl, V)
    check_all(w, q, gamma, out, sel, H.params_of(w))


def test_append_chunking_invariance(dev):
    w = si.custom("chunks", 2, 8, 2, 128, 64, 8, [3333, 2049], kind="block_offsets", code=123)
    a = run_decode(w, dev, slab=4096)
    b = run_decode(w, dev, slab=100)
    assert np.array_equal(a[4], b[4])
    assert H.row_rel_err(b[3], a[3]) < 1e-3
    sa = a[0].stats_logical()[0].cpu().numpy()
    sb = b[0].stats_logical()[0].cpu().numpy()
    np.testing.assert_allclose(sa, sb, rtol=0, atol=2e-6)


def test_decode_is_deterministic_and_leaves_cache_unchanged(dev):
    w = si.custom("det", 2, 8, 2, 128, 64, 8, [3000, 4000], kind="iid", code=124)
    cache, q, gamma, out, sel = run_decode(w, dev)
    before = [t.clone() for t in (cache.stats, cache.state, cache.norm, cache.seq_lens)]
    out2, sel2 = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    assert np.array_equal(out2.float().cpu().numpy(), out)
    assert np.array_equal(sel2.cpu().numpy(), sel)
    for t0, t1 in zip(before, (cache.stats, cache.state, cache.norm, cache.seq_lens)):
        assert torch.equal(t0, t1)


def test_capacity_overflow_is_clamped_and_flagged(dev):
    w = si.custom("cap", 2, 4, 1, 64, 32, 6, [300, 100], kind="iid", capacity=256, code=125)
    cfg = H.config_of(w)
    cache = spla.SplaCache(cfg, dev)
    for t0, t1 in [(0, 200), (200, 300)]:
        K, V, n = si.gen_kv_slab(w, t0, t1, lengths=[300, 100])
        cache.append(H.to_dev(K, w, dev), H.to_dev(V, w, dev), torch.from_numpy(n).to(dev))
    torch.cuda.synchronize()
    with pytest.raises(spla.SplaError):   # more rows than the capacity: rejected on the host
        cache.append(*(H.to_dev(np.zeros((2, 1, 257, 64), np.float32), w, dev),) * 2)
    assert cache.seq_lens.cpu().tolist() == [256, 100]
    assert int(cache.err.item()) & spla.DEVERR_CAPACITY
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    p = H.params_of(w)
    H.check_kv_head(w, 0, 0, out.float().cpu().numpy()[0], sel.cpu().numpy()[0, 0], q[0], gamma,
                    p, L=256)


def test_step_appends_then_decodes(dev):
    """spla_step: one token appended per (sequence, KV head), then the decode
    sees it; two consecutive steps."""
    w = si.custom("step", 3, 8, 2, 128, 128, 6, [300, 1000, 129], kind="iid", code=126,
                  capacity=1152, appends_per_step=1)
    cfg = H.config_of(w)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, device=dev)
    gamma = si.gen_gamma(w)
    p = H.params_of(w)
    for step in range(2):
        lens = [w.lengths[b] + step for b in range(w.batch)]
        kn = np.stack([np.stack([si.gen_kv(w, b, h, lens[b] - 1, lens[b])[0][0]
                                 for h in range(w.n_kv_heads)]) for b in range(w.batch)])
        vn = np.stack([np.stack([si.gen_kv(w, b, h, lens[b] - 1, lens[b])[1][0]
                                 for h in range(w.n_kv_heads)]) for b in range(w.batch)])
        q = si.gen_q_batch(w, step)
        out, sel = cache.step(H.to_dev(kn, w, dev), H.to_dev(vn, w, dev), H.to_dev(q, w, dev),
                              torch.from_numpy(gamma).to(dev))
        torch.cuda.synchronize()
        assert cache.seq_lens.cpu().tolist() == lens
        out = out.float().cpu().numpy()
        sel = sel.cpu().numpy()
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p, L=lens[b])
