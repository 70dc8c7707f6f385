"""GPU parity of strided block selection (Sec. 3.1: Taylor masses on windows
of C tokens every s tokens, max-pooled into blocks) against the oracle.

The caches are filled through spla_append with sel_window / sel_stride set,
so the append keeps one statistics entry per window; the decode then runs
the score, select, sparse and merge launches. Selections must match the
oracle's except for blocks within 1e-6 (relative) of the cutoff; outputs
within 2e-2 (bf16) or 1e-4 (fp32) max row-relative error.
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


def run(w, dev, C, s, slab=None, flags=0):
    cfg = H.config_of(w, flags=flags, sel_window=C, sel_stride=s)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, lengths=list(w.lengths), slab=slab, device=dev)
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    return cache, q, gamma, out.float().cpu().numpy(), sel.cpu().numpy()


CASES = {
    # the paper's windows at B = 64, ragged lengths (partial windows and blocks)
    "bf16_C32_s16_B64": (dict(batch=4, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                              top_k=8, lengths=[1, 40, 5000, 9001], kind="iid"), 32, 16),
    "bf16_C32_s16_B64_planted": (dict(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128,
                                      block_size=64, top_k=12, lengths=[20000],
                                      kind="pareto_planted", n_planted=4), 32, 16),
    "f32_C32_s16_B32": (dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, block_size=32,
                             top_k=6, lengths=[3071, 700], dtype="f32", kind="block_offsets"),
                        32, 16),
    "bf16_C64_s32_B64": (dict(batch=2, n_q_heads=10, n_kv_heads=2, head_dim=128, block_size=64,
                              top_k=8, lengths=[4097, 2500], kind="drift"), 64, 32),
    "bf16_C32_s16_B128": (dict(batch=1, n_q_heads=4, n_kv_heads=1, head_dim=128,
                               block_size=128, top_k=6, lengths=[7000], kind="iid"), 32, 16),
    "bf16_C16_s16_B64": (dict(batch=1, n_q_heads=16, n_kv_heads=2, head_dim=64, block_size=64,
                              top_k=10, lengths=[12345], kind="block_offsets"), 16, 16),
    # G = 16 (the VALU pass; the selection takes its heads four at a time)
    "bf16_C32_s16_g16": (dict(batch=1, n_q_heads=16, n_kv_heads=1, head_dim=64, block_size=32,
                              top_k=10, lengths=[9000], kind="drift"), 32, 16),
    # an odd number of statistics tiles (two tiles per scoring item)
    "bf16_C32_s16_odd_tiles": (dict(batch=2, n_q_heads=4, n_kv_heads=1, head_dim=128,
                                    block_size=64, top_k=8, lengths=[3 * 1024 + 17, 1000],
                                    capacity=3 * 1024 + 64, kind="iid"), 32, 16),
}


@pytest.mark.parametrize("name", list(CASES))
def test_strided_selection_matches_oracle(dev, name):
    spec, C, s = CASES[name]
    w = si.custom(name, code=140 + list(CASES).index(name), **spec)
    H.log(f"case {name} C={C} s={s}")
    cache, q, gamma, out, sel = run(w, dev, C, s)
    p = H.params_of(w, window=C, stride=s)
    infos = [H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p)
             for b in range(w.batch) for h in range(w.n_kv_heads)]
    H.log(f"{name}: worst row rel err {max(i['rel_err'] for i in infos):.3e}, "
          f"tie swaps {sum(i['n_swapped'] for i in infos)}")


def test_window_statistics_after_uneven_appends(dev):
    """Every window's mean and M2 after appends in slabs that cut windows
    equal the oracle's two-pass statistics of exactly its tokens; the K/V
    rows land once each."""
    w = si.custom("winstats", 2, 4, 2, 128, 64, 8, [5000, 2345], kind="drift", code=150)
    C, s = 32, 16
    cache, q, gamma, out, sel = run(w, dev, C, s, slab=777)
    mean, m2 = (x.cpu().numpy() for x in cache.stats_logical())
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            L = w.lengths[b]
            K, V = si.gen_kv(w, b, h, 0, L)
            mu, var, cnt = O.window_stats(K, L, C, s)
            nw = len(cnt)
            assert nw == -(-L // s)
            np.testing.assert_allclose(mean[b, h, :nw], mu, rtol=0, atol=2e-6)
            np.testing.assert_allclose(m2[b, h, :nw] / cnt[:, None], var, rtol=2e-5, atol=1e-6)
            assert np.all(mean[b, h, nw:] == 0) and np.all(m2[b, h, nw:] == 0)
            kl = cache.k_logical()[b, h, :L].float().cpu().numpy()
            vl = cache.v_logical()[b, h, :L].float().cpu().numpy()
            assert np.array_equal(kl, K) and np.array_equal(vl, V)


def test_strided_step_appends_one_token_then_decodes(dev):
    """spla_step (append one token, decode) keeps the window statistics
    current across window and block boundaries."""
    w = si.custom("winstep", 1, 4, 1, 128, 64, 6, [1023], kind="iid", code=151, capacity=2048)
    C, s = 32, 16
    cfg = H.config_of(w, sel_window=C, sel_stride=s)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, lengths=[1023], device=dev)
    p = H.params_of(w, window=C, stride=s)
    gamma = si.gen_gamma(w)
    K, V = si.gen_kv(w, 0, 0, 0, 1030)
    for L in range(1023, 1030):  # crosses the window start at 1024 and the block at 1024
        q = si.gen_q_batch(w, L)
        kn = H.to_dev(K[L][None, None], w, dev)
        vn = H.to_dev(V[L][None, None], w, dev)
        out, sel = cache.step(kn, vn, H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
        torch.cuda.synchronize()
        assert cache.seq_lens.cpu().tolist() == [L + 1]
        st = O.build_state(K, V, L + 1, w.block_size, C, s)
        H.check_kv_head(w, 0, 0, out.float().cpu().numpy()[0], sel.cpu().numpy()[0, 0], q[0],
                        gamma, p, L=L + 1, state=st)


@pytest.mark.parametrize("flags,kw", [
    (spla.FLAG_FIRST_ORDER, dict(first_order=True)),
    (spla.FLAG_NO_RLA | spla.FLAG_FIRST_ORDER, dict(no_rla=True, first_order=True)),
    (spla.FLAG_RLA_NORMALIZE, dict(rla_normalize=True)),
])
def test_strided_selection_with_variant_flags(dev, flags, kw):
    """The ablation switches of Sec. 4 combined with strided windows."""
    w = si.custom("winflags", 2, 8, 2, 128, 64, 8, [3000, 4100], kind="block_offsets", code=152)
    H.log(f"strided flags {flags}")
    cache, q, gamma, out, sel = run(w, dev, 32, 16, flags=flags)
    p = H.params_of(w, window=32, stride=16, **kw)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p)
