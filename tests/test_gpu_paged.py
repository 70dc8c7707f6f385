"""GPU parity of the paged KV cache (block = page, Sec. 2.1): the K/V caches
are pools of pages addressed through a caller-owned block table.

The same appends go into a contiguous cache and into a paged one whose table
is a seeded shuffle of a larger pool. Both decodes must give the same
selection and bit-identical outputs (the arithmetic is the same, only the
addresses differ), and the paged one must match the oracle like every
other case.
"""

import numpy as np
import pytest
import torch

import gpu_harness as H
import spla_inputs as si
from paper_2601_22379_amd import spla

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spla.lib()
    return torch.device("cuda:0")


def shuffled_table(w, extra, seed):
    nb = w.capacity // w.block_size
    pages = w.batch * nb + extra
    rng = np.random.default_rng([seed, w.code])
    tab = rng.permutation(pages)[:w.batch * nb].reshape(w.batch, nb).astype(np.int32)
    return pages, tab


def paged_config(w, pages, **kw):
    return spla.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size,
                            w.top_k, w.capacity, w.dtype, n_sink=w.n_sink, n_local=w.n_local,
                            kv_pages=pages, **kw)


CASES = {
    "bf16_g4_B64_mfma": (dict(batch=3, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                              top_k=8, lengths=[5000, 63, 9001], kind="block_offsets"), {}),
    "f32_g2_B32_valu": (dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, block_size=32,
                             top_k=6, lengths=[3071, 700], dtype="f32", kind="drift"), {}),
    "bf16_g16_valu": (dict(batch=1, n_q_heads=16, n_kv_heads=1, head_dim=64, block_size=32,
                           top_k=10, lengths=[6000], kind="pareto_planted", n_planted=4), {}),
    "bf16_strided_paged": (dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                                top_k=8, lengths=[4097, 2500], kind="iid"),
                           dict(sel_window=32, sel_stride=16)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_paged_equals_contiguous_and_matches_oracle(dev, name):
    spec, kw = CASES[name]
    w = si.custom(name, code=160 + list(CASES).index(name), **spec)
    H.log(f"case {name}")
    pages, tab = shuffled_table(w, extra=7, seed=1)
    flat = spla.SplaCache(H.config_of(w, **kw), dev)
    paged = spla.SplaCache(paged_config(w, pages, **kw), dev,
                           block_table=torch.from_numpy(tab).to(dev))
    for c in (flat, paged):
        H.fill_cache(w, c, lengths=list(w.lengths), slab=1000, device=dev)
    q = si.gen_q_batch(w)
    gamma = si.gen_gamma(w)
    qd, gd = H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev)
    out_f, sel_f = flat.decode(qd, gd)
    out_p, sel_p = paged.decode(qd, gd)
    torch.cuda.synchronize()
    assert paged.err.item() == 0
    assert torch.equal(sel_f, sel_p)
    assert torch.equal(out_f, out_p)
    assert torch.equal(flat.stats, paged.stats)
    for b in range(w.batch):
        L = w.lengths[b]
        for h in range(w.n_kv_heads):
            K, V = si.gen_kv(w, b, h, 0, L)
            assert np.array_equal(paged.k_logical()[b, h, :L].float().cpu().numpy(), K)
            assert np.array_equal(paged.v_logical()[b, h, :L].float().cpu().numpy(), V)
    p = H.params_of(w, window=kw.get("sel_window"), stride=kw.get("sel_stride"))
    out = out_p.float().cpu().numpy()
    sel = sel_p.cpu().numpy()
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p)


def test_paged_step_and_out_of_range_entry(dev):
    """spla_step on a paged pool appends into the table's pages; an append
    into a block whose entry is outside the pool writes nothing there and
    sets SPLA_DEVERR_PAGE."""
    w = si.custom("pagedstep", 1, 4, 1, 128, 64, 6, [1000], kind="iid", code=170, capacity=2048)
    pages, tab = shuffled_table(w, extra=3, seed=2)
    tab[0, 1000 // 64 + 1] = pages + 5  # the block after the one token 1000 lands in
    cache = spla.SplaCache(paged_config(w, pages), dev, block_table=torch.from_numpy(tab).to(dev))
    H.fill_cache(w, cache, lengths=[1000], device=dev)
    p = H.params_of(w)
    gamma = si.gen_gamma(w)
    K, V = si.gen_kv(w, 0, 0, 0, 1001)
    q = si.gen_q_batch(w, 3)
    out, sel = cache.step(H.to_dev(K[1000][None, None], w, dev),
                          H.to_dev(V[1000][None, None], w, dev), H.to_dev(q, w, dev),
                          torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    assert cache.err.item() == 0 and cache.seq_lens.cpu().tolist() == [1001]
    H.check_kv_head(w, 0, 0, out.float().cpu().numpy()[0], sel.cpu().numpy()[0, 0], q[0], gamma,
                    p, L=1001)
    # tokens 1001 .. 1087 reach block 16, whose entry lies outside the pool
    K2, V2 = si.gen_kv(w, 0, 0, 1001, 1088)
    cache.append(H.to_dev(K2[None, None], w, dev), H.to_dev(V2[None, None], w, dev))
    torch.cuda.synchronize()
    assert cache.err.item() & spla.DEVERR_PAGE
    assert cache.seq_lens.cpu().tolist() == [1088]
