"""GPU parity of the causal prefill (spla_prefill) against the oracle.

A chunk of T tokens per sequence is appended position by position and the
queries at each position decoded. The query at position L_b + t must match
the oracle's decode over the first L_b + t + 1 tokens, which is the oracle
prefill. The chunks cross block (and window) boundaries.
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


CASES = {
    # single-launch decode at every position
    "bf16_g4_B64": (dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                         top_k=6, lengths=[1000, 60], capacity=1088, kind="block_offsets"),
                    {}, 9),
    # fp32, VALU pass
    "f32_g2_B32": (dict(batch=2, n_q_heads=4, n_kv_heads=2, head_dim=64, block_size=32,
                        top_k=5, lengths=[700, 29], capacity=768, dtype="f32", kind="drift"),
                   {}, 6),
    # strided selection windows
    "bf16_strided": (dict(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                          top_k=8, lengths=[2040], capacity=2112, kind="iid"),
                     dict(sel_window=32, sel_stride=16), 12),
}


@pytest.mark.parametrize("name", list(CASES))
def test_prefill_matches_oracle_at_every_position(dev, name):
    spec, kw, T = CASES[name]
    w = si.custom(name, code=180 + list(CASES).index(name), **spec)
    H.log(f"case {name} T={T}")
    cache = spla.SplaCache(H.config_of(w, **kw), dev)
    H.fill_cache(w, cache, lengths=list(w.lengths), device=dev)
    kn = np.zeros((T, w.batch, w.n_kv_heads, w.head_dim), np.float32)
    vn = np.zeros_like(kn)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            K, V = si.gen_kv(w, b, h, w.lengths[b], w.lengths[b] + T)
            kn[:, b, h], vn[:, b, h] = K, V
    q = np.stack([si.gen_q_batch(w, t) for t in range(T)])
    gamma = si.gen_gamma(w)
    out, sel = cache.prefill(H.to_dev(kn, w, dev), H.to_dev(vn, w, dev), H.to_dev(q, w, dev),
                             torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    assert cache.seq_lens.cpu().tolist() == [L + T for L in w.lengths]
    assert cache.err.item() == 0
    out = out.float().cpu().numpy()
    sel = sel.cpu().numpy()
    p = H.params_of(w, window=kw.get("sel_window"), stride=kw.get("sel_stride"))
    for t in range(T):
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                H.check_kv_head(w, b, h, out[t, b], sel[t, b, h], q[t, b], gamma, p,
                                L=w.lengths[b] + t + 1)
