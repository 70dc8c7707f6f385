"""Pins of the oracle's causal prefill (Sec. 2: the decode formulation
applied at every position of a chunk).

With a budget that selects every block, the residual is zero and each
position's output is causal dense attention, checked against torch's
float64 scaled_dot_product_attention with a causal mask. The global linear
branch obeys the chunkwise identity phi(Q) S_bar = the causally masked
product (phi(Q) phi(K)^T . mask) V plus the state before the chunk. Changing
a later token never changes an earlier output.
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O


def _rng(*s):
    return np.random.default_rng(list(s))


@pytest.mark.parametrize("L0,T", [(0, 9), (5, 12), (31, 4)])
def test_p1_all_blocks_selected_is_causal_dense_attention(L0, T):
    r = _rng(1, L0, T)
    G, d, B = 3, 16, 8
    n = L0 + T
    K = r.standard_normal((n, d))
    V = r.standard_normal((n, d))
    Q = r.standard_normal((T, G, d))
    p = O.SplaParams(block_size=B, top_k=-(-n // B), n_sink=1, n_local=1)
    res = O.prefill_kv_head(Q, K, V, L0, np.ones((G, d)), p)
    s = 1 / math.sqrt(d)
    # dense causal attention of the chunk's queries over every earlier token
    qt = torch.tensor(Q.transpose(1, 0, 2))[None]            # [1, G, T, d]
    kt = torch.tensor(K)[None, None].expand(1, G, n, d)
    vt = torch.tensor(V)[None, None].expand(1, G, n, d)
    mask = torch.tensor(np.arange(n)[None, :] <= (L0 + np.arange(T))[:, None])
    ref = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=s)[0].numpy()
    for i in range(T):
        np.testing.assert_allclose(res[i].r, 0.0, atol=0)
        np.testing.assert_allclose(res[i].out, ref[:, i], rtol=1e-12, atol=1e-13)


def test_p2_global_linear_branch_is_the_chunkwise_form():
    """o_bar at every position equals phi(q) (S_before + sum over the chunk's
    earlier-or-equal tokens of phi(k)^T v): the masked quadratic form a
    chunkwise kernel evaluates."""
    r = _rng(2)
    G, d, B, L0, T = 2, 8, 4, 10, 7
    n = L0 + T
    K = r.standard_normal((n, d))
    V = r.standard_normal((n, d))
    Q = r.standard_normal((T, G, d))
    p = O.SplaParams(block_size=B, top_k=2, n_sink=1, n_local=1)
    res = O.prefill_kv_head(Q, K, V, L0, np.ones((G, d)), p)

    def phi(x):
        e = np.exp(x - x.max(-1, keepdims=True))
        return e / e.sum(-1, keepdims=True)
    s_before = phi(K[:L0]).T @ V[:L0]
    pk, pv = phi(K[L0:]), V[L0:]
    mask = np.tril(np.ones((T, T)))
    for g in range(G):
        pq = phi(Q[:, g])
        chunk = ((pq @ pk.T) * mask) @ pv
        ref = pq @ s_before + chunk
        got = np.stack([res[i].o_bar[g] for i in range(T)])
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)


def test_p3_later_tokens_do_not_change_earlier_outputs():
    r = _rng(3)
    G, d, B, L0, T = 2, 8, 4, 6, 10
    n = L0 + T
    K = r.standard_normal((n, d))
    V = r.standard_normal((n, d))
    Q = r.standard_normal((T, G, d))
    p = O.SplaParams(block_size=B, top_k=3, n_sink=1, n_local=1)
    a = O.prefill_kv_head(Q, K, V, L0, np.ones((G, d)), p)
    K2, V2 = K.copy(), V.copy()
    K2[L0 + 5:] += 3.0
    V2[L0 + 5:] -= 2.0
    b = O.prefill_kv_head(Q, K2, V2, L0, np.ones((G, d)), p)
    for i in range(5):
        np.testing.assert_array_equal(a[i].out, b[i].out)
        np.testing.assert_array_equal(a[i].sel, b[i].sel)
    assert not np.allclose(a[5].out, b[5].out)
