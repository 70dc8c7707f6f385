"""Pins of the oracle's strided block selection (Sec. 3.1, "Strided Block
Selection": Taylor masses on windows of C tokens every s tokens, max-pooled
into blocks).

The paper gives no numbers for this step, so the pins are a hand-worked
closed form, brute-force token sums, brute-force pooling over token sets, a
planted-token case whose outcome the reading fixes, and the streaming
statistics against two-pass ones computed here.
"""

import math

import numpy as np
import pytest

import oracle as O


def _rng(*s):
    return np.random.default_rng(list(s))


def _decode(q, K, V, L, B, k, C, s, n_sink=1, n_local=1):
    p = O.SplaParams(block_size=B, top_k=k, n_sink=n_sink, n_local=n_local, window=C, stride=s)
    st = O.build_state(K, V, L, B, C, s)
    return O.decode_kv_head(q, st, K, V, np.ones(q.shape), p)


# -------------------------------------------------------------------- X15
def test_x15_constant_keys_window_and_block_scores_closed_form():
    """Equal keys everywhere: every token has the same mass, so a window's
    share of a head's total is n_w / sum n, the group score is G times that,
    and a block takes the largest share among the windows touching it.
    L = 40, C = 32, s = 16, B = 32: windows [0,32), [16,40), [32,40) hold
    32, 24, 8 tokens (total 64); block 0 = tokens 0..31 touches windows 0
    and 1, block 1 = tokens 32..39 touches windows 1 and 2."""
    G, d, L = 3, 8, 40
    r = _rng(15)
    K = np.repeat(r.standard_normal((1, d)), L, 0)
    V = r.standard_normal((L, d))
    q = r.standard_normal((G, d))
    res = _decode(q, K, V, L, B=32, k=4, C=32, s=16)
    np.testing.assert_allclose(res.extras["window_score"], G * np.array([32, 24, 8]) / 64,
                               rtol=1e-13)
    np.testing.assert_allclose(res.score, [G / 2, 3 * G / 8], rtol=1e-13)
    assert list(res.sel) == [0, 1]


# -------------------------------------------------------------------- X16
@pytest.mark.parametrize("C,s", [(32, 16), (24, 8), (20, 8), (16, 16)])
def test_x16_window_mass_matches_token_sum(C, s):
    """For keys close to their window mean the second-order estimate (Eq. 10)
    of a window's mass equals the brute-force sum of exp(s q.k) over exactly
    the window's tokens, partial windows at the end included. What is left is
    the dropped off-diagonal covariance, of the order of the squared spread
    of s q.k (about 1e-6 here); a token too many or too few is a 1/n change."""
    r = _rng(16, C, s)
    G, d = 2, 8
    L = 16 * 7 + 5
    mu = r.standard_normal(d)
    K = mu + 1e-3 * r.standard_normal((L, d))
    q = r.standard_normal((G, d))
    sc = 0.35
    mean, var, counts = O.window_stats(K, L, C, s)
    ell = O.log_block_mass(q, mean, var, counts, sc)
    nw = -(-L // s)
    assert ell.shape == (G, nw)
    for w in range(nw):
        toks = [t for t in range(L) if w * s <= t < w * s + C]
        brute = np.exp(sc * q @ K[toks].T).sum(axis=1)
        np.testing.assert_allclose(np.exp(ell[:, w]), brute, rtol=2e-6)
        assert counts[w] == len(toks)


# -------------------------------------------------------------------- X17
@pytest.mark.parametrize("L,B,C,s", [(40, 32, 32, 16), (117, 32, 32, 16), (200, 64, 32, 16),
                                     (77, 16, 24, 8), (99, 16, 16, 16), (64, 64, 32, 16),
                                     (1, 64, 32, 16)])
def test_x17_pooling_matches_token_set_overlap(L, B, C, s):
    """Max-pooling by brute force over token sets: block i takes the maximum
    over the windows whose token set meets block i's token set. With
    C = s = B that is the window of the block itself."""
    r = _rng(17, L, B)
    nw = -(-L // s)
    wscore = r.random(nw)
    nb = -(-L // B)
    got = O.pool_windows_to_blocks(wscore, L, B, C, s)
    assert got.shape == (nb,)
    for i in range(nb):
        blk = set(range(i * B, min(i * B + B, L)))
        cands = [wscore[w] for w in range(nw) if blk & set(range(w * s, min(w * s + C, L)))]
        assert got[i] == max(cands)
    if C == s == B:
        np.testing.assert_array_equal(got, wscore)


# -------------------------------------------------------------------- X18
def test_x18_planted_tokens_at_a_block_end_select_both_blocks():
    """Eight keys aligned with the query at the end of block j lie in the
    windows starting at jB + 32 and jB + 48; the second reaches into block
    j + 1, so under max-pooling both blocks outscore all others and, with
    one sink and one local block forced, the budget k = 4 takes exactly
    {0, j, j + 1, nb - 1}. With one window per block (C = s = B) block j + 1
    has nothing special and is not taken."""
    r = _rng(18)
    d, B, nb, j = 16, 64, 12, 5
    L = nb * B
    q = r.standard_normal((1, d))
    K = r.standard_normal((L, d))
    V = r.standard_normal((L, d))
    s_att = 1 / math.sqrt(d)
    K[j * B + 56:j * B + 64] = 8.0 / (s_att * np.linalg.norm(q)) * q / np.linalg.norm(q)
    res = _decode(q, K, V, L, B, k=4, C=32, s=16)
    assert list(res.sel) == [0, j, j + 1, nb - 1]
    top2 = set(int(i) for i in np.argsort(-res.score)[:2])
    assert top2 == {j, j + 1}
    blocks = _decode(q, K, V, L, B, k=4, C=B, s=B)
    assert j in set(int(i) for i in blocks.sel) and j + 1 not in set(int(i) for i in blocks.sel)


# -------------------------------------------------------------------- X19
@pytest.mark.parametrize("C,s", [(32, 16), (24, 8), (16, 16)])
def test_x19_streaming_window_stats_match_two_pass(C, s):
    """Appending token by token, or in uneven chunks, gives every window the
    two-pass mean and population variance of exactly its tokens."""
    r = _rng(19, C, s)
    d, B, L = 6, 32, 32 * 4 + 11
    K = r.standard_normal((L, d)) * 2 + 3
    V = r.standard_normal((L, d))
    whole = O.append_state(None, K, V, B, window=C, stride=s)
    st = None
    for a, b in zip([0, 1, 5, 16, 17, 50, 100], [1, 5, 16, 17, 50, 100, L]):
        st = O.append_state(st, K[a:b], V[a:b], B, window=C, stride=s)
    nw = -(-L // s)
    for x in (whole, st):
        assert x.mean.shape == (nw, d) and x.length == L
        for w in range(nw):
            win = K[w * s:min(w * s + C, L)]
            np.testing.assert_allclose(x.mean[w], win.mean(0), rtol=1e-12)
            np.testing.assert_allclose(x.var[w], ((win - win.mean(0)) ** 2).mean(0),
                                       rtol=1e-10, atol=1e-13)
            assert x.counts[w] == len(win)
    with pytest.raises(ValueError):
        O.append_state(whole, K[:1], V[:1], B)


def test_x20_one_window_per_block_is_the_block_path():
    """C = s = B is the block path: same statistics, selection and output."""
    r = _rng(20)
    G, d, B, L = 2, 16, 16, 16 * 13 + 3
    q = r.standard_normal((G, d))
    K = r.standard_normal((L, d))
    V = r.standard_normal((L, d))
    gamma = np.ones((G, d))
    a = O.decode_kv_head(q, O.build_state(K, V, L, B), K, V, gamma,
                         O.SplaParams(block_size=B, top_k=5, n_local=2))
    b = O.decode_kv_head(q, O.build_state(K, V, L, B), K, V, gamma,
                         O.SplaParams(block_size=B, top_k=5, n_local=2, window=B, stride=B))
    np.testing.assert_array_equal(a.sel, b.sel)
    np.testing.assert_array_equal(a.out, b.out)
    with pytest.raises(ValueError):
        O.decode_kv_head(q, O.build_state(K, V, L, B), K, V, gamma,
                         O.SplaParams(block_size=B, top_k=5, window=32, stride=16))
