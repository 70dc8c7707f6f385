"""Pins of the fp64 oracle to what the paper and the mathematics fix.

The paper prints no worked numeric example, so every pin here is a closed
form, a textbook routine (torch's float64 CPU softmax and
scaled_dot_product_attention), brute force over tokens, or an invariant the
paper's definitions imply. Reference values are computed in the tests with
code of their own, never with the oracle's helpers.
"""

import math

import numpy as np
import pytest
import scipy.linalg
import torch
import torch.nn.functional as F

import oracle as O
import spla_inputs as si


def _rng(*s):
    return np.random.default_rng(list(s))


def t_softmax(x):
    return torch.softmax(torch.as_tensor(np.asarray(x), dtype=torch.float64), dim=-1).numpy()


def sdpa(q, K, V, s, mask=None):
    """Dense attention (Eq. 1) via torch: q [Hq, d], K/V [Hkv, L, d]."""
    qt = torch.as_tensor(q, dtype=torch.float64)[None, :, None, :]
    kt = torch.as_tensor(K, dtype=torch.float64)[None]
    vt = torch.as_tensor(V, dtype=torch.float64)[None]
    m = None if mask is None else torch.as_tensor(mask)[None, :, None, :]
    o = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, scale=s,
                                       enable_gqa=q.shape[0] != K.shape[0])
    return o[0, :, 0, :].numpy()


# --------------------------------------------------------------------- X1
@pytest.mark.parametrize("seed", range(4))
def test_x1_subtraction_residual_equals_bruteforce_recurrence(seed):
    """Eqs. (12)-(16): phi(q)(S_bar - S_tilde) equals the naive recurrence
    summed over the unselected tokens only."""
    r = _rng(1, seed)
    d, L, B, G = 16, 203, 16, 3
    q = r.standard_normal((G, d))
    K = r.standard_normal((L, d)) + 0.3 * r.standard_normal((1, d))
    V = r.standard_normal((L, d))
    p = O.SplaParams(block_size=B, top_k=5, n_sink=1, n_local=1)
    st = O.build_state(K, V, L, B)
    res = O.decode_kv_head(q, st, K, V, np.ones((G, d)), p)
    sel = set(int(i) for i in res.sel)
    phq, phk = t_softmax(q), t_softmax(K)
    S = np.zeros((d, d))
    for t in range(L):                       # Eq. (12): I_t on unselected tokens
        if t // B not in sel:
            S += np.outer(phk[t], V[t])
    brute = phq @ S                          # Eq. (13)
    scale = np.abs(res.o_bar).max()
    np.testing.assert_allclose(res.r, brute, rtol=0, atol=1e-12 * scale)
    assert np.abs(brute).max() > 1e-3 * scale


# --------------------------------------------------------------------- X2
@pytest.mark.parametrize("L", [100, 128, 1])
def test_x2_selecting_every_block_is_dense_attention(L):
    """k >= nb: the residual is exactly zero and the output is Eq. (1), with
    GQA head m reading KV head m // G."""
    r = _rng(2, L)
    Hq, Hkv, d, B = 6, 2, 32, 16
    q = r.standard_normal((Hq, d))
    K = r.standard_normal((Hkv, L, d))
    V = r.standard_normal((Hkv, L, d))
    gamma = 1 + 0.1 * r.standard_normal((Hq, d))
    p = O.SplaParams(block_size=B, top_k=8)
    res = O.decode_sequence(q, K, V, L, gamma, p)
    out = np.concatenate([x.out for x in res])
    assert all(np.all(x.r == 0) for x in res)
    ref = sdpa(q, K, V, 1 / math.sqrt(d))
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


# --------------------------------------------------------------------- X3
@pytest.mark.parametrize("seed", range(3))
def test_x3_exact_branch_is_masked_dense_attention(seed):
    """Eq. (5): the exact branch is softmax attention with every unselected
    token masked out (Z over the selected tokens only)."""
    r = _rng(3, seed)
    Hq, Hkv, d, B, L = 4, 2, 16, 8, 77
    q = r.standard_normal((Hq, d))
    K = r.standard_normal((Hkv, L, d))
    V = r.standard_normal((Hkv, L, d))
    p = O.SplaParams(block_size=B, top_k=4, n_sink=1, n_local=1)
    res = O.decode_sequence(q, K, V, L, np.ones((Hq, d)), p)
    mask = np.zeros((Hkv, L), dtype=bool)
    for h, x in enumerate(res):
        for i in x.sel:
            mask[h, i * B:min((i + 1) * B, L)] = True
    assert not mask.all()
    mask_q = np.repeat(mask, Hq // Hkv, axis=0)
    ref = sdpa(q, np.repeat(K, Hq // Hkv, 0), np.repeat(V, Hq // Hkv, 0), 1 / math.sqrt(d),
               mask=mask_q)
    got = np.concatenate([x.o_sparse for x in res])
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


# --------------------------------------------------------------------- X4
def test_x4_identical_keys_taylor_mass_is_exact():
    """Eq. (8) with Eq. (10): when all keys of a block are equal the
    covariance vanishes and n * exp(s q.mu) is the exact block mass, also for
    a partial last block (real count n_i)."""
    r = _rng(4)
    d, B, G = 8, 16, 2
    mus = r.standard_normal((5, d))
    L = 4 * B + 7
    K = np.concatenate([np.repeat(mus[i][None], min(B, L - i * B), 0) for i in range(5)])
    q = r.standard_normal((G, d))
    s = 0.7
    mean, var, counts = O.block_stats(K, L, B)
    ell = O.log_block_mass(q, mean, var, counts, s)
    for i in range(5):
        blk = K[i * B:min((i + 1) * B, L)]
        brute = np.exp(s * q @ blk.T).sum(axis=1)
        np.testing.assert_allclose(np.exp(ell[:, i]), brute, rtol=1e-13)
    assert counts[-1] == 7


# --------------------------------------------------------------------- X5
@pytest.mark.parametrize("eps", [0.05, 0.3, 1.0])
def test_x5_pm_eps_blocks_closed_form(eps):
    """Blocks {mu +- eps e_j} (2d keys): Cov = (eps^2/d) I is exactly
    diagonal, Eq. (10) gives exp(s q.mu)(1 + eps^2 s^2 |q|^2 / (2d)) per key,
    the brute-force mean is exp(s q.mu) (1/d) sum_j cosh(eps s q_j), and their
    gap is the quartic-and-higher tail of cosh."""
    r = _rng(5, int(eps * 100))
    d, G, s = 6, 3, 0.8
    B = 2 * d
    nb = 4
    mus = r.standard_normal((nb, d))
    E = np.eye(d)
    K = np.concatenate([np.concatenate([mus[i] + eps * E, mus[i] - eps * E]) for i in range(nb)])
    q = r.standard_normal((G, d))
    mean, var, counts = O.block_stats(K, nb * B, B)
    ell = O.log_block_mass(q, mean, var, counts, s)
    ell1 = O.log_block_mass(q, mean, var, counts, s, first_order=True)
    for i in range(nb):
        base = np.exp(s * q @ mus[i])
        taylor = B * base * (1 + eps ** 2 * s ** 2 * (q * q).sum(axis=1) / (2 * d))
        np.testing.assert_allclose(np.exp(ell[:, i]), taylor, rtol=1e-13)
        np.testing.assert_allclose(np.exp(ell1[:, i]), B * base, rtol=1e-13)
        x = eps * s * q
        brute = 2 * base * np.cosh(x).sum(axis=1)
        tail = 2 * base * (np.cosh(x) - 1 - x * x / 2).sum(axis=1)
        np.testing.assert_allclose(brute - np.exp(ell[:, i]), tail, rtol=1e-6,
                                   atol=1e-14 * brute.max())


# --------------------------------------------------------------------- X6
def test_x6_taylor_error_is_third_order_with_known_coefficient():
    """Keys mu + eps delta_t with delta from a Sylvester-Hadamard design
    (zero mean, orthogonal columns, so the population covariance is exactly
    diagonal). The second-order polynomial's mean is exactly
    1 + s^2/2 sum_j q_j^2 var_j (population variance, 1/n), and the estimate's
    error divided by eps^3 tends to exp(s q.mu) s^3/6 E[(q.delta)^3]."""
    H = scipy.linalg.hadamard(8).astype(float)
    scales = np.array([1.0, 0.7, 1.3])
    delta = H[:, [1, 2, 3]] * scales            # col1*col2 = col3: non-zero 3rd moment
    n, d = delta.shape
    r = _rng(6)
    mu = r.standard_normal(d)
    q = r.standard_normal((2, d))
    s = 0.9
    third = ((q @ delta.T) ** 3).mean(axis=1)
    assert np.all(np.abs(third) > 1e-3)
    coef = np.exp(s * q @ mu) * s ** 3 / 6 * third
    prev = None
    for eps in [1e-2, 5e-3, 2.5e-3]:
        K = mu + eps * delta
        mean, var, counts = O.block_stats(K, n, n)
        ell = O.log_block_mass(q, mean, var, counts, s)[:, 0]
        taylor_mean = np.exp(ell) / n
        x = s * (q @ (eps * delta).T)            # [G, n]
        poly = (1 + x + x * x / 2).mean(axis=1)  # exact mean of the 2nd-order polynomial
        np.testing.assert_allclose(taylor_mean, np.exp(s * q @ mu) * poly, rtol=1e-13)
        brute = np.exp(s * q @ K.T).mean(axis=1)
        ratio = (brute - taylor_mean) / eps ** 3
        np.testing.assert_allclose(ratio, coef, rtol=5 * eps)
        err = np.abs(brute - taylor_mean)
        if prev is not None:
            np.testing.assert_allclose(prev / err, 8.0, rtol=0.05)
        prev = err


# --------------------------------------------------------------------- X7
@pytest.mark.parametrize("G,nb", [(1, 5), (4, 37), (5, 200), (8, 3)])
def test_x7_group_scores_sum_to_G(G, nb):
    """Eq. (6) with Eq. (9): every head contributes a distribution over the
    blocks, so the group scores sum to G."""
    ell = _rng(7, G, nb).standard_normal((G, nb)) * 5
    sc = O.group_block_scores(ell)
    assert sc.shape == (nb,)
    np.testing.assert_allclose(sc.sum(), G, rtol=1e-13)
    for m in range(G):  # each head separately normalised: a softmax over blocks
        single = O.group_block_scores(ell[m:m + 1])
        np.testing.assert_allclose(single, t_softmax(ell[m]), rtol=1e-13)


# --------------------------------------------------------------------- X8
def test_x8_identical_heads_in_a_group():
    """G identical query heads: the group score is G times the single-head
    score, the selection is the same, and every head's output is equal."""
    r = _rng(8)
    d, B, L, G = 16, 8, 150, 4
    q1 = r.standard_normal((1, d))
    K = r.standard_normal((L, d)) + r.standard_normal((1, d))
    V = r.standard_normal((L, d))
    p = O.SplaParams(block_size=B, top_k=6, n_sink=1, n_local=2)
    st = O.build_state(K, V, L, B)
    one = O.decode_kv_head(q1, st, K, V, np.ones((1, d)), p)
    grp = O.decode_kv_head(np.repeat(q1, G, 0), st, K, V, np.ones((G, d)), p)
    np.testing.assert_allclose(grp.score, G * one.score, rtol=1e-13)
    assert np.array_equal(grp.sel, one.sel)
    for m in range(G):
        np.testing.assert_allclose(grp.out[m], one.out[0], rtol=0, atol=1e-13)


# --------------------------------------------------------------------- X9
@pytest.mark.parametrize("seed", range(12))
def test_x9_selection_brute_force_with_ties(seed):
    """Top-k with forced blocks (Sec. 4): the forced blocks are in, the
    budget is exactly k, and every admitted non-forced block beats every
    rejected one in (score, lower index) order; ties come from duplicated
    scores."""
    r = _rng(9, seed)
    nb = int(r.integers(1, 17))
    k = int(r.integers(1, 10))
    n_sink, n_local = int(r.integers(0, 2)), int(r.integers(0, 3))
    k = max(k, n_sink + n_local)
    score = r.integers(0, 4, size=nb).astype(float) / 7.0   # many exact ties
    sel = O.select_blocks(score, k, n_sink, n_local)
    assert list(sel) == sorted(set(int(i) for i in sel))
    if nb <= k:
        assert list(sel) == list(range(nb))
        return
    forced = set(range(n_sink)) | set(range(nb - n_local, nb))
    assert len(sel) == k and forced <= set(int(i) for i in sel)
    admitted = [int(i) for i in sel if int(i) not in forced]
    rejected = [i for i in range(nb) if i not in forced and i not in set(admitted)]
    for i in admitted:
        for j in rejected:
            assert (score[i], -i) > (score[j], -j)


# -------------------------------------------------------------------- X10
def test_x10_config1_planted_blocks_are_selected():
    """Config 1: the two blocks whose keys were shifted by 2 q/|q| carry the
    largest mass and are selected."""
    w = si.config(1)
    q = si.gen_q(w, 0)
    K, V = si.gen_kv(w, 0, 0, 0, w.lengths[0])
    p = O.SplaParams(block_size=w.block_size, top_k=w.top_k)
    res = O.decode_sequence(q, K[None], V[None], w.lengths[0], np.ones_like(q), p)[0]
    planted = si.planted_blocks(w, 0, 0)
    assert set(int(i) for i in planted) <= set(int(i) for i in res.sel)
    top2 = np.argsort(-res.score)[:2]
    assert set(int(i) for i in top2) == set(int(i) for i in planted)


# -------------------------------------------------------------------- X11
def test_x11_rla_normaliser_is_scale_only():
    """RMSNorm is invariant to a positive rescaling of its input when eps is
    negligible, so dividing the residual by <phi(q), z_bar - z_tilde> (> 0)
    leaves the output unchanged."""
    r = _rng(11)
    Hq, Hkv, d, B, L = 4, 2, 16, 8, 99
    q = r.standard_normal((Hq, d))
    K = r.standard_normal((Hkv, L, d))
    V = r.standard_normal((Hkv, L, d))
    g = 1 + 0.1 * r.standard_normal((Hq, d))
    a = O.SplaParams(block_size=B, top_k=4, n_local=1, rms_eps=1e-300)
    b = O.SplaParams(block_size=B, top_k=4, n_local=1, rms_eps=1e-300, rla_normalize=True)
    ra = O.decode_sequence(q, K, V, L, g, a)
    rb = O.decode_sequence(q, K, V, L, g, b)
    for x, y in zip(ra, rb):
        np.testing.assert_allclose(x.out, y.out, rtol=0, atol=1e-12)
        assert not np.allclose(x.r, y.r)


# -------------------------------------------------------------------- X12
def test_x12_constant_values_closed_form():
    """V = v0 for every token: the exact branch returns v0, the residual is a
    positive multiple of v0, so o = v0 + gamma v0 / rms(v0) (eps -> 0)."""
    r = _rng(12)
    d, B, L, G = 16, 8, 90, 2
    v0 = r.standard_normal(d)
    K = r.standard_normal((L, d))
    V = np.repeat(v0[None], L, 0)
    q = r.standard_normal((G, d))
    g = 1 + 0.1 * r.standard_normal((G, d))
    p = O.SplaParams(block_size=B, top_k=3, n_local=1, rms_eps=1e-300)
    res = O.decode_kv_head(q, O.build_state(K, V, L, B), K, V, g, p)
    ref = v0 + g * v0 / np.sqrt((v0 * v0).mean())
    np.testing.assert_allclose(res.out, ref, rtol=0, atol=1e-12)


def test_x12_identical_keys_closed_form():
    """All keys equal: exact attention is the mean of the selected values,
    every phi(q).phi(k_t) is the same constant, so the residual is a positive
    multiple of the sum of the unselected values; with the block scores all
    equal (full blocks) the tie rule picks the lowest-index blocks."""
    r = _rng(121)
    d, B, L, G, k = 16, 8, 8 * 12 + 3, 3, 5
    K = np.repeat(r.standard_normal((1, d)), L, 0)
    V = r.standard_normal((L, d))
    q = r.standard_normal((G, d))
    g = 1 + 0.1 * r.standard_normal((G, d))
    eps = 1e-6
    p = O.SplaParams(block_size=B, top_k=k, n_sink=1, n_local=1, rms_eps=eps)
    st = O.build_state(K, V, L, B)
    res = O.decode_kv_head(q, st, K, V, g, p)
    nb = 13
    assert list(res.sel) == [0, 1, 2, 3, nb - 1]
    tok = np.concatenate([np.arange(i * B, min((i + 1) * B, L)) for i in res.sel])
    uns = np.setdiff1d(np.arange(L), tok)
    c = t_softmax(q) @ t_softmax(K[0])          # [G]
    rr = c[:, None] * V[uns].sum(axis=0)[None]
    ref = V[tok].mean(axis=0)[None] + g * rr / np.sqrt((rr * rr).mean(axis=1, keepdims=True) + eps)
    np.testing.assert_allclose(res.out, ref, rtol=0, atol=1e-12)


# -------------------------------------------------------------------- X13
def test_x13_streaming_stats_and_state_match_textbook():
    """Welford streaming statistics equal the two-pass mean / population
    variance; S_bar equals phi(K)^T V and z_bar the column sums of phi(K);
    phi is the softmax over the feature dimension."""
    r = _rng(13)
    d, B, L = 12, 16, 16 * 5 + 9
    K = r.standard_normal((L, d)) * 3 + 5
    V = r.standard_normal((L, d))
    st = O.append_state(None, K, V, B)
    for i in range(-(-L // B)):
        blk = K[i * B:min((i + 1) * B, L)]
        np.testing.assert_allclose(st.mean[i], blk.mean(0), rtol=1e-13)
        np.testing.assert_allclose(st.var[i], blk.var(0), rtol=1e-11)
        assert st.counts[i] == len(blk)
    phk = t_softmax(K)
    np.testing.assert_allclose(st.s_bar, torch.einsum("ti,tj->ij", torch.tensor(phk),
                                                      torch.tensor(V)).numpy(), rtol=1e-12)
    np.testing.assert_allclose(st.z_bar, phk.sum(0), rtol=1e-12)
    np.testing.assert_allclose(O.feature_map(K), phk, rtol=1e-13)
    np.testing.assert_allclose(O.feature_map(K).sum(-1), 1.0, rtol=1e-14)
    two = O.build_state(K, V, L, B)
    np.testing.assert_allclose(two.s_bar, st.s_bar, rtol=1e-12)


# -------------------------------------------------------------------- X14
def test_x14_append_chunking_invariance():
    """Appending tokens in chunks of any size gives the same state as
    appending them all at once (and as building it from scratch)."""
    r = _rng(14)
    d, B, L = 8, 8, 61
    K = r.standard_normal((L, d))
    V = r.standard_normal((L, d))
    whole = O.append_state(None, K, V, B)
    st = None
    cuts = [0, 1, 2, 9, 16, 17, 40, 61]
    for a, b in zip(cuts[:-1], cuts[1:]):
        st = O.append_state(st, K[a:b], V[a:b], B)
    ref = O.build_state(K, V, L, B)
    for x in (st, whole):
        assert x.length == L
        np.testing.assert_allclose(x.mean, ref.mean, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(x.var, ref.var, rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(x.s_bar, ref.s_bar, rtol=1e-12)
        np.testing.assert_allclose(x.z_bar, ref.z_bar, rtol=1e-12)
        assert np.array_equal(x.counts, ref.counts)


# --------------------------------------------------------------- extras
def test_forced_blocks_always_selected_even_with_lowest_scores():
    """The sink block and the n_local most recent blocks are selected even
    when their keys point away from the query (Sec. 4)."""
    r = _rng(15)
    d, B, L = 16, 8, 8 * 20
    q = r.standard_normal((1, d))
    K = r.standard_normal((L, d))
    K[:B] -= 3 * q / np.linalg.norm(q)
    K[-3 * B:] -= 3 * q / np.linalg.norm(q)
    V = r.standard_normal((L, d))
    p = O.SplaParams(block_size=B, top_k=6, n_sink=1, n_local=3)
    res = O.decode_kv_head(q, O.build_state(K, V, L, B), K, V, np.ones((1, d)), p)
    assert {0, 17, 18, 19} <= set(int(i) for i in res.sel)
    assert len(res.sel) == 6
    low = np.argsort(res.score)[:4]
    assert set(int(i) for i in low) == {0, 17, 18, 19}


def test_no_rla_returns_exact_branch_and_first_order_drops_variance():
    r = _rng(16)
    d, B, L, G = 16, 8, 70, 2
    q = r.standard_normal((G, d))
    K = r.standard_normal((L, d))
    V = r.standard_normal((L, d))
    st = O.build_state(K, V, L, B)
    p = O.SplaParams(block_size=B, top_k=3, n_local=1, no_rla=True)
    res = O.decode_kv_head(q, st, K, V, np.ones((G, d)), p)
    np.testing.assert_array_equal(res.out, res.o_sparse)
    p1 = O.SplaParams(block_size=B, top_k=3, n_local=1, first_order=True)
    res1 = O.decode_kv_head(q, st, K, V, np.ones((G, d)), p1)
    s = 1 / math.sqrt(d)
    nb = -(-L // B)
    cnt = np.array([min(B, L - i * B) for i in range(nb)])
    mus = np.array([K[i * B:min((i + 1) * B, L)].mean(0) for i in range(nb)])
    np.testing.assert_allclose(res1.ell, s * q @ mus.T + np.log(cnt), rtol=1e-13)


def test_empty_sequence_decodes_to_zero():
    d = 8
    st = O.build_state(np.zeros((0, d)), np.zeros((0, d)), 0, 4)
    res = O.decode_kv_head(np.ones((2, d)), st, np.zeros((0, d)), np.zeros((0, d)),
                           np.ones((2, d)), O.SplaParams(block_size=4, top_k=2))
    assert np.all(res.out == 0) and len(res.sel) == 0


def test_block_ranges_cover_ragged_lengths():
    for L, B in [(1, 64), (64, 64), (65, 64), (1000, 64), (131, 128)]:
        rg = O.block_ranges(L, B)
        assert len(rg) == -(-L // B)
        assert sum(b - a for a, b in rg) == L
        assert rg[-1][1] == L


# -------------------------------------------------------------------- X21
# Hand-worked top-k cutoffs. Each case: scores, k, n_sink, n_local, the
# selection worked out by hand, the cutoff (score of the lowest-scored
# non-forced admitted block, None when every block is taken or nothing is
# admitted by rank) and the blocks whose score equals the cutoff.
CUTOFF_CASES = {
    # forced {0, 8, 9} hold the three lowest scores; kp = 2 admits 2 and 4
    "forced_lowest": ([0.01, 0.5, 0.9, 0.3, 0.7, 0.2, 0.6, 0.4, 0.02, 0.03], 5, 1, 2,
                      [0, 2, 4, 8, 9], 0.7, [4]),
    # forced {0, 7}; kp = 2: block 2 (0.8), then the first of the three-way
    # tie at 0.5 (blocks 1, 3, 4) by the lower id
    "tie_at_cutoff": ([0.1, 0.5, 0.8, 0.5, 0.5, 0.2, 0.3, 0.05], 4, 1, 1,
                      [0, 1, 2, 7], 0.5, [1, 3, 4]),
    # no forced blocks: the plain top 3 of 6
    "no_forced": ([0.3, 0.1, 0.6, 0.6, 0.2, 0.5], 3, 0, 0, [2, 3, 5], 0.5, [5]),
    # nb <= k: every block, no cutoff
    "all_selected": ([0.4, 0.1, 0.3, 0.2], 4, 1, 2, [0, 1, 2, 3], None, []),
    # k equals the forced count: nothing admitted by rank, no cutoff
    "forced_only": ([0.9, 0.8, 0.7, 0.1, 0.2, 0.3], 3, 1, 2, [0, 4, 5], None, []),
}


@pytest.mark.parametrize("name", list(CUTOFF_CASES))
def test_x21_cutoff_score_hand_worked(name):
    """The tie window of index parity is measured from the cutoff: the score
    of the last block admitted by rank (forced blocks excluded)."""
    score, k, n_sink, n_local, sel_want, cut_want, at_cut = CUTOFF_CASES[name]
    score = np.array(score, dtype=float)
    sel = O.select_blocks(score, k, n_sink, n_local)
    assert [int(i) for i in sel] == sel_want
    c = O.cutoff_score(score, sel, k, n_sink, n_local)
    if cut_want is None:
        assert c is None
    else:
        assert c == cut_want
        assert [i for i in range(len(score)) if abs(score[i] - c) <= 1e-6 * c] == at_cut


# -------------------------------------------------------------------- X22
@pytest.mark.parametrize("seed", range(3))
def test_x22_rla_normaliser_is_the_unselected_linear_mass(seed):
    """With the normaliser switched on, the residual is divided by
    <phi(q), z_bar - z_tilde>, which is the linear-attention weight of the
    unselected tokens, sum over t not in T_I of <phi(q), phi(k_t)>, summed
    here by brute force with an independent softmax."""
    r = _rng(22, seed)
    G, d, B, L, k = 3, 16, 8, 83, 4
    q = 0.7 * r.standard_normal((G, d))
    K = r.standard_normal((L, d))
    V = r.standard_normal((L, d))
    g = np.ones((G, d))
    st = O.build_state(K, V, L, B)
    pa = O.SplaParams(block_size=B, top_k=k, n_local=1)
    pb = O.SplaParams(block_size=B, top_k=k, n_local=1, rla_normalize=True)
    a = O.decode_kv_head(q, st, K, V, g, pa)
    b = O.decode_kv_head(q, st, K, V, g, pb, force_selection=a.sel)
    sel_tok = set()
    for i in a.sel:
        sel_tok |= set(range(int(i) * B, min((int(i) + 1) * B, L)))
    unsel = [t for t in range(L) if t not in sel_tok]
    assert len(unsel) > 0
    phq = t_softmax(q)
    phk = t_softmax(K[unsel])
    den = np.array([sum(float(np.dot(phq[m], phk[j])) for j in range(len(unsel)))
                    for m in range(G)])
    ratio = a.r / b.r                     # the denominator, once per coordinate
    for m in range(G):
        np.testing.assert_allclose(ratio[m], den[m], rtol=1e-10, atol=0)


# -------------------------------------------------------------------- X23
@pytest.mark.parametrize("L", [37, 64])
def test_x23_every_block_selected_with_zero_eps_is_dense_attention(L):
    """k >= nb with eps = 0: no token is unselected, the residual branch is
    absent, and the output is dense attention (Eq. 1), not 0 / 0."""
    r = _rng(23, L)
    Hq, Hkv, d, B = 4, 2, 16, 8
    q = r.standard_normal((Hq, d))
    K = r.standard_normal((Hkv, L, d))
    V = r.standard_normal((Hkv, L, d))
    gamma = 1 + 0.1 * r.standard_normal((Hq, d))
    p = O.SplaParams(block_size=B, top_k=8, rms_eps=0.0)
    res = O.decode_sequence(q, K, V, L, gamma, p)
    out = np.concatenate([x.out for x in res])
    assert np.all(np.isfinite(out))
    ref = sdpa(q, K, V, 1 / math.sqrt(d))
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
