"""GPU guards: edge cases of the decode and append paths that the parity
tests do not reach on their own.

* eps = 0 with every block selected (no residual: the output is exact
  attention, not 0 / 0), on both decode paths;
* the RLA normaliser with an eps large enough that a wrong denominator
  would move the output past the tolerance (checked on the CPU first);
* exact ties in the top-k: duplicated key blocks inside one statistics tile,
  where the selection must equal the oracle's lower-id choice with no tie
  window;
* spla_append without a per-sequence count (n_new = NULL);
* spla_step on a sequence already at capacity: state untouched, flag set.
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


def _decode(cache, w, q, gamma, dev):
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), sel.cpu().numpy()


def _softmax(x):
    e = np.exp(x - x.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


@pytest.mark.parametrize("separate", [False, True])
def test_zero_eps_with_every_block_selected(dev, separate):
    w = si.custom("eps0", 3, 8, 2, 128, 64, 8, [512, 300, 1], kind="block_offsets", code=130)
    flags = spla.FLAG_SEPARATE_KERNELS if separate else 0
    cfg = H.config_of(w, flags=flags, rms_eps=0.0)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, device=dev)
    q, gamma = si.gen_q_batch(w), si.gen_gamma(w)
    out, sel = _decode(cache, w, q, gamma, dev)
    assert np.all(np.isfinite(out))
    p = H.params_of(w, rms_eps=0.0)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p)
    assert cache.device_errors() == 0


def test_rla_normaliser_is_visible_in_the_output(dev):
    """eps of the order of mean((r / den)^2): the output then depends on the
    denominator <phi(q), z_bar - z_tilde>, and the oracle computed with
    <phi(q), z_bar> instead (a plausible kernel mistake) is shown to differ by
    more than the tolerance before the GPU is compared with the right one."""
    w = si.custom("normeps", 2, 8, 2, 128, 64, 8, [1500, 2000], kind="block_offsets", code=131)
    q, gamma = si.gen_q_batch(w), si.gen_gamma(w)
    pn = H.params_of(w, rla_normalize=True)
    ms = []
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            res, _, _, _ = H.oracle_kv_head(w, b, h, gamma, q[b], pn)
            ms.extend(float(np.mean(r * r)) for r in res.r)
    eps = float(np.float32(np.median(ms)))
    p = H.params_of(w, rla_normalize=True, rms_eps=eps)
    G = w.group
    gap = []
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            res, st, K, V = H.oracle_kv_head(w, b, h, gamma, q[b], p)
            tok = O.selected_token_indices(res.sel, w.lengths[b], w.block_size)
            phq = _softmax(q[b, h * G:(h + 1) * G].astype(np.float64))
            r_num = res.o_bar - res.o_tilde
            wrong = r_num / (phq @ st.z_bar)[:, None]
            g = gamma[h * G:(h + 1) * G]
            o_wrong = res.o_sparse + g * wrong / np.sqrt((wrong ** 2).mean(-1, keepdims=True) + eps)
            gap.append(H.row_rel_err(o_wrong, res.out))
            assert len(tok) < w.lengths[b]
    assert min(gap) > 3 * H.TOL["bf16"], gap
    for separate in (False, True):
        flags = spla.FLAG_RLA_NORMALIZE | (spla.FLAG_SEPARATE_KERNELS if separate else 0)
        cfg = H.config_of(w, flags=flags, rms_eps=eps)
        cache = spla.SplaCache(cfg, dev)
        H.fill_cache(w, cache, device=dev)
        out, sel = _decode(cache, w, q, gamma, dev)
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p)


# copies of one strongly relevant block; k leaves room for five of them. The
# selection's output stage reads 32 blocks per lane: the cutoff falls between
# two lanes (the first set), inside a lane that keeps part of its ties (the
# second) and inside the second lane after the first lane's tie (the third).
TIE_CASES = [
    ([5, 9, 17, 23, 30, 41], [0, 5, 9, 17, 23, 30, 46, 47]),
    ([5, 9, 17, 23, 30, 31, 41], [0, 5, 9, 17, 23, 30, 46, 47]),
    ([3, 40, 41, 42, 43, 44], [0, 3, 40, 41, 42, 43, 46, 47]),
]


@pytest.mark.parametrize("separate", [False, True])
@pytest.mark.parametrize("hot,expect", TIE_CASES)
def test_duplicated_blocks_tie_to_the_lower_id(dev, separate, hot, expect):
    """Copies of one strongly relevant block inside the first statistics
    tile; k leaves room for five of them, so the tie falls exactly on the
    cutoff and only the lowest five ids may be taken."""
    B, d, L, k = 64, 128, 48 * 64, 8
    w = si.custom("ties", 1, 4, 1, d, B, k, [L], kind="iid", code=132, n_sink=1, n_local=2)
    K, V = si.gen_kv(w, 0, 0, 0, L)
    qv = si.gen_q_batch(w)
    qdir = qv[0].astype(np.float64).mean(axis=0)
    qdir /= np.linalg.norm(qdir)
    base = K[hot[0] * B:(hot[0] + 1) * B] + si.round_bf16((3.0 * qdir).astype(np.float32))
    base = si.round_bf16(base)
    for i in hot:
        K[i * B:(i + 1) * B] = base
    cfg = H.config_of(w, flags=spla.FLAG_SEPARATE_KERNELS if separate else 0)
    cache = spla.SplaCache(cfg, dev)
    cache.append(H.to_dev(K[None, None], w, dev), H.to_dev(V[None, None], w, dev),
                 torch.tensor([L], dtype=torch.int32, device=dev))
    gamma = si.gen_gamma(w)
    out, sel = _decode(cache, w, qv, gamma, dev)
    p = H.params_of(w)
    st = O.build_state(K, V, L, B)
    res = O.decode_kv_head(qv[0], st, K, V, gamma, p)
    assert [int(x) for x in res.sel] == expect
    assert res.score[hot[5]] == res.score[hot[4]]
    assert [int(x) for x in sel[0, 0]] == [int(x) for x in res.sel]
    assert H.row_rel_err(out[0], res.out) <= H.TOL["bf16"]


def test_append_without_counts(dev):
    """n_new = NULL appends all max_new rows of every sequence."""
    w = si.custom("nonull", 2, 8, 2, 128, 64, 8, [1500, 1500], kind="drift", code=133,
                  capacity=4096)
    cfg = H.config_of(w)
    cache = spla.SplaCache(cfg, dev)
    for t0, t1 in [(0, 1000), (1000, 1500)]:
        K, V, _ = si.gen_kv_slab(w, t0, t1)
        cache.append(H.to_dev(K, w, dev), H.to_dev(V, w, dev), None)
    torch.cuda.synchronize()
    assert cache.seq_lens.cpu().tolist() == [1500, 1500]
    mean, m2 = (x.cpu().numpy() for x in cache.stats_logical())
    S, z = (x.cpu().numpy() for x in cache.state_logical())
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            K, V = si.gen_kv(w, b, h, 0, 1500)
            st = O.build_state(K, V, 1500, w.block_size)
            nb = len(st.counts)
            np.testing.assert_allclose(mean[b, h, :nb], st.mean, rtol=0, atol=2e-6)
            np.testing.assert_allclose(m2[b, h, :nb] / st.counts[:, None], st.var, rtol=2e-5,
                                       atol=1e-6)
            np.testing.assert_allclose(S[b, h], st.s_bar, rtol=2e-4, atol=2e-4)
            np.testing.assert_allclose(z[b, h], st.z_bar, rtol=2e-5, atol=1e-5)
    q, gamma = si.gen_q_batch(w), si.gen_gamma(w)
    out, sel = _decode(cache, w, q, gamma, dev)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, H.params_of(w))
    assert cache.device_errors() == 0


@pytest.mark.parametrize("separate", [False, True])
def test_step_at_capacity_leaves_the_state_unchanged(dev, separate):
    w = si.custom("stepcap", 2, 8, 2, 128, 64, 6, [512, 300], kind="iid", code=134,
                  capacity=512)
    cfg = H.config_of(w, flags=spla.FLAG_SEPARATE_KERNELS if separate else 0)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, device=dev)
    torch.cuda.synchronize()
    before = {n: getattr(cache, n).clone() for n in ("stats", "state", "norm", "seq_lens")}
    assert cache.device_errors() == 0
    rng = np.random.default_rng(134)
    kn = si.round_bf16(rng.standard_normal((2, 2, 128)).astype(np.float32))
    vn = si.round_bf16(rng.standard_normal((2, 2, 128)).astype(np.float32))
    q, gamma = si.gen_q_batch(w), si.gen_gamma(w)
    out, sel = cache.step(H.to_dev(kn, w, dev), H.to_dev(vn, w, dev), H.to_dev(q, w, dev),
                          torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    assert cache.device_errors() & spla.DEVERR_CAPACITY
    assert cache.seq_lens.cpu().tolist() == [512, 301]
    # sequence 0 (full) untouched; sequence 1 gained its token
    for n in ("stats", "state", "norm"):
        a = before[n].view(2, -1)[0]
        b = getattr(cache, n).view(2, -1)[0]
        assert torch.equal(a, b), n
    out = out.float().cpu().numpy()
    sel = sel.cpu().numpy()
    p = H.params_of(w)
    for h in range(w.n_kv_heads):
        H.check_kv_head(w, 0, h, out[0], sel[0, h], q[0], gamma, p, L=512)
    # the clipped token never reached sequence 0, and sequence 1 sees its new row
    S, z = (x.cpu().numpy() for x in cache.state_logical())
    for h in range(w.n_kv_heads):
        K, V = si.gen_kv(w, 1, h, 0, 300)
        K = np.concatenate([K, kn[1, h][None]])
        V = np.concatenate([V, vn[1, h][None]])
        st = O.build_state(K, V, 301, w.block_size)
        np.testing.assert_allclose(S[1, h], st.s_bar, rtol=2e-5, atol=2e-5)
        res = O.decode_kv_head(q[1, h * w.group:(h + 1) * w.group], st, K, V,
                               gamma[h * w.group:(h + 1) * w.group], p)
        assert [int(x) for x in sel[1, h][:len(res.sel)]] == [int(x) for x in res.sel]
        assert H.row_rel_err(out[1, h * w.group:(h + 1) * w.group], res.out) <= H.TOL["bf16"]


@pytest.mark.parametrize("d,B,k", [(128, 128, 16), (128, 64, 32)])
def test_fused_step_equals_separate_step(dev, d, B, k):
    """spla_step folds the token's rank-one update of S_bar into the rows the
    decode's sparse pass reads, on the single launch and on the separate
    launches alike; three steps must leave the same cache (statistics,
    S_bar, z_bar, K/V rows, lengths) and give the same outputs and
    selections, bit for bit, on both, also for a sequence at capacity. The
    state after the steps matches the oracle's state built from every row
    the cache holds, and the outputs match the oracle."""
    cap = 32 * B
    w = si.custom(f"fstep{B}", 3, 8, 2, d, B, k, [cap - 700, 17 * B + 5, cap], kind="drift",
                  code=135 + B, capacity=cap)
    caches = []
    for flags in (0, spla.FLAG_SEPARATE_KERNELS):
        c = spla.SplaCache(H.config_of(w, flags=flags), dev)
        H.fill_cache(w, c, device=dev)
        caches.append(c)
    assert spla.decode_phases(caches[0].cfg) == ["decode"]
    gamma = si.gen_gamma(w)
    rng = np.random.default_rng(136)
    p = H.params_of(w)
    for step in range(3):
        kn = si.round_bf16(rng.standard_normal((3, 2, d)).astype(np.float32))
        vn = si.round_bf16(rng.standard_normal((3, 2, d)).astype(np.float32))
        q = si.gen_q_batch(w, step)
        res = [c.step(H.to_dev(kn, w, dev), H.to_dev(vn, w, dev), H.to_dev(q, w, dev),
                      torch.from_numpy(gamma).to(dev)) for c in caches]
        torch.cuda.synchronize()
        assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1]), step
        for n in ("k", "v", "stats", "state", "norm", "seq_lens"):
            assert torch.equal(getattr(caches[0], n), getattr(caches[1], n)), (step, n)
    assert caches[0].device_errors() & spla.DEVERR_CAPACITY
    # the oracle on sequence 1 after the three steps (its appended rows are the
    # random ones above)
    out = res[0][0].float().cpu().numpy()
    sel = res[0][1].cpu().numpy()
    L = w.lengths[1] + 3
    kl = caches[0].k_logical()[1, :, :L].float().cpu().numpy()
    vl = caches[0].v_logical()[1, :, :L].float().cpu().numpy()
    S, z = (x.cpu().numpy() for x in caches[0].state_logical())
    for b in range(3):
        Lb = min(w.lengths[b] + 3, cap)
        kb = caches[0].k_logical()[b, :, :Lb].float().cpu().numpy()
        vb = caches[0].v_logical()[b, :, :Lb].float().cpu().numpy()
        for h in range(2):
            st = O.build_state(kb[h], vb[h], Lb, B)
            np.testing.assert_allclose(S[b, h], st.s_bar, rtol=2e-4, atol=2e-4)
            np.testing.assert_allclose(z[b, h], st.z_bar, rtol=2e-5, atol=1e-5)
    for h in range(2):
        st = O.build_state(kl[h], vl[h], L, B)
        r = O.decode_kv_head(q[1, h * 4:(h + 1) * 4], st, kl[h], vl[h],
                             gamma[h * 4:(h + 1) * 4], p)
        assert [int(x) for x in sel[1, h][:len(r.sel)]] == [int(x) for x in r.sel]
        assert H.row_rel_err(out[1, h * 4:(h + 1) * 4], r.out) <= H.TOL["bf16"]
