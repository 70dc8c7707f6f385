"""GPU tests of the two-stage selection (more than 4096 blocks per sequence on
the separate launches): slices of 1024 blocks take their own top candidates,
then one workgroup per (sequence, KV head) picks from them.

The slices' keys are formed with the single workgroup's arithmetic, so at a
shape the single-launch kernel also covers (at most 8192 blocks) both paths
must agree bit for bit; every unit is also checked against the oracle, and
exact ties spread over several slices must go to the lower block ids.
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


def test_two_stage_matches_single_launch_and_oracle(dev):
    """4608 blocks of capacity: the separate launches select in two stages,
    the single launch in one workgroup. Lengths cover every slice, fewer
    slices than the capacity holds, and a sequence whose blocks all fit in k."""
    B, cap = 32, 4608 * 32
    w = si.custom("two_stage", 3, 8, 2, 128, B, 24, [cap - 37, 70001, 200], kind="block_offsets",
                  code=200, capacity=cap)
    res = []
    for flags in (0, spla.FLAG_SEPARATE_KERNELS):
        cfg = H.config_of(w, flags=flags)
        cache = spla.SplaCache(cfg, dev)
        H.fill_cache(w, cache, device=dev)
        q, gamma = si.gen_q_batch(w), si.gen_gamma(w)
        out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
        torch.cuda.synchronize()
        assert cache.device_errors() == 0
        res.append((out, sel))
    assert spla.decode_phases(H.config_of(w)) == ["decode"]
    assert torch.equal(res[0][1], res[1][1]) and torch.equal(res[0][0], res[1][0])
    out = res[1][0].float().cpu().numpy()
    sel = res[1][1].cpu().numpy()
    p = H.params_of(w)
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], q[b], gamma, p)


def test_two_stage_ties_across_slices_go_to_the_lower_ids(dev):
    """Seven copies of one strongly relevant block in five different slices;
    k leaves room for five of them, so the tie at the cutoff spans slices and
    only the five lowest ids may be taken."""
    B, d, k = 32, 128, 8
    L = 4200 * B
    w = si.custom("ties2", 1, 4, 1, d, B, k, [L], kind="iid", code=201, n_sink=1, n_local=2)
    K, V = si.gen_kv(w, 0, 0, 0, L)
    qv = si.gen_q_batch(w)
    hot = [5, 700, 1030, 1500, 2100, 3100, 4150]
    qdir = qv[0].astype(np.float64).mean(axis=0)
    qdir /= np.linalg.norm(qdir)
    base = si.round_bf16(K[hot[0] * B:(hot[0] + 1) * B] +
                         si.round_bf16((3.0 * qdir).astype(np.float32)))
    for i in hot:
        K[i * B:(i + 1) * B] = base
    cache = spla.SplaCache(H.config_of(w, flags=spla.FLAG_SEPARATE_KERNELS), dev)
    cache.append(H.to_dev(K[None, None], w, dev), H.to_dev(V[None, None], w, dev),
                 torch.tensor([L], dtype=torch.int32, device=dev))
    gamma = si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(qv, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    st = O.build_state(K, V, L, B)
    r = O.decode_kv_head(qv[0], st, K, V, gamma, H.params_of(w))
    nb = L // B
    assert [int(x) for x in r.sel] == [0] + hot[:5] + [nb - 2, nb - 1]
    assert r.score[hot[5]] == r.score[hot[4]]
    assert [int(x) for x in sel.cpu().numpy()[0, 0]] == [int(x) for x in r.sel]
    assert H.row_rel_err(out.float().cpu().numpy()[0], r.out) <= H.TOL["bf16"]


def test_two_stage_with_many_candidates(dev):
    """k = 256 over ten slices (2560 candidate slots, four per thread of the
    pick), G = 8, d = 64."""
    w = si.custom("two_stage_k256", 1, 8, 1, 64, 32, 256, [300000], kind="pareto_planted",
                  n_planted=12, code=202)
    cache = spla.SplaCache(H.config_of(w), dev)
    H.fill_cache(w, cache, device=dev)
    q, gamma = si.gen_q_batch(w), si.gen_gamma(w)
    out, sel = cache.decode(H.to_dev(q, w, dev), torch.from_numpy(gamma).to(dev))
    torch.cuda.synchronize()
    assert cache.device_errors() == 0
    H.check_kv_head(w, 0, 0, out.float().cpu().numpy()[0], sel.cpu().numpy()[0, 0], q[0], gamma,
                    H.params_of(w))
