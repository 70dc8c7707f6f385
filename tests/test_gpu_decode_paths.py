"""The single-launch decode kernel against the separate-kernel path.

Both run the same device arithmetic (block scoring, selection, fused sparse
pass, merge), so on the same cache and query they must agree bit for bit,
selection included. Also checks the single-launch kernel's workspace
protocol: its counters are zero after every call, repeated calls give the same
bits, and a counter that no call left behind (a workspace not prepared by
spla_workspace_init) makes the affected waits give up at their bound, which
is reported through err_flags, until spla_workspace_init repairs it.
"""

import ctypes

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


SYNC_LINE = 32  # int32 words per counter line


def sync_area(cfg, cache):
    """The synchronisation area at the end of the decode workspace: a line
    with the error word, then per (sequence, KV head) a score-item counter
    line and a record counter line, then the selection words ([bh][k], then
    4 words of padding, rounded up to whole lines). Returns the words and
    the offset of the score-item counters."""
    bh = cfg.batch * cfg.n_kv_heads
    items_done = SYNC_LINE
    n = items_done + 2 * bh * SYNC_LINE + -(-(bh * cfg.top_k + 4) // SYNC_LINE) * SYNC_LINE
    span = -(-n * 4 // spla.WORKSPACE_ALIGN) * spla.WORKSPACE_ALIGN
    total = spla.workspace_bytes(cfg)
    return cache.workspace[total - span:total - span + 4 * n].view(torch.int32), items_done


def sync_words(cfg, cache):
    return sync_area(cfg, cache)[0]


def decode_with(cache, cfg, q, gamma):
    out = torch.empty_like(q)
    sel = torch.full((cfg.batch, cfg.n_kv_heads, cfg.top_k), -7, dtype=torch.int32,
                     device=q.device)
    st = spla.lib().spla_decode(ctypes.byref(cfg), ctypes.byref(cache.struct),
                                spla._ptr(q), spla._ptr(gamma), spla._ptr(out), spla._ptr(sel),
                                spla._ptr(cache.workspace), cache.workspace.numel(),
                                spla._stream(q.device))
    assert st == 0, spla.STATUS.get(st)
    return out, sel


def prepare(name, dev, code, **spec):
    w = si.custom(name, code=code, **spec)
    cfg = H.config_of(w)
    cache = spla.SplaCache(cfg, dev)
    H.fill_cache(w, cache, lengths=list(w.lengths), device=dev)
    q = H.to_dev(si.gen_q_batch(w), w, dev)
    gamma = torch.from_numpy(si.gen_gamma(w)).to(dev)
    return w, cfg, cache, q, gamma


SHAPES = {
    "g4_B64_ragged": dict(batch=7, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64,
                          top_k=8, lengths=[1, 63, 64, 65, 512, 513, 9000], kind="iid"),
    "g5_B64": dict(batch=2, n_q_heads=10, n_kv_heads=2, head_dim=128, block_size=64, top_k=8,
                   lengths=[4097, 2500], kind="block_offsets"),
    "g1_B32_empty": dict(batch=3, n_q_heads=4, n_kv_heads=4, head_dim=128, block_size=32,
                         top_k=6, lengths=[0, 300, 31], kind="iid"),
    "g6_B128_var": dict(batch=5, n_q_heads=12, n_kv_heads=2, head_dim=128, block_size=128,
                        top_k=7, lengths=[70000, 16384, 4000, 128, 40000], capacity=70016,
                        kind="iid"),
    "g3_B64_8k_blocks": dict(batch=1, n_q_heads=6, n_kv_heads=2, head_dim=128, block_size=64,
                             top_k=24, lengths=[8192 * 64 - 5], kind="pareto_planted",
                             n_planted=4),
    # 128 units x (4 score + 4 sparse items) = 1024 items: the four-wave build
    "g4_B32_four_waves": dict(batch=32, n_q_heads=16, n_kv_heads=4, head_dim=128,
                              block_size=32, top_k=16, lengths=[8192 - 37 * i for i in range(32)],
                              capacity=8192, kind="block_offsets"),
}


@pytest.mark.parametrize("name", list(SHAPES))
def test_single_launch_matches_separate_kernels(dev, name):
    H.log(f"case {name}")
    w, cfg, cache, q, gamma = prepare(name, dev, 300 + list(SHAPES).index(name),
                                      **SHAPES[name])
    cfg_sep = H.config_of(w, flags=spla.FLAG_SEPARATE_KERNELS)
    o1, s1 = decode_with(cache, cfg, q, gamma)
    o2, s2 = decode_with(cache, cfg_sep, q, gamma)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert int(cache.err.item()) == 0
    assert int(sync_words(cfg, cache).abs().sum().item()) == 0
    # and the single-launch result is the oracle's on a few (sequence, KV head) units
    qn, gn = q.float().cpu().numpy(), gamma.cpu().numpy()
    out, sel = o1.float().cpu().numpy(), s1.cpu().numpy()
    p = H.params_of(w)
    for b in range(min(w.batch, 3)):
        for h in range(w.n_kv_heads):
            H.check_kv_head(w, b, h, out[b], sel[b, h], qn[b], gn, p)


def test_repeated_calls_leave_counters_zero(dev):
    w, cfg, cache, q, gamma = prepare("repeat", dev, 320, **SHAPES["g4_B64_ragged"])
    ref_o, ref_s = decode_with(cache, cfg, q, gamma)
    for _ in range(5):
        o, s = decode_with(cache, cfg, q, gamma)
        torch.cuda.synchronize()
        assert torch.equal(s, ref_s)
        assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
        assert int(sync_words(cfg, cache).abs().sum().item()) == 0
    assert int(cache.err.item()) == 0


def test_counter_left_behind_is_reported_then_repaired(dev):
    w, cfg, cache, q, gamma = prepare("unprepared", dev, 321, **SHAPES["g5_B64"])
    ref_o, ref_s = decode_with(cache, cfg, q, gamma)
    torch.cuda.synchronize()
    words, items_done = sync_area(cfg, cache)
    # the score-item counter of (sequence 0, KV head 0) as no call leaves it:
    # its selection never runs, so the workgroups left waiting for its sparse
    # items give up at their bound
    words[items_done] = 1 << 20
    torch.cuda.synchronize()
    H.log("decode with a stale counter (the waits of one head give up after about a second)")
    decode_with(cache, cfg, q, gamma)
    torch.cuda.synchronize()
    assert int(cache.err.item()) & spla.DEVERR_SYNC
    st = spla.lib().spla_workspace_init(ctypes.byref(cfg), spla._ptr(cache.workspace),
                                        cache.workspace.numel(), spla._stream(dev))
    assert st == 0
    cache.err.zero_()
    o, s = decode_with(cache, cfg, q, gamma)
    torch.cuda.synchronize()
    assert torch.equal(s, ref_s)
    assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
    assert int(cache.err.item()) == 0
    assert int(sync_words(cfg, cache).abs().sum().item()) == 0
