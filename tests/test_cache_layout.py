"""The bf16 K/V cache step order documented in include/spla.h against the
Python inverse (SplaCache.k_logical / v_logical): filling the raw buffers by
the documented formula from a known logical tensor must read back as that
tensor. The device side writes through the same formula (k_off / v_off) and
the GPU parity tests read its caches back through k_logical / v_logical."""

import numpy as np
import pytest
import torch

from paper_2601_22379_amd import spla


class _Cfg:
    def __init__(self, d, B, T, dtype, kv_pages=0):
        self.batch, self.n_kv_heads, self.head_dim = 2, 3, d
        self.block_size, self.max_seq_len, self.dtype = B, T, dtype
        self.kv_pages = kv_pages


def _cache(cfg, k_raw, v_raw, table=None):
    c = object.__new__(spla.SplaCache)
    c.cfg, c.k, c.v, c.block_table = cfg, k_raw, v_raw, table
    return c


def k_chunk(tt, c, d):
    return (((tt // 4) % 2) * (d // 32) + c // 32) * 64 + (c // 8) % 4 * 16 + 4 * (tt // 8) + tt % 4


def v_chunk(tt, c):
    return (c // 16) * 64 + (tt // 8) * 16 + c % 16


@pytest.mark.parametrize("d", [64, 128])
def test_bf16_step_order_roundtrip(d):
    cfg = _Cfg(d, 64, 128, spla.BF16)
    n = cfg.batch * cfg.n_kv_heads
    rng = np.random.default_rng(5)
    kl = rng.standard_normal((n, cfg.max_seq_len, d)).astype(np.float32)
    vl = rng.standard_normal((n, cfg.max_seq_len, d)).astype(np.float32)
    k_raw = np.zeros(n * cfg.max_seq_len * d, np.float32)
    v_raw = np.zeros_like(k_raw)
    for bh in range(n):
        for t in range(cfg.max_seq_len):
            base = (bh * cfg.max_seq_len + (t // 32) * 32) * d
            tt = t % 32
            for c in range(d):
                k_raw[base + k_chunk(tt, c, d) * 8 + c % 8] = kl[bh, t, c]
                v_raw[base + v_chunk(tt, c) * 8 + tt % 8] = vl[bh, t, c]
    cache = _cache(cfg, torch.from_numpy(k_raw), torch.from_numpy(v_raw))
    shape = (cfg.batch, cfg.n_kv_heads, cfg.max_seq_len, d)
    assert np.array_equal(cache.k_logical().numpy(), kl.reshape(shape))
    assert np.array_equal(cache.v_logical().numpy(), vl.reshape(shape))


def test_step_order_is_a_permutation():
    for d in (64, 128):
        ks = {k_chunk(tt, c, d) * 8 + c % 8 for tt in range(32) for c in range(d)}
        vs = {v_chunk(tt, c) * 8 + tt % 8 for tt in range(32) for c in range(d)}
        assert ks == set(range(32 * d)) and vs == set(range(32 * d))


def test_f32_layout_unchanged():
    cfg = _Cfg(64, 32, 64, spla.F32)
    n = cfg.batch * cfg.n_kv_heads
    k = torch.arange(n * 64 * 64, dtype=torch.float32)
    v = torch.arange(n * 64 * 64, dtype=torch.float32)
    cache = _cache(cfg, k, v)
    assert torch.equal(cache.k_logical().reshape(-1), k)
    vl = cache.v_logical()  # [b][h][t][c] from [b][h][t/B][c][t%B]
    assert vl[0, 0, 33, 5].item() == ((1 * 64 + 5) * 32 + 1)


@pytest.mark.parametrize("dtype", [spla.BF16, spla.F32])
def test_paged_pool_reads_back_through_the_block_table(dtype):
    """A paged pool (page p holds one block of every KV head at element
    (p * Hkv + h) * B * d) filled from a per-sequence buffer through a
    shuffled block table reads back as that buffer; unused pages are
    ignored."""
    d, B, T = 64, 32, 128
    flat = _Cfg(d, B, T, dtype)
    n = flat.batch * flat.n_kv_heads
    nb = T // B
    k = torch.arange(n * T * d, dtype=torch.float32)
    v = -torch.arange(n * T * d, dtype=torch.float32)
    pages = flat.batch * nb + 5
    rng = np.random.default_rng(9)
    table = torch.from_numpy(rng.permutation(pages)[:flat.batch * nb].reshape(flat.batch, nb)
                             .astype(np.int32))
    kp = torch.full((pages * flat.n_kv_heads * B * d,), 7.0)
    vp = kp.clone()
    for b in range(flat.batch):
        for h in range(flat.n_kv_heads):
            for i in range(nb):
                src = ((b * flat.n_kv_heads + h) * nb + i) * B * d
                dst = (int(table[b, i]) * flat.n_kv_heads + h) * B * d
                kp[dst:dst + B * d] = k[src:src + B * d]
                vp[dst:dst + B * d] = v[src:src + B * d]
    ref = _cache(flat, k, v)
    got = _cache(_Cfg(d, B, T, dtype, kv_pages=pages), kp, vp, table)
    assert torch.equal(got.k_logical(), ref.k_logical())
    assert torch.equal(got.v_logical(), ref.v_logical())
