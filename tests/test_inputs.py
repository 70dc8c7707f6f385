"""The seeded input generators: determinism, slicing invariance, structure."""

import numpy as np
import pytest

import spla_inputs as si


def test_slicing_does_not_change_values():
    w = si.custom("t", 2, 4, 2, 32, 16, 4, [9000, 5000], kind="block_offsets", code=5)
    K, V = si.gen_kv(w, 1, 1, 0, 5000)
    for a, b in [(0, 1), (4095, 4097), (100, 4999), (4096, 5000)]:
        k2, v2 = si.gen_kv(w, 1, 1, a, b)
        assert np.array_equal(k2, K[a:b]) and np.array_equal(v2, V[a:b])
    k3, _ = si.gen_kv(w, 1, 1, 0, 5000, threads=4)
    assert np.array_equal(k3, K)


def test_bf16_rounding_is_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5 - 2 ** -9, 3.0e38], np.float32)
    r = si.round_bf16(x)
    assert np.all(r.view(np.uint32) & 0xFFFF == 0)
    assert r[1] == 1.0                      # tie, to even
    assert r[2] == np.float32(1.0 + 4 * 2 ** -8)  # tie, to even (upwards)
    torch = pytest.importorskip("torch")
    y = torch.from_numpy(np.random.default_rng(0).standard_normal(10000).astype(np.float32))
    assert np.array_equal(si.round_bf16(y.numpy()), y.to(torch.bfloat16).float().numpy())


def test_workloads_shapes_and_dtypes():
    for i in ["1", "2", "3", "4", "5", "g5"]:
        w = si.config(i)
        assert w.n_q_heads % w.n_kv_heads == 0
        assert w.capacity % w.block_size == 0
        assert len(w.lengths) == w.batch and max(w.lengths) <= w.capacity
        q = si.gen_q(w, 0)
        assert q.shape == (w.n_q_heads, w.head_dim) and q.dtype == np.float32
        if w.dtype == "bf16":
            assert np.all(q.view(np.uint32) & 0xFFFF == 0)
    w4 = si.config(4)
    assert min(w4.lengths) >= 16384 and max(w4.lengths) <= 65536 - 512
    assert w4.prefill_length(0) == w4.lengths[0] - 1


def test_planted_blocks_avoid_forced_blocks():
    w = si.config(1)
    pb = si.planted_blocks(w, 0, 0)
    assert len(pb) == 2 and pb.min() >= 1 and pb.max() < 60
    w3 = si.config(3)
    for b in range(2):
        for h in range(2):
            pb = si.planted_blocks(w3, b, h)
            assert len(set(pb.tolist())) == 8 and pb.min() >= 1 and pb.max() < 2048 - 4


def test_planted_shift_present_in_config1():
    w = si.config(1)
    q = si.gen_q(w, 0)[0].astype(np.float64)
    K, _ = si.gen_kv(w, 0, 0, 0, 4096)
    proj = (K @ q) / np.linalg.norm(q)
    per_block = proj.reshape(64, 64).mean(axis=1)
    top = set(np.argsort(-per_block)[:2].tolist())
    assert top == set(si.planted_blocks(w, 0, 0).tolist())


def test_slab_zero_pads_past_lengths():
    w = si.custom("t", 3, 2, 1, 16, 8, 2, [10, 3, 0], capacity=16, code=6)
    K, V, n = si.gen_kv_slab(w, 0, 12)
    assert list(n) == [10, 3, 0]
    assert np.all(K[0, :, 10:] == 0) and np.all(K[1, :, 3:] == 0) and np.all(K[2] == 0)
    assert np.array_equal(K[0, 0, :10], si.gen_kv(w, 0, 0, 0, 10)[0])
