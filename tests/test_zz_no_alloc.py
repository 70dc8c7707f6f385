"""spla_decode_noalloc, the decode on the library's own device scratch,
against spla_decode with a caller workspace: the same kernels, so outputs
and selections must be bit-identical, on consecutive calls whose shapes
shrink (the scratch keeps the previous call's contents)."""

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


# consecutive calls, each smaller than the one before: the single-launch
# kernel at two shapes, then the separate launches (fp32)
CALLS = [
    dict(batch=4, n_q_heads=16, n_kv_heads=4, head_dim=128, block_size=64, top_k=16,
         lengths=[20000, 9000, 5000, 100], kind="block_offsets"),
    dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=64, top_k=8,
         lengths=[3000, 700], kind="iid"),
    dict(batch=1, n_q_heads=2, n_kv_heads=1, head_dim=64, block_size=32, top_k=6,
         lengths=[1000], dtype="f32", kind="drift"),
]


def test_noalloc_matches_the_workspace_decode(dev):
    for i, spec in enumerate(CALLS):
        w = si.custom(f"noalloc{i}", code=140 + i, **spec)
        H.log(f"no-alloc call {i}: {spec}")
        cfg = H.config_of(w)
        cache = spla.SplaCache(cfg, dev)
        H.fill_cache(w, cache, device=dev)
        q = H.to_dev(si.gen_q_batch(w), w, dev)
        gamma = torch.from_numpy(si.gen_gamma(w)).to(dev)
        ref_out, ref_sel = cache.decode(q, gamma)
        out = torch.full_like(q, float("nan"))
        sel = torch.full_like(ref_sel, -7)
        cache.decode_noalloc(q, gamma, out, sel)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16 if w.dtype == "bf16" else torch.int32),
                           ref_out.view(torch.int16 if w.dtype == "bf16" else torch.int32))
        assert torch.equal(sel, ref_sel)
        assert cache.device_errors() == 0
        # and against the oracle on one (sequence, KV head)
        H.check_kv_head(w, 0, 0, out.float().cpu().numpy()[0], sel.cpu().numpy()[0, 0],
                        si.gen_q_batch(w)[0], si.gen_gamma(w), H.params_of(w))
        # a second call on the same shape, without a selection output
        out2 = torch.zeros_like(q)
        cache.decode_noalloc(q, gamma, out2)
        torch.cuda.synchronize()
        assert torch.equal(out2, ref_out)
