"""The allocation-free decode step (spec_step_noalloc) against spec_step with
a caller workspace: two calls in a row, the second on a smaller input, must
give the same selections bit for bit and the same outputs within the
attention bound (the kernels are the same, so the outputs are in fact
identical), with and without elastic loading.  Each call goes through the C
ABI (ctypes) on inputs generated on the GPU."""
import numpy as np
import pytest
import torch

import paper_2512_00722_amd as spec
from tests.gpu_helpers import TOL_ATTN, announce, need_gpu
from workloads import generate, small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def _outputs(w, dev):
    return {"idx": torch.full((w.B, w.k), -7, dtype=torch.int32, device=dev),
            "counts": torch.full((w.B,), -7, dtype=torch.int32, device=dev),
            "out": torch.full((w.n_layers, w.B, w.H_q, w.d), float("nan"), device=dev),
            "lse": torch.full((w.n_layers, w.B, w.H_q), float("nan"), device=dev),
            "scores": torch.full((w.B, w.L_cap), float("nan"), device=dev)}


def _same(a, b, what):
    assert torch.equal(a["idx"], b["idx"]), what
    assert torch.equal(a["counts"], b["counts"]), what
    assert torch.isfinite(a["out"]).all() and torch.isfinite(a["scores"][:, 0]).all(), what
    err = (a["out"] - b["out"]).abs().max().item()
    assert err <= TOL_ATTN, (what, err)
    assert torch.equal(a["out"], b["out"]) and torch.equal(a["lse"], b["lse"]), what
    assert torch.equal(a["scores"], b["scores"]), what


# a larger input, then a smaller one (fewer sequences, shorter contexts)
SIZES = [dict(B=6, L=9000, H_r=8, d_r=64, n_layers=3, H_q=32, H_kv=8, k=1500, ragged_min=2000,
              heavy_frac=0.02),
         dict(B=2, L=3000, H_r=16, d_r=64, n_layers=2, H_q=32, H_kv=8, k=400, heavy_frac=0.05)]


@pytest.mark.parametrize("elastic", [False, True], ids=["indexed", "elastic"])
def test_step_noalloc_matches_step(dev, elastic):
    for i, kw in enumerate(SIZES):
        w = small_workload(**kw)
        announce(f"no-alloc step call {i} {kw} elastic={elastic}")
        x = generate(w, seed=11 + i, device=dev)
        args = (x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"], x["V"])
        st_a = st_b = None
        if elastic:
            st_a = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
            st_b = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
        a = spec.step_noalloc(*args, k_max=w.k, elastic=st_a, outputs=_outputs(w, dev))
        b = spec.step(*args, k_max=w.k, elastic=st_b, outputs=_outputs(w, dev))
        torch.cuda.synchronize()
        _same(a, b, f"call {i}")
        if elastic:
            assert torch.equal(st_a.slot_tok, st_b.slot_tok)
            assert torch.equal(st_a.n_changed, st_b.n_changed)
        ks = np.minimum(x["ks"].cpu().numpy(), x["seq_lens"].cpu().numpy())
        assert a["counts"].cpu().numpy().tolist() == ks.tolist()
