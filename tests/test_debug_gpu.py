"""SPEC_DEBUG=1: the entry points check the device-resident lengths and
indices on the host before launching (values the kernels would clamp are
rejected with nothing enqueued) and synchronise after the launch."""
import numpy as np
import pytest
import torch

import paper_2512_00722_amd as spec
from tests.gpu_helpers import announce, need_gpu
from workloads import generate, small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def test_debug_mode_rejects_and_matches(dev, monkeypatch):
    announce("SPEC_DEBUG checks")
    w = small_workload(B=2, L=500, H_r=4, d_r=64, n_layers=2, H_q=8, H_kv=2, k=64)
    x = generate(w, seed=1, device=dev)
    ref = spec.step(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"], x["V"], k_max=w.k)
    torch.cuda.synchronize()
    monkeypatch.setenv("SPEC_DEBUG", "1")
    # valid inputs: same results as without the checks
    got = spec.step(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"], x["V"], k_max=w.k)
    assert torch.equal(got["idx"], ref["idx"]) and torch.equal(got["out"], ref["out"])
    # a length past L_max, a negative budget
    bad_len = torch.tensor([500, 501], dtype=torch.int32, device=dev)
    with pytest.raises(spec.SpecError) as e:
        spec.score(x["q_r"], x["K_r"], bad_len)
    assert e.value.status == 1
    with pytest.raises(spec.SpecError) as e:
        spec.topk(torch.zeros((2, 500), device=dev), x["seq_lens"],
                  torch.tensor([3, -1], dtype=torch.int32, device=dev), 8)
    assert e.value.status == 1
    # an index outside the cache, a count above k_max
    idx = ref["idx"].clone()
    idx[1, 0] = 500
    with pytest.raises(spec.SpecError) as e:
        spec.gather(x["K"], x["V"], idx, ref["counts"])
    assert e.value.status == 1
    with pytest.raises(spec.SpecError) as e:
        spec.sparse_decode_attn(x["q"], x["K"], x["V"],
                                torch.tensor([64, 65], dtype=torch.int32, device=dev),
                                idx=ref["idx"])
    assert e.value.status == 1
    # indices past counts[b] are not looked at
    idx2 = ref["idx"].clone()
    idx2[0, 63] = 10 ** 6
    cnt = torch.tensor([63, 64], dtype=torch.int32, device=dev)
    spec.gather(x["K"], x["V"], idx2, cnt)
    torch.cuda.synchronize()
    monkeypatch.delenv("SPEC_DEBUG")


def test_debug_mode_offload(dev, monkeypatch):
    """SPEC_DEBUG=1 on the host-offload entry points: a count above k_max is
    rejected before anything is enqueued; valid calls match the plain ones."""
    announce("SPEC_DEBUG offload")
    w = small_workload(B=2, L=600, H_r=4, d_r=64, n_layers=2, H_q=8, H_kv=2, k=64)
    x = generate(w, seed=2, device=dev)
    host_k = torch.empty(x["K"][1:].shape, dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty_like(host_k, pin_memory=True)
    host_k.copy_(x["K"][1:])
    host_v.copy_(x["V"][1:])
    st = spec.ElasticState(1, w.B, w.k, w.H_kv, w.d, dev)
    ref = spec.step_offload(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"][:1],
                            x["V"][:1], host_k, host_v, w.k, st)
    torch.cuda.synchronize()
    ref_out = ref["out"].clone()
    monkeypatch.setenv("SPEC_DEBUG", "1")
    st.reset()
    got = spec.step_offload(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"][:1],
                            x["V"][:1], host_k, host_v, w.k, st, copy_stream=torch.cuda.Stream())
    assert torch.equal(got["out"], ref_out)
    bad = torch.tensor([64, 65], dtype=torch.int32, device=dev)
    before = st.slot_tok.clone()
    with pytest.raises(spec.SpecError) as e:
        spec.offload_load(ref["idx"], bad, host_k, host_v, st)
    assert e.value.status == 1
    torch.cuda.synchronize()
    assert torch.equal(st.slot_tok, before)          # nothing was enqueued
    monkeypatch.delenv("SPEC_DEBUG")


def test_debug_mode_elastic_attention(dev, monkeypatch):
    """SPEC_DEBUG=1 on the elastic attention: a count above k_max or a slot
    source outside [-1, L_cap) is rejected with nothing enqueued (the output
    keeps its sentinel); valid state gives the same bits as without the
    checks."""
    announce("SPEC_DEBUG elastic attention")
    w = small_workload(B=2, L=500, H_r=4, d_r=64, n_layers=2, H_q=8, H_kv=2, k=64)
    x = generate(w, seed=2, device=dev)
    st = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
    r = spec.step(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"], x["V"], k_max=w.k,
                  elastic=st)
    ref, _ = spec.sparse_decode_attn_elastic(x["q"], x["K"], x["V"], st, r["counts"])
    torch.cuda.synchronize()
    monkeypatch.setenv("SPEC_DEBUG", "1")
    got, _ = spec.sparse_decode_attn_elastic(x["q"], x["K"], x["V"], st, r["counts"])
    assert torch.equal(got, ref)
    out = torch.full_like(ref, 7.0)
    with pytest.raises(spec.SpecError) as e:
        spec.sparse_decode_attn_elastic(x["q"], x["K"], x["V"], st,
                                        torch.tensor([64, 65], dtype=torch.int32, device=dev),
                                        out=out)
    assert e.value.status == 1
    for bad in (500, -2):
        saved = st.slot_src.clone()
        st.slot_src[1, 3] = bad
        with pytest.raises(spec.SpecError) as e:
            spec.sparse_decode_attn_elastic(x["q"], x["K"], x["V"], st, r["counts"], out=out)
        assert e.value.status == 1
        st.slot_src.copy_(saved)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
    monkeypatch.delenv("SPEC_DEBUG")
