"""The fused step captured in a HIP graph (through torch's graph capture on
the launch stream): several replays, with eager work and synchronisations
between them, each match the eager result bit for bit.  The library records
no memset nodes: every scratch clear is a kernel."""
import pytest
import torch

import paper_2512_00722_amd as spec
from tests.gpu_helpers import announce, need_gpu
from workloads import generate, small_workload

pytestmark = pytest.mark.gpu


def test_step_graph_replays_match_eager():
    dev = need_gpu()
    announce("graph replay of the fused step")
    w = small_workload(B=3, L=3000, H_r=8, d_r=64, n_layers=3, H_q=32, H_kv=8, k=512,
                       heavy_frac=0.02, ragged_min=1500)
    x = generate(w, seed=11, device=dev)
    args = dict(q_r=x["q_r"], K_r=x["K_r"], seq_lens=x["seq_lens"], ks=x["ks"], q=x["q"],
                K=x["K"], V=x["V"], k_max=w.k)
    dims = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_STEP), dtype=torch.uint8, device=dev)
    eager = spec.step(**args, with_scores=True, with_lse=True)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in eager.items() if v is not None}

    outputs = {}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        spec.step(**args, with_scores=True, with_lse=True, outputs=outputs, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        spec.step(**args, with_scores=True, with_lse=True, outputs=outputs, ws=ws)
    for rep in range(4):
        for v in outputs.values():
            if v is not None:
                v.fill_(7)                      # stale values must be overwritten
        spec.score(x["q_r"], x["K_r"], x["seq_lens"])   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(outputs[k], v), (rep, k)


def test_step_graph_ragged_batch_replays_match_eager():
    """A ragged batch large enough for the attention to deal its work by
    selection size (96 sequences x 6 layers, several units per wavefront):
    graph replays match the eager step bit for bit."""
    dev = need_gpu()
    announce("graph replay of a ragged 96-sequence step")
    w = small_workload(B=96, L=2048, H_r=8, d_r=64, n_layers=6, H_q=32, H_kv=8, k=256,
                       heavy_frac=0.02, ragged_min=300, k_frac_den=4)
    x = generate(w, seed=17, device=dev)
    assert len(set(x["ks"].clamp(max=w.k).tolist())) > 1   # unequal selections
    args = dict(q_r=x["q_r"], K_r=x["K_r"], seq_lens=x["seq_lens"], ks=x["ks"], q=x["q"],
                K=x["K"], V=x["V"], k_max=w.k)
    dims = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_STEP), dtype=torch.uint8, device=dev)
    eager = spec.step(**args, with_lse=True)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in eager.items() if v is not None}
    outputs = {}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        spec.step(**args, with_lse=True, outputs=outputs, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        spec.step(**args, with_lse=True, outputs=outputs, ws=ws)
    for rep in range(3):
        for v in outputs.values():
            if v is not None:
                v.fill_(7)
        spec.score(x["q_r"], x["K_r"], x["seq_lens"])   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(outputs[k], v), (rep, k)


def test_step_offload_graph_replays_match_eager():
    """The step with host-offloaded layers captured in a graph: the copy
    stream joins the capture through the caller's events (fork after the
    slot plan, one join per offloaded layer).  Each replay, from an empty
    slot state set eagerly, matches the eager step bit for bit."""
    dev = need_gpu()
    announce("graph replay of the offloaded step")
    w = small_workload(B=3, L=2500, H_r=8, d_r=64, n_layers=3, H_q=32, H_kv=8, k=300,
                       heavy_frac=0.02, ragged_min=1000)
    x = generate(w, seed=12, device=dev)
    n_dev = 1
    host_k = torch.empty(x["K"][n_dev:].shape, dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty_like(host_k, pin_memory=True)
    host_k.copy_(x["K"][n_dev:])
    host_v.copy_(x["V"][n_dev:])
    n_off = w.n_layers - n_dev
    args = (x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"][:n_dev], x["V"][:n_dev],
            host_k, host_v, w.k)
    copy = torch.cuda.Stream()
    events = spec.OffloadEvents(n_off, dev)
    st = spec.ElasticState(n_off, w.B, w.k, w.H_kv, w.d, dev)
    dims = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_OFFLOAD), dtype=torch.uint8, device=dev)
    eager = spec.step_offload(*args, st, copy_stream=copy, events=events, with_scores=True,
                              with_lse=True, ws=ws)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in eager.items() if isinstance(v, torch.Tensor)}
    ref_slots = st.slot_tok.clone()
    ref_nch = st.n_changed.clone()

    outputs = {}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st.reset()
        spec.step_offload(*args, st, copy_stream=copy, events=events, with_scores=True,
                          with_lse=True, ws=ws, outputs=outputs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        spec.step_offload(*args, st, copy_stream=copy, events=events, with_scores=True,
                          with_lse=True, ws=ws, outputs=outputs)
    for rep in range(4):
        for v in outputs.values():
            if isinstance(v, torch.Tensor):
                v.fill_(7)                      # stale values must be overwritten
        st.reset()                              # each replay is a full load
        st.kbuf.fill_(0)
        spec.score(x["q_r"], x["K_r"], x["seq_lens"])   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(outputs[k], v), (rep, k)
        assert torch.equal(st.slot_tok, ref_slots) and torch.equal(st.n_changed, ref_nch), rep


@pytest.mark.parametrize("path", ["auto", "fused"])
def test_step_elastic_graph_replays_match_eager(path, monkeypatch):
    """The elastic step captured in a graph (plan, copy of the sequences with
    small updates, attention that loads the rows of mostly-new ones): each
    replay from the same slot state matches the eager step bit for bit,
    outputs, slot maps and slot buffers."""
    dev = need_gpu()
    if path == "fused":
        monkeypatch.setenv("SPEC_ELASTIC_PATH", "fused")
    announce(f"graph replay of the elastic step, path {path}")
    w = small_workload(B=3, L=2500, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=300,
                       heavy_frac=0.02, ragged_min=1000)
    x = generate(w, seed=13, device=dev)
    args = dict(q_r=x["q_r"], K_r=x["K_r"], seq_lens=x["seq_lens"], ks=x["ks"], q=x["q"],
                K=x["K"], V=x["V"], k_max=w.k)
    dims = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_STEP), dtype=torch.uint8, device=dev)
    st = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
    # a state from smaller budgets (the same scores: a subset of the step's
    # selection): sequence 0 gets two thirds of its rows new (loaded by the
    # attention), sequence 1 ten rows and sequence 2 half (copied first)
    ks = x["ks"].cpu()
    ks_pre = torch.tensor([max(1, int(ks[0]) // 3), int(ks[1]) - 10, max(1, int(ks[2]) // 2)],
                          dtype=torch.int32, device=dev)
    spec.step(**{**args, "ks": ks_pre}, elastic=st, ws=ws)
    torch.cuda.synchronize()
    st0 = {k: getattr(st, k).clone() for k in ("slot_tok", "kbuf", "vbuf")}
    eager = spec.step(**args, elastic=st, with_lse=True, ws=ws)
    torch.cuda.synchronize()
    nch, cnt = st.n_changed.cpu(), eager["counts"].cpu()
    assert 2 * nch[0] > cnt[0] and 2 * nch[1] < cnt[1] and 2 * nch[2] <= cnt[2]  # a mix
    ref = {k: v.clone() for k, v in eager.items() if v is not None}
    ref_state = {k: getattr(st, k).clone() for k in ("slot_tok", "slot_src", "n_changed", "kbuf", "vbuf")}

    def restore():
        for k, v in st0.items():
            getattr(st, k).copy_(v)

    outputs = {}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        restore()
        spec.step(**args, elastic=st, with_lse=True, outputs=outputs, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        spec.step(**args, elastic=st, with_lse=True, outputs=outputs, ws=ws)
    for rep in range(3):
        for v in outputs.values():
            if v is not None:
                v.fill_(7)
        restore()
        spec.score(x["q_r"], x["K_r"], x["seq_lens"])   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(outputs[k], v), (rep, k)
        for k, v in ref_state.items():
            assert torch.equal(getattr(st, k), v), (rep, k)
