"""Concurrent calls: two fused steps with their own workspaces, enqueued on
two streams at once (default priority), give the same bits as the same
steps run one after the other.  The header promises reentrant calls that
share nothing but the inputs; this pins it, including the elastic step,
whose slot state belongs to its caller."""
import pytest
import torch

import paper_2512_00722_amd as spec
from tests.gpu_helpers import announce, need_gpu
from workloads import generate, small_workload

pytestmark = pytest.mark.gpu


def _step_fn(w, x, dev, elastic=False):
    dims = spec.Dims.make(B=w.B, L_cap=w.L_cap, L_max=w.L_cap, k_max=w.k, H_r=w.H_r, d_r=w.d_r,
                          n_layers=w.n_layers, H_q=w.H_q, H_kv=w.H_kv, d=w.d,
                          kr_stride_b=x["K_r"].stride(0), kv_stride_layer=x["K"].stride(0),
                          kv_stride_b=x["K"].stride(1))
    ws = torch.zeros(spec.workspace_size(dims, spec.OP_STEP), dtype=torch.uint8, device=dev)
    st = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev) if elastic else None
    outputs = {}

    def run():
        if st is not None:
            st.reset()
        spec.step(q_r=x["q_r"], K_r=x["K_r"], seq_lens=x["seq_lens"], ks=x["ks"], q=x["q"],
                  K=x["K"], V=x["V"], k_max=w.k, with_scores=True, with_lse=True,
                  elastic=st, outputs=outputs, ws=ws)
    return run, outputs, st


def test_concurrent_steps_match_sequential():
    dev = need_gpu()
    announce("two fused steps on two streams at once")
    wa = small_workload(B=4, L=20000, H_r=8, d_r=64, n_layers=4, H_q=32, H_kv=8, k=1024,
                        heavy_frac=0.02, ragged_min=9000)
    wb = small_workload(B=1, L=70000, H_r=8, d_r=128, n_layers=3, H_q=64, H_kv=8, k=2048,
                        heavy_frac=0.01)
    wc = small_workload(B=6, L=6000, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=700,
                        heavy_frac=0.02, ragged_min=2000)
    xa, xb, xc = (generate(w, seed=s, device=dev) for w, s in ((wa, 1), (wb, 2), (wc, 3)))
    runs = [_step_fn(wa, xa, dev), _step_fn(wb, xb, dev), _step_fn(wc, xc, dev, elastic=True)]
    # sequential reference
    refs = []
    for run, outputs, st in runs:
        run()
        torch.cuda.synchronize()
        ref = {k: v.clone() for k, v in outputs.items() if v is not None}
        if st is not None:
            ref["kbuf"], ref["slot_tok"] = st.kbuf.clone(), st.slot_tok.clone()
        refs.append(ref)
    streams = [torch.cuda.Stream() for _ in runs]
    main = torch.cuda.current_stream()
    for rep in range(3):
        for (run, outputs, st), s in zip(runs, streams):
            for v in outputs.values():
                if v is not None:
                    v.fill_(7)          # stale values must be overwritten
            s.wait_stream(main)
        for (run, outputs, st), s in zip(runs, streams):
            with torch.cuda.stream(s):
                run()
                run()                  # twice: the second reuses the workspace
        for s in streams:
            main.wait_stream(s)
        torch.cuda.synchronize()
        for i, ((run, outputs, st), ref) in enumerate(zip(runs, refs)):
            got = dict(outputs)
            if st is not None:
                got["kbuf"], got["slot_tok"] = st.kbuf, st.slot_tok
            for k, v in ref.items():
                assert torch.equal(got[k], v), (rep, i, k)
