"""Full-size decode-step workloads through the fused step (the launch
configuration the benchmark times), checked against the fp64 oracle on
sampled sequences and layers, and by properties that hold at any size on all
sequences."""
import numpy as np
import pytest
import torch

import oracle
import paper_2512_00722_amd as spec
from tests.gpu_helpers import SCORE_ABS, SCORE_REL, TOL_ATTN, announce, f64, need_gpu
from workloads import WORKLOADS, elastic_sequence, generate

pytestmark = pytest.mark.gpu

FIXED = ["b1_l4096_k512_1layer", "b8_l32768_k2048_32layers", "b32_l16384_k1024_hr16",
         "b1_l131072_k4096_g8"]


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def _sample_layers(n):
    return sorted({0, n // 2, n - 1})


@pytest.mark.parametrize("name", FIXED)
def test_full_size_step(dev, name):
    w = WORKLOADS[name]
    announce(f"full-size step {name}")
    x = generate(w, seed=0, device=dev)
    r = spec.step(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"], x["V"], k_max=w.k,
                  with_scores=True, with_lse=True)
    torch.cuda.synchronize()
    idx = r["idx"].cpu().numpy()
    cnt = r["counts"].cpu().numpy()
    sc = r["scores"].cpu().numpy().astype(np.float64)
    lens = x["seq_lens"].cpu().numpy()
    ks = x["ks"].cpu().numpy()

    # properties on every sequence
    for b in range(w.B):
        L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
        assert cnt[b] == kb
        sel = idx[b, :kb]
        assert np.all(np.diff(sel) > 0) and sel[0] >= 0 and sel[-1] < L
        assert np.all(idx[b, kb:] == -1)
        assert abs(sc[b, :L].sum() - w.H_r) < 1e-3 * w.H_r       # softmax rows sum to 1
        assert sel.tolist() == oracle.topk_indices(sc[b, :L], kb).tolist()  # exact on fp32 keys
    assert np.all(np.isfinite(r["out"].cpu().numpy()))

    # element-wise parity on sampled sequences and layers
    for b in sorted({0, w.B - 1}):
        L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
        s64 = oracle.retrieval_scores(f64(x["q_r"][b]), f64(x["K_r"][b, :L]), L)
        err = np.abs(sc[b, :L] - s64)
        assert np.all(err <= SCORE_ABS + SCORE_REL * s64), err.max()
        ok, info = oracle.accept_index_set(s64, kb, idx[b, :kb])
        assert ok, info
        print(f"b={b}: tie-band population {info['band_pop']}, set difference {info['sym_diff']}")
        heavy = x["heavy"][b]
        if len(heavy):
            recall = np.isin(heavy, idx[b, :kb]).mean()
            print(f"b={b}: planted-token recall {recall:.4f}")
            assert recall >= 0.99
        sel_t = torch.as_tensor(idx[b, :kb], device=dev, dtype=torch.long)
        for layer in _sample_layers(w.n_layers):
            Ks = f64(x["K"][layer, b, sel_t])
            Vs = f64(x["V"][layer, b, sel_t])
            want, wl = oracle.sparse_gqa_attention(f64(x["q"][layer, b]), Ks, Vs, np.arange(kb))
            got = r["out"][layer, b].cpu().numpy()
            assert np.abs(got - want).max() <= TOL_ATTN, (layer, np.abs(got - want).max())
            assert np.abs(r["lse"][layer, b].cpu().numpy() - wl).max() <= TOL_ATTN
    del x, r
    torch.cuda.empty_cache()


def test_full_size_elastic_sequence(dev):
    """The ragged 64-sequence workload over its 16 appended-token steps with
    elastic loading.  Every sequence, every step: the slot buffer holds
    exactly the selected set, and the rows loaded equal |S_now - S_last|.
    Sampled sequences: scores vs fp64, index-set acceptance, the slot->token
    map equals the oracle's elastic update of the previous map, held K/V rows
    are bit-exact copies, and attention matches the oracle on sampled layers."""
    w = WORKLOADS["b64_ragged_l2k_16k_elastic"]
    announce(f"full-size elastic sequence {w.name}")
    x = generate(w, seed=0, device=dev)
    e = elastic_sequence(w, x, seed=0, device=dev)
    st = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
    ks = x["ks"].cpu().numpy()
    sample = sorted({0, w.B // 2, w.B - 1})
    slot_ref = {b: np.full(w.k, -1, dtype=np.int64) for b in sample}
    prev = [np.zeros(0, dtype=np.int64) for _ in range(w.B)]
    overlap = []
    for s in range(w.steps):
        lens_t = e["seq_lens"][s]
        r = spec.step(q_r=e["q_r"][s], K_r=x["K_r"], seq_lens=lens_t, ks=x["ks"], q=e["q"][s],
                      K=x["K"], V=x["V"], k_max=w.k, elastic=st, with_scores=True, with_lse=True)
        torch.cuda.synchronize()
        lens = lens_t.cpu().numpy()
        idx = r["idx"].cpu().numpy()
        cnt = r["counts"].cpu().numpy()
        sc = r["scores"].cpu().numpy().astype(np.float64)
        slots = st.slot_tok.cpu().numpy()
        nch = st.n_changed.cpu().numpy()
        for b in range(w.B):
            L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
            sel = idx[b, :kb].astype(np.int64)
            assert cnt[b] == kb
            assert sel.tolist() == oracle.topk_indices(sc[b, :L], kb).tolist(), (s, b)
            assert sorted(slots[b, :kb].tolist()) == sel.tolist(), (s, b)
            assert np.all(slots[b, kb:] == -1)
            assert nch[b] == len(np.setdiff1d(sel, prev[b])), (s, b)
            if s > 0:
                overlap.append(len(np.intersect1d(sel, prev[b])) / kb)
            prev[b] = sel
        for b in sample:
            L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
            s64 = oracle.retrieval_scores(f64(e["q_r"][s, b]), f64(x["K_r"][b, :L]), L)
            err = np.abs(sc[b, :L] - s64)
            assert np.all(err <= SCORE_ABS + SCORE_REL * s64), (s, b, err.max())
            ok, info = oracle.accept_index_set(s64, kb, idx[b, :kb])
            assert ok, (s, b, info)
            slot_ref[b], loads = oracle.elastic_update(slot_ref[b], idx[b, :kb])
            assert slots[b].tolist() == slot_ref[b].tolist(), (s, b)
            assert len(loads) == nch[b]
            held = torch.as_tensor(np.nonzero(slot_ref[b] >= 0)[0], device=dev)
            toks = torch.as_tensor(slot_ref[b][slot_ref[b] >= 0], device=dev)
            for layer in (0, w.n_layers - 1):
                assert torch.equal(st.kbuf[layer, b, held].view(torch.int16),
                                   x["K"][layer, b, toks].view(torch.int16)), (s, b, layer)
                assert torch.equal(st.vbuf[layer, b, held].view(torch.int16),
                                   x["V"][layer, b, toks].view(torch.int16)), (s, b, layer)
            if s in (0, w.steps - 1):
                sel_t = torch.as_tensor(idx[b, :kb], device=dev, dtype=torch.long)
                for layer in _sample_layers(w.n_layers):
                    Ks = f64(x["K"][layer, b, sel_t])
                    Vs = f64(x["V"][layer, b, sel_t])
                    want, wl = oracle.sparse_gqa_attention(f64(e["q"][s, layer, b]), Ks, Vs,
                                                           np.arange(kb))
                    got = r["out"][layer, b].cpu().numpy()
                    assert np.abs(got - want).max() <= TOL_ATTN, (s, b, layer)
                    assert np.abs(r["lse"][layer, b].cpu().numpy() - wl).max() <= TOL_ATTN
    print(f"adjacent-step overlap: min {min(overlap):.3f} mean {np.mean(overlap):.3f}")
    assert np.mean(overlap) > 0.7
    del x, e, st, r
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["b8_l32768_k2048_32layers", "b32_l16384_k1024_hr16"])
def test_full_size_step_head_level(dev, name):
    """One token set per KV head at full size: every row's selection is the
    exact top-k of its fp32 scores; sampled sequences match the fp64 oracle
    (scores, accepted sets, attention over each head's own set)."""
    w = WORKLOADS[name]
    announce(f"full-size head-level step {name}")
    x = generate(w, seed=0, device=dev)
    r = spec.step(x["q_r"], x["K_r"], x["seq_lens"], x["ks"], x["q"], x["K"], x["V"], k_max=w.k,
                  with_scores=True, with_lse=True, head_level=True)
    torch.cuda.synchronize()
    idx = r["idx"].cpu().numpy()
    cnt = r["counts"].cpu().numpy()
    sc = r["scores"].cpu().numpy().astype(np.float64)
    lens = x["seq_lens"].cpu().numpy()
    ks = x["ks"].cpu().numpy()
    for b in range(w.B):
        L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
        assert cnt[b] == kb
        for h in range(w.H_kv):
            assert idx[b, h, :kb].tolist() == oracle.topk_indices(sc[b, h, :L], kb).tolist()
            assert np.all(idx[b, h, kb:] == -1)
    for b in sorted({0, w.B - 1}):
        L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
        s64 = oracle.head_level_scores(f64(x["q_r"][b]), f64(x["K_r"][b, :L]), L, w.H_kv)
        for h in range(w.H_kv):
            err = np.abs(sc[b, h, :L] - s64[h])
            assert np.all(err <= SCORE_ABS + SCORE_REL * s64[h]), (b, h, err.max())
            ok, info = oracle.accept_index_set(s64[h], kb, idx[b, h, :kb])
            assert ok, (b, h, info)
        rows = sorted(set(np.concatenate([idx[b, h, :kb] for h in range(w.H_kv)]).tolist()))
        rows_t = torch.as_tensor(rows, device=dev, dtype=torch.long)
        pos = {t: i for i, t in enumerate(rows)}
        sets = [np.array([pos[t] for t in idx[b, h, :kb]]) for h in range(w.H_kv)]
        for layer in _sample_layers(w.n_layers):
            Ks = f64(x["K"][layer, b, rows_t])      # only the rows some head selected
            Vs = f64(x["V"][layer, b, rows_t])
            want, wl = oracle.sparse_gqa_attention_sets(f64(x["q"][layer, b]), Ks, Vs, sets)
            got = r["out"][layer, b].cpu().numpy()
            assert np.abs(got - want).max() <= TOL_ATTN, (layer, np.abs(got - want).max())
            assert np.abs(r["lse"][layer, b].cpu().numpy() - wl).max() <= TOL_ATTN
    del x, r
    torch.cuda.empty_cache()
