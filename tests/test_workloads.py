"""The seeded input generators (CPU): shapes, determinism, the planted
structure, and the appended-token sequence of the elastic workload."""
import dataclasses

import numpy as np
import torch

import oracle
from workloads import (WORKLOADS, algorithmic_bytes, elastic_sequence, frontend_bytes,
                       frontend_inputs, generate, small_workload)


def test_generate_is_seeded_and_shaped():
    w = small_workload(B=2, L=300, H_r=4, d_r=64, n_layers=2, H_q=8, H_kv=2, k=32,
                       heavy_frac=0.05, recent=16)
    a, b = generate(w, seed=3), generate(w, seed=3)
    for name in ("q_r", "K_r", "q", "K", "V", "seq_lens", "ks"):
        assert torch.equal(a[name], b[name]), name
    assert tuple(a["K_r"].shape) == (2, 300, 4, 64)
    assert tuple(a["K"].shape) == (2, 2, 300, 2, 128)
    assert a["K"].dtype == torch.bfloat16
    c = generate(w, seed=4)
    assert not torch.equal(a["K_r"], c["K_r"])
    for b_ in range(2):
        h = a["heavy"][b_]
        assert len(h) == round(0.05 * 300) and np.all(h < 300 - 16)


def test_ragged_lengths_and_budgets():
    w = WORKLOADS["b64_ragged_l2k_16k_elastic"]
    w = dataclasses.replace(w, B=16, n_layers=1)
    x = generate(w, seed=0, with_kv=False)
    lens = x["seq_lens"].numpy()
    assert np.all((lens >= 2048) & (lens <= 16384))
    assert x["ks"].tolist() == np.minimum(2048, lens // 4).tolist()
    assert w.L_cap == 16400


def test_elastic_sequence_appends_and_drifts():
    w = small_workload(B=3, L=600, k=64, ragged_min=300, k_frac_den=4, extra_cap=16, steps=16,
                       heavy_frac=0.02)
    x = generate(w, seed=0)
    e = elastic_sequence(w, x, seed=0)
    lens0 = x["seq_lens"].numpy()
    assert e["seq_lens"].numpy().tolist() == [(lens0 + s).tolist() for s in range(16)]
    assert torch.equal(e["q_r"][0], x["q_r"])
    # AR(1) with coefficient 0.95: adjacent queries stay close, distant ones drift
    qs = e["q_r"].float().reshape(16, -1)
    cos = torch.nn.functional.cosine_similarity(qs[:-1], qs[1:], dim=1)
    assert torch.all(cos > 0.9) and torch.all(cos < 0.99)
    assert torch.nn.functional.cosine_similarity(qs[0], qs[15], dim=0) < 0.8
    e2 = elastic_sequence(w, x, seed=0)
    assert torch.equal(e["q"], e2["q"]) and torch.equal(e["q_r"], e2["q_r"])
    # the oracle's selections of adjacent steps overlap heavily (the premise
    # of elastic loading), but not completely
    f = lambda t: t.float().numpy().astype(np.float64)
    ov = []
    for b in range(w.B):
        prev = None
        for s in range(16):
            L = int(e["seq_lens"][s, b])
            sel = oracle.topk_indices(oracle.retrieval_scores(f(e["q_r"][s, b]),
                                                              f(x["K_r"][b, :L]), L), 64)
            if prev is not None:
                ov.append(len(np.intersect1d(sel, prev)) / 64)
            prev = sel
    assert 0.5 < np.mean(ov) < 1.0


def test_algorithmic_bytes_formula():
    w = WORKLOADS["b8_l32768_k2048_32layers"]
    assert algorithmic_bytes(w, [32768] * 8, [2048] * 8) == 2_422_218_752
    w4 = WORKLOADS["b1_l131072_k4096_g8"]
    assert algorithmic_bytes(w4, [131072], [4096]) == 806_881_280
    w1 = WORKLOADS["b1_l4096_k512_1layer"]
    assert algorithmic_bytes(w1, [4096], [512]) == 6_317_056
    # elastic rows: a write of K and V per changed row and layer (the read is
    # among the selected rows)
    assert (algorithmic_bytes(w, [32768] * 8, [2048] * 8, delta_rows=10)
            - algorithmic_bytes(w, [32768] * 8, [2048] * 8)) == 10 * 8 * 128 * 2 * 2 * 32


def test_frontend_inputs_seeded_and_shaped():
    w = small_workload(B=4, H_r=2, d_r=64, hidden=256, vocab=97)
    lens = np.array([10, 1, 64, 33])
    a, b = frontend_inputs(w, lens, seed=2), frontend_inputs(w, lens, seed=2)
    for name in ("tokens", "pos", "emb", "w_q", "w_k"):
        assert torch.equal(a[name], b[name]), name
    assert a["pos"].tolist() == (lens - 1).tolist()
    assert a["tokens"].dtype == torch.int32 and 0 <= int(a["tokens"].min())
    assert int(a["tokens"].max()) < 97
    assert tuple(a["emb"].shape) == (97, 256) and tuple(a["w_q"].shape) == (128, 256)
    # projected vectors have about unit variance
    x = a["emb"].float()[a["tokens"].long()]
    assert 0.7 < float((x @ a["w_q"].float().T).std()) < 1.3
    assert not torch.equal(a["w_q"], a["w_k"])
    c = frontend_inputs(w, lens, seed=3)
    assert not torch.equal(a["emb"], c["emb"])


def test_frontend_scale_and_bytes():
    w = WORKLOADS["b8_l32768_k2048_32layers"]
    assert w.yarn_scale == 16.0 and WORKLOADS["b1_l131072_k4096_g8"].yarn_scale == 64.0
    assert WORKLOADS["b1_l4096_k512_1layer"].yarn_scale == 2.0
    # two 512 x 4096 bf16 matrices, 8 embedding rows, q_r and the new K_r row
    assert frontend_bytes(w) == 2 * 512 * 4096 * 2 + 8 * 4096 * 2 + 2 * 8 * 512 * 2
