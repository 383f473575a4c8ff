"""Retrieval-head front end on the GPU against the fp64 oracle: the new
token's embedding row, the Q/K projection, the rotary embedding with YaRN
scaling, and the append of the new key into K_r (Sec. 4.3).

Tolerance (bf16 inputs, fp32 accumulation, bf16 output):
    |got - want| <= 2^-8 |want| + 2^-16 * m * (S_i + S_i')
where 2^-8 covers the output rounding (2^-9) twice over, S_i = sum_k |W[i,k]|
|x_k| bounds the fp32 accumulation error of feature i, and i' is its rotary
partner (the rotation mixes the two).  The accumulation runs about 30
additions deep per output (16 MFMA steps per wave, the eight-wave sum, the
32-term MFMA dot), so its error stays below 2^-19 S: the margin is 8x.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2512_00722_amd as spec
from tests.gpu_helpers import SCORE_ABS, SCORE_REL, announce, f64, need_gpu
from workloads import WORKLOADS, frontend_inputs, generate, small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def _expected(fe, b, H_r, d_r, theta, m, vocab):
    """Oracle q_r, k_r of sequence b and the accumulation bound per output."""
    tok = min(max(int(fe["tokens"][b]), 0), vocab - 1)     # ids are clamped into the table
    pos = int(fe["pos"][b])
    row = f64(fe["emb"][tok:tok + 1])
    wq, wk = f64(fe["w_q"]), f64(fe["w_k"])
    q, k = oracle.retrieval_qk(0, pos, row, wq, wk, H_r, theta, m)
    # magnitudes: the same projection on |x|, |W| at position 0 (no rotation)
    sq, sk = oracle.retrieval_qk(0, 0, np.abs(row), np.abs(wq), np.abs(wk), H_r,
                                 np.zeros_like(theta), m)
    bound = lambda s_: s_ + np.roll(s_, d_r // 2, axis=-1)
    return q, k, bound(sq), bound(sk)


def _check(got, want, bound, what):
    err = np.abs(got - want)
    lim = 2.0 ** -8 * np.abs(want) + 2.0 ** -16 * bound
    bad = err > lim
    assert not bad.any(), (what, int(bad.sum()), float(err.max()), float(lim.min()))


def _run_case(dev, B, H_r, d_r, hidden, vocab, L_cap, scale, seed, pos=None, tokens=None,
              alpha=0.0, beta=0.0, orig_ctx=2048, base=500000.0):
    w = small_workload(B=B, L=L_cap, H_r=H_r, d_r=d_r, hidden=hidden, vocab=vocab,
                       rope_base=base, orig_ctx=orig_ctx)
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, L_cap + 1, size=B)
    fe = frontend_inputs(w, lens, seed=seed, device=dev)
    if pos is not None:
        fe["pos"] = torch.as_tensor(pos, dtype=torch.int32, device=dev)
    if tokens is not None:
        fe["tokens"] = torch.as_tensor(tokens, dtype=torch.int32, device=dev)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    K_r = torch.randn((B, L_cap, H_r, d_r), generator=g, device=dev).to(torch.bfloat16)
    before = K_r.clone()
    q_r = spec.retrieval_qk(fe["tokens"], fe["pos"], fe["emb"], fe["w_q"], fe["w_k"], K_r,
                            rope_base=base, yarn_scale=scale, yarn_orig_ctx=orig_ctx,
                            yarn_alpha=alpha, yarn_beta=beta)
    torch.cuda.synchronize()
    theta, m = oracle.yarn_frequencies(d_r, base, scale, orig_ctx,
                                       alpha if alpha or beta else 1.0,
                                       beta if alpha or beta else 32.0)
    pos_h = fe["pos"].cpu().numpy()
    expect_cache = before.clone()
    for b in range(B):
        q, k, bq, bk = _expected(fe, b, H_r, d_r, theta, m, vocab)
        _check(f64(q_r[b]), q, bq, f"q_r b={b}")
        p = int(pos_h[b])
        if 0 <= p < L_cap:
            _check(f64(K_r[b, p]), k, bk, f"K_r b={b} pos={p}")
            expect_cache[b, p] = K_r[b, p]
    # nothing but the appended rows changed
    assert torch.equal(K_r.view(torch.int16), expect_cache.view(torch.int16))
    return q_r, K_r


# (B, H_r, d_r, hidden, vocab, L_cap, yarn scale): one 16-token tile, two,
# four with a ragged second block, fewer hidden steps than waves, a single
# hidden step, d_r = 128, no scaling
CASES = [
    (1, 8, 64, 4096, 1000, 64, 2.0),
    (8, 8, 64, 4096, 3000, 256, 16.0),
    (20, 4, 128, 1024, 500, 64, 1.0),
    (70, 2, 64, 640, 300, 32, 64.0),
    (3, 16, 128, 128, 100, 16, 8.0),
    (16, 16, 64, 2048, 4096, 40, 4.0),
]


@pytest.mark.parametrize("case", CASES, ids=[f"B{c[0]}_hr{c[1]}_dr{c[2]}_h{c[3]}_s{c[6]:g}"
                                             for c in CASES])
def test_retrieval_qk_cases(dev, case):
    B, H_r, d_r, hidden, vocab, L_cap, scale = case
    announce(f"retrieval_qk {case}")
    _run_case(dev, B, H_r, d_r, hidden, vocab, L_cap, scale, seed=11 + CASES.index(case))


def test_retrieval_qk_large_positions(dev):
    """Angles at 128K positions (fp64 angle formation) with a 64x extension."""
    announce("retrieval_qk large positions")
    L_cap = 131072
    pos = [131071, 65537, 0, 99999]
    _run_case(dev, 4, 8, 128, 1024, 256, L_cap, 64.0, seed=5, pos=pos)


def test_retrieval_qk_custom_ramp_and_base(dev):
    announce("retrieval_qk custom YaRN ramp and base")
    _run_case(dev, 5, 4, 64, 512, 64, 48, 8.0, seed=6, alpha=2.0, beta=16.0, base=10000.0,
              orig_ctx=4096)


def test_retrieval_qk_edges(dev):
    """Out-of-range ids are clamped into the table; a position outside
    [0, L_cap) appends nothing (q_r is still rotated by it)."""
    announce("retrieval_qk edge ids and positions")
    tokens = [-5, 99, 103, 0, 50, 7]
    pos = [-1, 32, 31, 0, 1000, 5]
    _run_case(dev, 6, 2, 64, 256, 100, 32, 4.0, seed=7, pos=pos, tokens=tokens)


def test_retrieval_qk_repeat_is_deterministic(dev):
    announce("retrieval_qk determinism")
    a, Ka = _run_case(dev, 8, 8, 64, 1024, 128, 64, 16.0, seed=8)
    b, Kb = _run_case(dev, 8, 8, 64, 1024, 128, 64, 16.0, seed=8)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(Ka.view(torch.int16), Kb.view(torch.int16))


@pytest.mark.parametrize("name", ["b8_l32768_k2048_32layers", "b1_l131072_k4096_g8",
                                  "b64_ragged_l2k_16k_elastic"])
def test_retrieval_qk_full_size(dev, name):
    """The workloads' front end at full size (the whole 128256-row embedding
    table, hidden 4096 or 8192), every sequence against the oracle; then the
    step scores with the new key in the cache."""
    w = WORKLOADS[name]
    announce(f"retrieval_qk full size {name}")
    x = generate(w, seed=0, device=dev, with_kv=False)
    fe = frontend_inputs(w, x["seq_lens"], seed=0, device=dev)
    K_r = x["K_r"]
    before = K_r.clone()
    q_r = spec.retrieval_qk(fe["tokens"], fe["pos"], fe["emb"], fe["w_q"], fe["w_k"], K_r,
                            rope_base=w.rope_base, yarn_scale=w.yarn_scale,
                            yarn_orig_ctx=w.orig_ctx)
    torch.cuda.synchronize()
    theta, m = oracle.yarn_frequencies(w.d_r, w.rope_base, w.yarn_scale, w.orig_ctx)
    pos_h = fe["pos"].cpu().numpy()
    for b in range(w.B):
        q, k, bq, bk = _expected(fe, b, w.H_r, w.d_r, theta, m, w.vocab)
        _check(f64(q_r[b]), q, bq, f"q_r b={b}")
        _check(f64(K_r[b, int(pos_h[b])]), k, bk, f"K_r b={b}")
        before[b, int(pos_h[b])] = K_r[b, int(pos_h[b])]
    assert torch.equal(K_r.view(torch.int16), before.view(torch.int16))
    # the scores of the step see the appended key: with the new q_r the last
    # token's score matches the oracle's on the device's own q_r / K_r
    sc = spec.score(q_r, K_r, x["seq_lens"])
    torch.cuda.synchronize()
    for b in sorted({0, w.B - 1}):
        L = int(x["seq_lens"][b])
        s64 = oracle.retrieval_scores(f64(q_r[b]), f64(K_r[b, :L]), L)
        got = sc[b, :L].cpu().numpy().astype(np.float64)
        assert np.all(np.abs(got - s64) <= SCORE_ABS + SCORE_REL * s64)
    del x, fe, K_r, before
    torch.cuda.empty_cache()
