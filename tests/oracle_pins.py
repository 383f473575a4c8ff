"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each pin takes an oracle namespace `o` (the real oracle, or a deliberately
broken copy in the mutation tests) and raises AssertionError when `o`
disagrees with a value fixed independently of it: a hand-derived worked
example, a closed form, an invariant, a brute-force enumeration, or an
independent library routine.
"""

from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _lnval(x):
    if isinstance(x, str):
        assert x.startswith("ln")
        return math.log(float(x[2:]))
    return float(x)


# --------------------------------------------------------------- retrieval

def pin_retrieval_worked_example(o):
    g = _load("retrieval_worked_example.json")
    H_r, d_r, L = g["H_r"], g["d_r"], g["L"]
    K_r = np.zeros((L, H_r, d_r))
    for t in range(L):
        for h in range(H_r):
            K_r[t, h, 0] = _lnval(g["K_r_dim0"][t][h])
            K_r[t, h, 1:] = g["K_r_other"]
    q_r = np.array(g["q_r"], dtype=np.float64)
    p = o.head_softmax(o.retrieval_logits(q_r, K_r, L))
    np.testing.assert_allclose(p, np.array(g["p"]), rtol=0, atol=1e-14)
    s = o.retrieval_scores(q_r, K_r, L)
    np.testing.assert_allclose(s, np.array(g["score"]), rtol=0, atol=1e-14)
    for k, want in g["topk"].items():
        got = o.topk_indices(s, int(k))
        assert got.tolist() == want, (k, got, want)


def pin_scores_sum_to_heads(o):
    """Each head's softmax sums to 1, so the head-summed scores sum to H_r."""
    rng = np.random.default_rng(11)
    for H_r, d_r, L in [(1, 64, 1), (2, 64, 7), (8, 64, 300), (16, 128, 257)]:
        q_r = rng.standard_normal((H_r, d_r))
        K_r = rng.standard_normal((L + 5, H_r, d_r)) * 3.0
        p = o.head_softmax(o.retrieval_logits(q_r, K_r, L))
        np.testing.assert_allclose(p.sum(axis=1), np.ones(H_r), atol=1e-12)
        s = o.retrieval_scores(q_r, K_r, L)
        assert s.shape == (L,)
        assert abs(s.sum() - H_r) < 1e-10 * max(1, H_r)


def pin_constant_keys_uniform(o):
    """Identical keys give equal logits, so every score is H_r / L."""
    rng = np.random.default_rng(12)
    H_r, d_r, L = 4, 64, 37
    q_r = rng.standard_normal((H_r, d_r))
    row = rng.standard_normal((1, H_r, d_r))
    K_r = np.repeat(row, L, axis=0)
    s = o.retrieval_scores(q_r, K_r, L)
    np.testing.assert_allclose(s, np.full(L, H_r / L), rtol=1e-12)


def pin_logits_bruteforce(o):
    """Logits against a naive triple loop with the 1/sqrt(d_r) scale."""
    rng = np.random.default_rng(13)
    H_r, d_r, L = 3, 64, 5
    q_r = rng.standard_normal((H_r, d_r))
    K_r = rng.standard_normal((L + 2, H_r, d_r))
    want = np.zeros((H_r, L))
    for h in range(H_r):
        for t in range(L):
            acc = 0.0
            for i in range(d_r):
                acc += q_r[h, i] * K_r[t, h, i]
            want[h, t] = acc / math.sqrt(d_r)
    np.testing.assert_allclose(o.retrieval_logits(q_r, K_r, L), want, rtol=1e-12, atol=1e-12)
    # softmax by its definition, one element at a time
    p = o.head_softmax(want)
    for h in range(H_r):
        z = sum(math.exp(want[h, t]) for t in range(L))
        for t in range(L):
            assert abs(p[h, t] - math.exp(want[h, t]) / z) < 1e-14


def pin_single_head_is_logit_order(o):
    """With H_r = 1 softmax is monotone, so top-k of scores = top-k of logits."""
    rng = np.random.default_rng(14)
    for L, k in [(50, 7), (200, 64), (33, 33)]:
        q_r = rng.standard_normal((1, 64))
        K_r = rng.standard_normal((L, 1, 64))
        s = o.retrieval_scores(q_r, K_r, L)
        lg = (K_r[:L, 0, :] @ q_r[0])
        want = np.sort(np.argsort(-lg, kind="stable")[:k])
        assert o.topk_indices(s, k).tolist() == want.tolist()


# --------------------------------------------------------------- top-k

def _valid_topk_set(score, S):
    """Pairwise definition: every chosen token beats every unchosen one,
    where a tie is won by the lower index."""
    inside = set(S)
    for i in inside:
        for j in range(len(score)):
            if j in inside:
                continue
            if not (score[i] > score[j] or (score[i] == score[j] and i < j)):
                return False
    return True


def pin_topk_bruteforce(o):
    """Enumerate every subset of tiny inputs: exactly one satisfies the
    pairwise definition, and it is the oracle's set."""
    rng = np.random.default_rng(15)
    for trial in range(60):
        L = int(rng.integers(1, 9))
        # few distinct values, so ties are frequent
        score = rng.integers(0, 4, size=L).astype(np.float64) / 4.0
        for k in range(0, L + 2):
            kb = min(k, L)
            valid = [S for S in itertools.combinations(range(L), kb)
                     if _valid_topk_set(score, S)]
            assert len(valid) == 1, (score, k, valid)
            got = o.topk_indices(score, k)
            assert got.tolist() == list(valid[0]), (score, k, got, valid)


def pin_topk_all_equal(o):
    for L, k in [(10, 3), (64, 64), (100, 1)]:
        assert o.topk_indices(np.full(L, 0.25), k).tolist() == list(range(k))


def pin_topk_permutations(o):
    """Every permutation of a small distinct-score row selects the same
    values; the chosen values are the k largest."""
    vals = np.array([0.9, 0.1, 0.5, 0.7, 0.3, 0.2])
    for perm in itertools.permutations(range(6)):
        s = vals[list(perm)]
        for k in (1, 3, 5):
            got = o.topk_indices(s, k)
            assert sorted(s[got].tolist()) == sorted(vals)[-k:]
            assert got.tolist() == sorted(got.tolist())


def pin_heavy_recovered(o):
    """Tokens whose retrieval keys are pushed along q_r (a strong plant)
    dominate the softmax and are always selected."""
    rng = np.random.default_rng(16)
    H_r, d_r, L, n_heavy = 4, 64, 400, 20
    q_r = rng.standard_normal((H_r, d_r))
    K_r = rng.standard_normal((L, H_r, d_r))
    heavy = np.sort(rng.choice(L, n_heavy, replace=False))
    K_r[heavy] += 2.0 * q_r  # logit shift 2|q_r|^2/sqrt(d_r), about 16
    s = o.retrieval_scores(q_r, K_r, L)
    got = o.topk_indices(s, n_heavy)
    assert got.tolist() == heavy.tolist()


# --------------------------------------------------------------- attention

def pin_attention_worked_example(o):
    g = _load("gqa_attention_worked_example.json")
    H_q, H_kv, d, L = g["H_q"], g["H_kv"], g["d"], g["L"]
    K = np.zeros((L, H_kv, d))
    for t in range(L):
        for kv in range(H_kv):
            K[t, kv, 0] = _lnval(g["K_dim0"][t][kv])
    V = np.array(g["V"], dtype=np.float64)
    q = np.array(g["q"], dtype=np.float64)
    out, lse = o.sparse_gqa_attention(q, K, V, np.array(g["idx"]))
    np.testing.assert_allclose(out, np.array(g["out"], dtype=np.float64), atol=1e-14)
    np.testing.assert_allclose(lse, [_lnval(x) for x in g["lse"]], atol=1e-14)


def _sdpa_dense(q, K, V, L, scale=None):
    """torch's scaled_dot_product_attention (fp64, CPU) as the textbook
    dense reference, with the KV heads repeated G times (repeat_kv)."""
    H_q, d = q.shape
    H_kv = K.shape[1]
    G = H_q // H_kv
    qt = torch.as_tensor(q, dtype=torch.float64).reshape(1, H_q, 1, d)
    kt = torch.as_tensor(K[:L], dtype=torch.float64).permute(1, 0, 2)
    vt = torch.as_tensor(V[:L], dtype=torch.float64).permute(1, 0, 2)
    kt = kt.repeat_interleave(G, dim=0).unsqueeze(0).contiguous()
    vt = vt.repeat_interleave(G, dim=0).unsqueeze(0).contiguous()
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o.reshape(H_q, d).numpy()


def pin_full_budget_is_dense(o):
    """With k = L every token is selected and sparse attention equals dense
    attention; checked against torch's SDPA (fp64, CPU)."""
    rng = np.random.default_rng(17)
    for H_q, H_kv, L in [(4, 1, 9), (8, 2, 33), (8, 8, 17), (16, 2, 64)]:
        d = 128
        q = rng.standard_normal((H_q, d))
        K = rng.standard_normal((L + 3, H_kv, d))
        V = rng.standard_normal((L + 3, H_kv, d))
        q_r = rng.standard_normal((2, 64))
        K_r = rng.standard_normal((L + 3, 2, 64))
        idx = o.topk_indices(o.retrieval_scores(q_r, K_r, L), L)
        assert idx.tolist() == list(range(L))
        out, _ = o.sparse_gqa_attention(q, K, V, idx)
        np.testing.assert_allclose(out, _sdpa_dense(q, K, V, L), rtol=1e-10, atol=1e-12)


def pin_dense_attention_matches_sdpa(o):
    """Dense decode attention over the first L rows of a longer cache equals
    torch's SDPA (fp64, CPU) on those rows, for the default and an explicit
    scale; lse equals torch's logsumexp of the scaled logits."""
    rng = np.random.default_rng(23)
    for H_q, H_kv, L, L_cap, scale in [(4, 1, 6, 9, None), (8, 2, 13, 20, 0.3),
                                        (6, 6, 1, 4, None), (16, 4, 31, 31, 0.05)]:
        d = 32
        q = rng.standard_normal((H_q, d))
        K = rng.standard_normal((L_cap, H_kv, d))
        V = rng.standard_normal((L_cap, H_kv, d))
        out, lse = o.dense_gqa_attention(q, K, V, L, scale)
        np.testing.assert_allclose(out, _sdpa_dense(q, K, V, L, scale), rtol=1e-10, atol=1e-12)
        sc = scale if scale is not None else 1.0 / math.sqrt(d)
        G = H_q // H_kv
        kt = torch.as_tensor(K[:L], dtype=torch.float64)
        for h in range(H_q):
            lg = (kt[:, h // G, :] @ torch.as_tensor(q[h], dtype=torch.float64)) * sc
            assert abs(lse[h] - float(torch.logsumexp(lg, 0))) < 1e-12


def _decode_step_case(rng):
    """A tiny batched, multi-layer, ragged decode step whose two scales
    differ from each other and from their defaults."""
    B, L_cap, n_layers, H_r, d_r, H_q, H_kv, d = 3, 14, 3, 2, 64, 4, 2, 16
    return dict(
        q_r=rng.standard_normal((B, H_r, d_r)), K_r=rng.standard_normal((B, L_cap, H_r, d_r)) * 2,
        seq_lens=np.array([5, 9, 12]), ks=np.array([3, 20, 7]),
        q=rng.standard_normal((n_layers, B, H_q, d)) * 2,
        K_layers=rng.standard_normal((n_layers, B, L_cap, H_kv, d)),
        V_layers=rng.standard_normal((n_layers, B, L_cap, H_kv, d)),
        scale_r=0.37, scale=0.21)


def pin_decode_step_composition(o):
    """The batched decode step against an independent composition in torch
    (fp64, CPU): per-head softmax of the retrieval logits at scale_r summed
    over heads; the k_b largest (ties to the lower index) by a plain sort;
    then, for every layer and sequence, SDPA at `scale` with a boolean mask
    that keeps only the selected tokens (KV heads repeated G times)."""
    c = _decode_step_case(np.random.default_rng(29))
    idxs, scores, out, lse = o.decode_step(c["q_r"], c["K_r"], c["seq_lens"], c["ks"], c["q"],
                                           c["K_layers"], c["V_layers"], c["scale_r"],
                                           c["scale"])
    n_layers, B, H_q, d = c["q"].shape
    H_kv = c["K_layers"].shape[3]
    G = H_q // H_kv
    for b in range(B):
        L = int(c["seq_lens"][b])
        kr = torch.as_tensor(c["K_r"][b, :L], dtype=torch.float64)      # [L, H_r, d_r]
        qr = torch.as_tensor(c["q_r"][b], dtype=torch.float64)          # [H_r, d_r]
        lg = torch.einsum("thi,hi->ht", kr, qr) * c["scale_r"]
        want_s = torch.softmax(lg, dim=1).sum(0).numpy()
        np.testing.assert_allclose(scores[b], want_s, rtol=1e-12, atol=1e-14)
        kb = min(int(c["ks"][b]), L)
        want_idx = sorted(sorted(range(L), key=lambda t: (-want_s[t], t))[:kb])
        assert idxs[b].tolist() == want_idx, (b, idxs[b], want_idx)
        mask = torch.zeros((1, 1, 1, L), dtype=torch.bool)
        mask[..., want_idx] = True
        for layer in range(n_layers):
            qt = torch.as_tensor(c["q"][layer, b], dtype=torch.float64).reshape(1, H_q, 1, d)
            kt = torch.as_tensor(c["K_layers"][layer, b, :L], dtype=torch.float64).permute(1, 0, 2)
            vt = torch.as_tensor(c["V_layers"][layer, b, :L], dtype=torch.float64).permute(1, 0, 2)
            kt = kt.repeat_interleave(G, dim=0).unsqueeze(0).contiguous()
            vt = vt.repeat_interleave(G, dim=0).unsqueeze(0).contiguous()
            want_o = torch.nn.functional.scaled_dot_product_attention(
                qt, kt, vt, attn_mask=mask, scale=c["scale"]).reshape(H_q, d).numpy()
            np.testing.assert_allclose(out[layer, b], want_o, rtol=1e-10, atol=1e-12)
            lg2 = (kt[0] @ qt[0].transpose(1, 2)).squeeze(-1) * c["scale"]   # [H_q, L]
            want_l = torch.logsumexp(lg2[:, want_idx], dim=1).numpy()
            np.testing.assert_allclose(lse[layer, b], want_l, rtol=0, atol=1e-12)


def pin_attention_special_cases(o):
    rng = np.random.default_rng(18)
    H_q, H_kv, d, L = 8, 2, 128, 20
    q = rng.standard_normal((H_q, d))
    K = rng.standard_normal((L, H_kv, d))
    V = rng.standard_normal((L, H_kv, d))
    # k = 1: the output is the one selected V row of the head's group
    out, lse = o.sparse_gqa_attention(q, K, V, np.array([7]))
    for h in range(H_q):
        np.testing.assert_array_equal(out[h], V[7, h // (H_q // H_kv)])
        assert abs(lse[h] - (q[h] @ K[7, h // 4]) / math.sqrt(d)) < 1e-12
    # identical keys: uniform weights, the mean of the selected V rows
    Kc = np.repeat(K[:1], L, axis=0)
    sel = np.array([1, 4, 5, 11, 19])
    out, _ = o.sparse_gqa_attention(q, Kc, V, sel)
    for h in range(H_q):
        np.testing.assert_allclose(out[h], V[sel, h // 4].mean(axis=0), atol=1e-13)
    # permutation invariance over the index order
    perm = sel[[3, 0, 4, 2, 1]]
    a, la = o.sparse_gqa_attention(q, K, V, sel)
    b, lb = o.sparse_gqa_attention(q, K, V, perm)
    np.testing.assert_allclose(a, b, atol=1e-13)
    np.testing.assert_allclose(la, lb, atol=1e-13)
    # empty selection
    e, le = o.sparse_gqa_attention(q, K, V, np.zeros((0,), dtype=np.int64))
    assert np.all(e == 0) and np.all(np.isneginf(le))


def pin_group_max_bruteforce(o):
    rng = np.random.default_rng(19)
    p = rng.random((8, 13))
    gm = o.group_max_scores(p, 2)
    for g in range(2):
        for t in range(13):
            assert gm[g, t] == max(p[h, t] for h in range(g * 4, g * 4 + 4))


def _sp_softmax(x):
    import scipy.special
    return scipy.special.softmax(x, axis=-1)


def _torch_logits(q_r, K_r, L):
    """q_r . K_r^T / sqrt(d_r) per head with torch in float64 (independent of the oracle)."""
    q = torch.as_tensor(q_r, dtype=torch.float64)          # [H, d]
    k = torch.as_tensor(K_r[:L], dtype=torch.float64)      # [L, H, d]
    return (torch.einsum("lhd,hd->hl", k, q) / math.sqrt(q.shape[1])).numpy()


def pin_head_level_one_head_per_set(o):
    # H_r = n_sets: each set's weights are one head's softmax (scipy)
    rng = np.random.default_rng(23)
    q_r = rng.standard_normal((4, 16))
    K_r = rng.standard_normal((30, 4, 16))
    got = o.head_level_scores(q_r, K_r, 25, 4)
    np.testing.assert_allclose(got, _sp_softmax(_torch_logits(q_r, K_r, 25)), rtol=1e-12,
                               atol=1e-15)


def pin_head_level_identical_heads(o):
    # two identical heads per set: the group maximum is that head's softmax
    rng = np.random.default_rng(29)
    q1 = rng.standard_normal((3, 8))
    K1 = rng.standard_normal((17, 3, 8))
    q_r = np.repeat(q1, 2, axis=0)                 # heads 2g, 2g+1 equal
    K_r = np.repeat(K1, 2, axis=1)
    got = o.head_level_scores(q_r, K_r, 17, 3)
    np.testing.assert_allclose(got, _sp_softmax(_torch_logits(q1, K1, 17)), rtol=1e-12,
                               atol=1e-15)


def pin_head_level_bounds(o):
    # a maximum of `per` distributions: at least each of them, at most 1, and
    # a row sum between 1 and `per`
    rng = np.random.default_rng(31)
    q_r = rng.standard_normal((8, 16))
    K_r = rng.standard_normal((40, 8, 16)) * 2
    got = o.head_level_scores(q_r, K_r, 40, 2)
    p = _sp_softmax(_torch_logits(q_r, K_r, 40))
    for g in range(2):
        assert np.all(got[g] >= p[4 * g:4 * g + 4].max(axis=0) - 1e-15)
        assert np.all(got[g] <= 1.0)
        assert 1.0 - 1e-12 <= got[g].sum() <= 4.0 + 1e-12
    assert o.head_level_scores(q_r, K_r, 0, 2).shape == (2, 0)


def pin_attention_sets_per_group_sdpa(o):
    # each group's heads against torch's SDPA over that group's own rows
    rng = np.random.default_rng(37)
    H_q, H_kv, d, L = 8, 2, 16, 30
    q = rng.standard_normal((H_q, d))
    K = rng.standard_normal((L, H_kv, d))
    V = rng.standard_normal((L, H_kv, d))
    sets = [np.array([1, 4, 9, 22]), np.array([0, 2, 3, 5, 28, 29])]
    out, lse = o.sparse_gqa_attention_sets(q, K, V, sets)
    G = H_q // H_kv
    for g in range(H_kv):
        Ks = torch.as_tensor(K[sets[g], g], dtype=torch.float64)
        Vs = torch.as_tensor(V[sets[g], g], dtype=torch.float64)
        qq = torch.as_tensor(q[g * G:(g + 1) * G], dtype=torch.float64)
        want = torch.nn.functional.scaled_dot_product_attention(qq[None], Ks[None], Vs[None])[0]
        np.testing.assert_allclose(out[g * G:(g + 1) * G], want.numpy(), rtol=1e-12, atol=1e-13)
        s = (qq @ Ks.T) / math.sqrt(d)
        np.testing.assert_allclose(lse[g * G:(g + 1) * G], torch.logsumexp(s, 1).numpy(),
                                   rtol=1e-12)
    # an empty set gives zero output and -inf lse for that group only
    out2, lse2 = o.sparse_gqa_attention_sets(q, K, V, [np.array([], dtype=np.int64), sets[1]])
    assert np.all(out2[:G] == 0) and np.all(np.isneginf(lse2[:G]))
    np.testing.assert_allclose(out2[G:], out[G:], rtol=0, atol=0)


# ------------------------------------------------- retrieval-head front end

def pin_yarn_worked_example(o):
    g = _load("yarn_worked_example.json")
    theta, m = o.yarn_frequencies(g["d_r"], g["base"], g["scale"], g["orig_ctx"])
    np.testing.assert_allclose(theta, g["theta"], rtol=1e-9)
    assert abs(m - g["m"]) < 1e-9
    got = o.rope_rotate(np.array(g["v"], dtype=np.float64), g["pos"], theta, m)
    np.testing.assert_allclose(got, g["rotated"], atol=1e-9)
    # no scaling: the plain rotary frequencies and no magnitude factor
    theta1, m1 = o.yarn_frequencies(8, 10000.0, 1.0, 2048)
    np.testing.assert_allclose(theta1, [1.0, 0.1, 0.01, 0.001], rtol=1e-12)
    assert m1 == 1.0


def pin_rope_is_complex_rotation(o):
    # pair (i, i + d/2) as the complex number x + iy, multiplied by e^{i pos theta_i}
    rng = np.random.default_rng(41)
    v = rng.standard_normal(16)
    theta = np.exp(-rng.random(8) * 5)
    for pos in (0, 1, 7, 100000):
        z = (v[:8] + 1j * v[8:]) * np.exp(1j * pos * theta)
        np.testing.assert_allclose(o.rope_rotate(v, pos, theta, 1.5),
                                   1.5 * np.concatenate([z.real, z.imag]), atol=1e-12)
    np.testing.assert_array_equal(o.rope_rotate(v, 0, theta), v)


def pin_rope_relative_position(o):
    # rotated q.k depends on the positions only through their difference, and
    # the rotation keeps the norm (times m)
    rng = np.random.default_rng(43)
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    theta, m = o.yarn_frequencies(64, 500000.0, 32.0, 2048)
    a = o.rope_rotate(q, 1000, theta, m) @ o.rope_rotate(k, 900, theta, m)
    b = o.rope_rotate(q, 5100, theta, m) @ o.rope_rotate(k, 5000, theta, m)
    assert abs(a - b) < 1e-9 * (1 + abs(a))
    assert abs(np.linalg.norm(o.rope_rotate(q, 777, theta, m)) - m * np.linalg.norm(q)) < 1e-12


def pin_retrieval_qk_projection(o):
    # embedding row -> torch linear layers (no bias) -> rotation as complex products
    rng = np.random.default_rng(47)
    V, hidden, H_r, d_r = 11, 32, 2, 8
    emb = rng.standard_normal((V, hidden))
    w_q = rng.standard_normal((H_r * d_r, hidden))
    w_k = rng.standard_normal((H_r * d_r, hidden))
    theta, m = o.yarn_frequencies(d_r, 10000.0, 4.0, 16)
    q_r, k_r = o.retrieval_qk(7, 20, emb, w_q, w_k, H_r, theta, m)
    x = torch.as_tensor(emb[7], dtype=torch.float64)
    for w, got in ((w_q, q_r), (w_k, k_r)):
        y = torch.nn.functional.linear(x, torch.as_tensor(w, dtype=torch.float64)).numpy()
        y = y.reshape(H_r, d_r)
        z = (y[:, :d_r // 2] + 1j * y[:, d_r // 2:]) * np.exp(1j * 20 * theta)
        np.testing.assert_allclose(got, m * np.concatenate([z.real, z.imag], axis=1),
                                   rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------- elastic

def pin_elastic_worked_example(o):
    g = _load("elastic_worked_example.json")
    new, loads = o.elastic_update(np.array(g["slot_tok"]), np.array(g["s_now"]))
    assert new.tolist() == g["new_slot_tok"]
    assert [list(x) for x in loads] == g["loads"]


def pin_elastic_identities(o):
    rng = np.random.default_rng(20)
    for trial in range(50):
        L = int(rng.integers(10, 200))
        k = int(rng.integers(1, L // 2 + 1))
        last = rng.choice(L, k, replace=False)
        now = np.sort(rng.choice(L, k, replace=False))
        slot = rng.permutation(last)
        new, loads = o.elastic_update(slot, now)
        d_in = set(now.tolist()) - set(last.tolist())
        d_out = set(last.tolist()) - set(now.tolist())
        assert len(d_in) == len(d_out) == len(loads)            # |S_now-S_last| = |S_last-S_now|
        assert sorted(new.tolist()) == now.tolist()              # slots hold S_now
        kept = [i for i, t in enumerate(slot.tolist()) if t in set(now.tolist())]
        for i in kept:                                           # survivors stay in place
            assert new[i] == slot[i]
        # from an empty state every token is loaded
        empty = np.full(k, -1)
        new2, loads2 = o.elastic_update(empty, now)
        assert sorted(new2.tolist()) == now.tolist() and len(loads2) == k
        # an unchanged selection loads nothing
        new3, loads3 = o.elastic_update(new, now)
        assert loads3 == [] and new3.tolist() == new.tolist()


# --------------------------------------------------------------- MLA (Sec. 4.3 "Support for MLA")

def _mla_case(rng, H=3, d_c=12, d_nope=5, d_rope=3, d_v=7, L=20):
    """Random MLA inputs with every dimension different, so that a
    transposed or swapped weight fails on shapes."""
    return dict(q_nope=rng.standard_normal((H, d_nope)), q_rope=rng.standard_normal((H, d_rope)),
                c=rng.standard_normal((L, d_c)), k_rope=rng.standard_normal((L, d_rope)),
                w_uk=rng.standard_normal((H, d_nope, d_c)) / math.sqrt(d_c),
                w_uv=rng.standard_normal((H, d_v, d_c)) / math.sqrt(d_c))


def pin_mla_worked_example(o):
    """One head, d_c = 2, d_nope = d_rope = d_v = 1, three cached tokens of
    which 0 and 2 are selected, by hand (W_UK = (1, 2), W_UV = (3, -1),
    query (1, 1), scale 1/sqrt(2)):
      token 0: c = (1, 0), k_rope = 0: key (1, 0), value 3, logit 1/sqrt(2);
      token 2: c = (1, 1), k_rope = 1: key (3, 1), value 2, logit 4/sqrt(2);
    the unselected token 1 (c = (0, 1), k_rope = 5) would change both."""
    c = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    kr = np.array([[0.0], [5.0], [1.0]])
    out, lse = o.mla_sparse_attention(np.array([[1.0]]), np.array([[1.0]]), c, kr,
                                      np.array([[[1.0, 2.0]]]), np.array([[[3.0, -1.0]]]),
                                      np.array([0, 2]))
    e0, e2 = math.exp(1.0 / math.sqrt(2.0)), math.exp(4.0 / math.sqrt(2.0))
    assert out.shape == (1, 1) and lse.shape == (1,)
    assert abs(out[0, 0] - (3.0 * e0 + 2.0 * e2) / (e0 + e2)) < 1e-13
    assert abs(lse[0] - math.log(e0 + e2)) < 1e-13


def pin_mla_identity_projection_is_mqa(o):
    """No rotary part and identity up-projections (d_c = d_nope = d_v): keys
    and values are the latents themselves, i.e. multi-query attention over c."""
    rng = np.random.default_rng(31)
    H, d, L = 4, 16, 40
    idx = np.sort(rng.choice(L, 11, replace=False))
    q, c = rng.standard_normal((H, d)), rng.standard_normal((L, d))
    eye = np.broadcast_to(np.eye(d), (H, d, d))
    out, lse = o.mla_sparse_attention(q, np.zeros((H, 0)), c, np.zeros((L, 0)), eye, eye, idx)
    want, wl = o.sparse_gqa_attention(q, c[:, None, :], c[:, None, :], idx)
    np.testing.assert_allclose(out, want, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, wl, atol=1e-12, rtol=0)


def pin_mla_dense_matches_sdpa(o):
    """Every token selected: equal to torch's scaled_dot_product_attention
    (fp64) on explicitly up-projected keys [W_UK c ; k_rope] and values W_UV c."""
    rng = np.random.default_rng(32)
    x = _mla_case(rng)
    L = x["c"].shape[0]
    out, lse = o.mla_sparse_attention(**x, idx=np.arange(L))
    t = {k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in x.items()}
    K = torch.cat([torch.einsum("lc,hnc->hln", t["c"], t["w_uk"]),
                   t["k_rope"].unsqueeze(0).expand(3, -1, -1)], dim=-1)      # [H, L, 8]
    V = torch.einsum("lc,hvc->hlv", t["c"], t["w_uv"])                     # [H, L, 7]
    Q = torch.cat([t["q_nope"], t["q_rope"]], dim=-1).unsqueeze(1)         # [H, 1, 8]
    want = torch.nn.functional.scaled_dot_product_attention(Q, K, V, scale=1.0 / math.sqrt(8))
    np.testing.assert_allclose(out, want[:, 0].numpy(), atol=1e-12, rtol=0)
    s = (Q @ K.transpose(1, 2))[:, 0] / math.sqrt(8)
    np.testing.assert_allclose(lse, torch.logsumexp(s, dim=-1).numpy(), atol=1e-12, rtol=0)


def pin_mla_single_token(o):
    """One selected token: the output is its value W_UV[h] c_j and the lse
    its logit."""
    rng = np.random.default_rng(33)
    x = _mla_case(rng)
    j = 13
    out, lse = o.mla_sparse_attention(**x, idx=np.array([j]))
    for h in range(3):
        np.testing.assert_allclose(out[h], x["w_uv"][h] @ x["c"][j], atol=1e-12, rtol=0)
        logit = (x["q_nope"][h] @ (x["w_uk"][h] @ x["c"][j]) + x["q_rope"][h] @ x["k_rope"][j])
        assert abs(lse[h] - logit / math.sqrt(8)) < 1e-12


def pin_mla_absorbed_form(o):
    """Absorbing W_UK into the query and applying W_UV after the weighted sum
    of the latents gives the same result:
      q~_h = W_UK[h]^T q_nope[h],  s_hj = (q~_h . c_j + q_rope[h] . k_rope_j) / sqrt(d_nope + d_rope),
      o_h = W_UV[h] sum_j softmax_j(s_h) c_j."""
    rng = np.random.default_rng(34)
    x = _mla_case(rng, L=30)
    idx = np.array([2, 3, 7, 19, 28])
    out, lse = o.mla_sparse_attention(**x, idx=idx)
    for h in range(3):
        qt = x["w_uk"][h].T @ x["q_nope"][h]                                  # [d_c]
        s = (x["c"][idx] @ qt + x["k_rope"][idx] @ x["q_rope"][h]) / math.sqrt(8)
        p = np.exp(s - s.max())
        lat = (p / p.sum()) @ x["c"][idx]                                    # [d_c]
        np.testing.assert_allclose(out[h], x["w_uv"][h] @ lat, atol=1e-12, rtol=0)
        assert abs(lse[h] - (s.max() + math.log(p.sum()))) < 1e-12


def pin_mla_unselected_rows_ignored(o):
    """Latents and rotary keys of unselected tokens do not matter; the empty
    selection gives 0 and -inf."""
    rng = np.random.default_rng(35)
    x = _mla_case(rng)
    idx = np.array([1, 4, 9, 15])
    out, lse = o.mla_sparse_attention(**x, idx=idx)
    y = dict(x)
    rest = np.setdiff1d(np.arange(20), idx)
    y["c"] = x["c"].copy()
    y["k_rope"] = x["k_rope"].copy()
    y["c"][rest] = 100.0
    y["k_rope"][rest] = -50.0
    out2, lse2 = o.mla_sparse_attention(**y, idx=idx)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)
    out3, lse3 = o.mla_sparse_attention(**x, idx=np.array([], dtype=np.int64))
    assert np.all(out3 == 0) and np.all(np.isneginf(lse3)) and out3.shape == (3, 7)


# --------------------------------------------------------------- helpers

def pin_bf16_decode(o):
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x7F80, 0x0001], dtype=np.uint16)
    got = o.bf16_to_f64(bits)
    assert got[0] == 1.0 and got[1] == -2.0 and got[2] == 1.0078125
    assert got[3] == 0.0 and got[4] == 0.0 and np.signbit(got[4])
    assert np.isposinf(got[5])
    assert got[6] == 2.0 ** -133
    # against torch's own bf16 -> float conversion
    x = torch.randn(1000, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    np.testing.assert_array_equal(o.bf16_to_f64(x.view(torch.int16).numpy().view(np.uint16)),
                                  x.double().numpy())


def pin_acceptance_checker(o):
    score = np.array([0.5, 0.1, 0.3, 0.3 + 5e-7, 0.9, 0.05])
    ok, _ = o.accept_index_set(score, 3, np.array([0, 3, 4]))
    assert ok
    ok, info = o.accept_index_set(score, 3, np.array([0, 2, 4]))   # tie-band swap
    assert ok and info["sym_diff"] == 2
    ok, _ = o.accept_index_set(score, 3, np.array([0, 1, 4]))      # below band
    assert not ok
    ok, _ = o.accept_index_set(score, 3, np.array([2, 3, 4]))      # misses 0.5
    assert not ok
    ok, _ = o.accept_index_set(score, 3, np.array([0, 4]))         # wrong size
    assert not ok
    ok, _ = o.accept_index_set(score, 3, np.array([0, 4, 4]))      # duplicate
    assert not ok


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
