"""HIP path vs the fp64 oracle, element by element, at sizes the oracle
finishes in seconds (several tiles plus ragged tails).  Calls go through the
C ABI via the thin Python binding."""
import numpy as np
import pytest
import torch

import oracle
import paper_2512_00722_amd as spec
from tests.gpu_helpers import SCORE_ABS, SCORE_REL, TOL_ATTN, announce, f64, need_gpu
from workloads import elastic_sequence, generate, small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def _rand_bf16(shape, gen, scale=1.0):
    return (torch.randn(shape, generator=gen) * scale).to(torch.bfloat16)


# ------------------------------------------------------------------ scoring

SCORE_CASES = [
    # B, L_cap, L_max, H_r, d_r, seq_lens
    (1, 130, 130, 1, 64, [130]),
    (2, 300, 300, 2, 64, [300, 1]),
    (3, 1000, 1000, 8, 64, [1000, 777, 129]),
    (2, 700, 640, 16, 64, [640, 513]),
    (2, 520, 520, 8, 128, [520, 200]),
    (1, 400, 400, 16, 128, [0]),
    (4, 2500, 2400, 8, 64, [2400, 2048, 2047, 2049]),
    (2, 900, 900, 3, 64, [900, 450]),
    (1, 600, 600, 5, 128, [600]),
    # more per-block softmax pairs per head than one pass of the merge holds
    (1, 70000, 70000, 16, 64, [70000]),
    # logits blocks of 128 tokens (one sequence, fewer than 256 blocks of 256)
    (1, 40000, 40000, 8, 64, [39999]),
    # blocks of 64 tokens, more pairs per head than one merge pass holds
    (1, 30000, 30000, 16, 64, [29999]),
]


@pytest.mark.parametrize("case", SCORE_CASES, ids=[str(c[:5]) for c in SCORE_CASES])
def test_score_parity(dev, case):
    B, L_cap, L_max, H_r, d_r, lens = case
    announce(f"score {case}")
    g = torch.Generator().manual_seed(1000 + B * L_cap + H_r)
    q_r = _rand_bf16((B, H_r, d_r), g)
    K_r = _rand_bf16((B, L_cap, H_r, d_r), g, 1.5)
    seq = torch.tensor(lens, dtype=torch.int32)
    got = spec.score(q_r.to(dev), K_r.to(dev), seq.to(dev), L_max=L_max)
    torch.cuda.synchronize()
    got = got.cpu().numpy().astype(np.float64)
    qn, Kn = f64(q_r), f64(K_r)
    for b in range(B):
        L = min(lens[b], L_max)
        want = oracle.retrieval_scores(qn[b], Kn[b], L)
        err = np.abs(got[b, :L] - want)
        assert np.all(err <= SCORE_ABS + SCORE_REL * want), (b, err.max())
        assert np.all(np.isneginf(got[b, L:]))
        if L:
            assert abs(got[b, :L].sum() - H_r) < 1e-4 * H_r


def test_score_strided_kr(dev):
    """K_r as a slice of a larger buffer (sequence stride > L_cap*H_r*d_r)."""
    announce("score strided")
    g = torch.Generator().manual_seed(7)
    big = _rand_bf16((3, 600, 8, 64), g)
    K_r = big[:, :500]
    q_r = _rand_bf16((3, 8, 64), g)
    seq = torch.tensor([500, 499, 300], dtype=torch.int32)
    got = spec.score(q_r.to(dev), big.to(dev)[:, :500], seq.to(dev)).cpu().numpy()
    for b in range(3):
        want = oracle.retrieval_scores(f64(q_r)[b], f64(K_r)[b], int(seq[b]))
        np.testing.assert_allclose(got[b, :int(seq[b])], want, rtol=SCORE_REL, atol=SCORE_ABS)


# ------------------------------------------------------------------ top-k

def _topk_rows(kind, B, L, g):
    if kind == "random":
        return torch.rand((B, L), generator=g)
    if kind == "ties":          # few distinct values: many exact ties
        return torch.randint(0, 5, (B, L), generator=g).float() / 4.0
    if kind == "equal":
        return torch.full((B, L), 0.125)
    if kind == "signed":        # negative keys and -inf too
        x = torch.randn((B, L), generator=g)
        x[:, ::7] = -float("inf")
        return x
    if kind == "narrow":        # scores packed in a narrow band (one radix bin)
        return 1e-4 * (1.0 + 1e-6 * torch.randint(0, 300, (B, L), generator=g).float())
    raise ValueError(kind)


TOPK_CASES = [
    # kind, B, L_max, k_max, seq_lens, ks
    ("random", 2, 5000, 700, [5000, 4097], [700, 1]),
    ("ties", 3, 3000, 512, [3000, 2999, 100], [512, 511, 100]),
    ("equal", 2, 4096, 300, [4096, 300], [300, 300]),
    ("signed", 2, 1500, 200, [1500, 1499], [200, 37]),
    ("narrow", 2, 9000, 1000, [9000, 8191], [1000, 999]),
    ("random", 4, 1024, 1024, [1024, 0, 5, 1024], [1024, 3, 9, 0]),
    ("random", 1, 32768, 2048, [32768], [2048]),
    # rows of 8193-32768 tokens (tiled): crowded bins, row lengths not a
    # multiple of 4, every token or none selected, a one-token budget
    ("equal", 2, 16384, 4000, [16384, 9000], [4000, 8999]),
    ("ties", 3, 32767, 3000, [32767, 20000, 0], [3000, 20000, 5]),
    ("signed", 2, 24000, 5000, [24000, 12345], [5000, 1]),
    ("narrow", 1, 32768, 4096, [32768], [4096]),
    ("ties", 1, 40000, 4096, [40000], [4096]),
    # rows whose start is not 16-byte aligned (row length not a multiple of 4)
    ("random", 3, 5001, 600, [5001, 4999, 17], [600, 600, 5]),
    # a row longer than one workgroup classifies (tiles classified across
    # workgroups) next to one it classifies itself
    ("random", 2, 140000, 3000, [140000, 131072], [3000, 2999]),
    # a threshold bin too crowded for the candidate lists: the general path
    ("narrow", 1, 131072, 4096, [131072], [4096]),
    # more tiles than the list gather takes (over 2M tokens): the general path
    ("random", 1, 2_100_000, 8192, [2_100_000], [8192]),
    ("ties", 1, 150000, 4096, [150000], [4096]),
]


@pytest.mark.parametrize("case", TOPK_CASES, ids=[f"{c[0]}-{c[2]}-{c[3]}" for c in TOPK_CASES])
@pytest.mark.parametrize("path", ["auto", "tiles"])
def test_topk_exact(dev, case, path, monkeypatch):
    """Same fp32 keys on both sides: the index sets must match bit-exactly,
    including the -1 padding and the counts.  Rows of up to 8192 tokens take
    the one-workgroup-per-row kernel unless path "tiles" forces the tiled
    kernels."""
    kind, B, L_max, k_max, lens, ks = case
    if path == "tiles":
        monkeypatch.setenv("SPEC_TOPK_PATH", "tiles")
    announce(f"topk {case[:4]} path={path}")
    g = torch.Generator().manual_seed(B * L_max + k_max)
    sc = _topk_rows(kind, B, L_max, g).float()
    seq = torch.tensor(lens, dtype=torch.int32)
    kt = torch.tensor(ks, dtype=torch.int32)
    idx, cnt = spec.topk(sc.to(dev), seq.to(dev), kt.to(dev), k_max)
    idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
    scn = sc.numpy().astype(np.float64)
    for b in range(B):
        L = min(lens[b], L_max)
        kb = max(0, min(ks[b], L, k_max))
        want = oracle.topk_indices(scn[b, :L], kb)
        assert cnt[b] == kb
        assert idx[b, :kb].tolist() == want.tolist(), b
        assert np.all(idx[b, kb:] == -1)


# ------------------------------------------------------------------ attention

ATTN_CASES = [
    # n_layers, B, L_cap, H_q, H_kv, counts, k_max
    (1, 1, 300, 4, 1, [200], 256),
    (2, 2, 700, 32, 8, [513, 64], 600),
    (1, 3, 400, 16, 8, [1, 0, 17], 64),
    (2, 1, 2000, 64, 8, [1500], 1600),
    (1, 2, 500, 8, 8, [129, 300], 300),
    (1, 1, 600, 32, 2, [520], 520),
    (3, 2, 256, 16, 16, [256, 255], 256),
    (2, 3, 300, 32, 8, [32, 0, 7], 32),
    # >= 1024 (layer, sequence, KV head) groups: one work unit per group, the
    # wavefront writes the output itself
    (4, 32, 160, 32, 8, [(37 * b) % 129 for b in range(32)], 128),
    # selections longer than 4 x 2048: splits merged by the second kernel
    (1, 2, 12000, 8, 2, [9000, 8193], 9000),
    (1, 3, 9000, 8, 1, [8400, 0, 3], 8400),
    # more than 16 query heads per KV head (MQA-like): 16-head column groups
    # over the same KV head; split selections; an empty selection
    (1, 2, 500, 32, 1, [300, 17], 300),
    (2, 1, 9000, 64, 1, [8500], 8500),
    (1, 2, 400, 64, 2, [200, 0], 256),
    # more work units than resident wavefronts (> 1024): units pipelined
    # across their boundaries, one per (layer, sequence, KV head) group with
    # empty selections breaking the chain; and split selections (partials)
    # whose empty splits restart the pipeline cold
    (5, 32, 160, 32, 8, [(37 * b) % 129 for b in range(32)], 128),
    (1, 3, 20000, 8, 8, [16384, 0, 9001], 16384),
]
PIPE_CASES = ATTN_CASES[-2:]


def _attn_inputs(case, g):
    n_layers, B, L_cap, H_q, H_kv, counts, k_max = case
    q = _rand_bf16((n_layers, B, H_q, 128), g)
    K = _rand_bf16((n_layers, B, L_cap, H_kv, 128), g)
    V = _rand_bf16((n_layers, B, L_cap, H_kv, 128), g)
    idx = torch.full((B, k_max), -1, dtype=torch.int32)
    for b in range(B):
        c = counts[b]
        sel = torch.randperm(L_cap, generator=g)[:c].sort().values
        idx[b, :c] = sel.to(torch.int32)
    return q, K, V, idx, torch.tensor(counts, dtype=torch.int32)


def _check_attn(out, lse, q, K, V, idx, counts, case):
    n_layers, B = case[0], case[1]
    qn, Kn, Vn = f64(q), f64(K), f64(V)
    worst = 0.0
    for layer in range(n_layers):
        for b in range(B):
            sel = idx[b, :counts[b]].numpy()
            want, wl = oracle.sparse_gqa_attention(qn[layer, b], Kn[layer, b], Vn[layer, b], sel)
            err = np.abs(out[layer, b] - want).max()
            worst = max(worst, err)
            assert err <= TOL_ATTN, (layer, b, err)
            if lse is not None:
                if counts[b] == 0:
                    assert np.all(np.isneginf(lse[layer, b]))
                else:
                    assert np.abs(lse[layer, b] - wl).max() <= TOL_ATTN
    return worst


@pytest.mark.parametrize("case", ATTN_CASES, ids=[str(c) for c in ATTN_CASES])
def test_attention_indexed(dev, case):
    announce(f"attn indexed {case}")
    g = torch.Generator().manual_seed(sum(case[:5]))
    q, K, V, idx, counts = _attn_inputs(case, g)
    out, lse = spec.sparse_decode_attn(q.to(dev), K.to(dev), V.to(dev), counts.to(dev),
                                       idx=idx.to(dev))
    worst = _check_attn(out.cpu().numpy(), lse.cpu().numpy(), q, K, V, idx, counts, case)
    print(f"max abs err {worst:.3e}")


@pytest.mark.parametrize("case", PIPE_CASES, ids=[str(c[:5]) for c in PIPE_CASES])
def test_pipelined_units_equal_cold_units(dev, case, monkeypatch):
    """The pipelined schedule (a wavefront's next unit fetched and staged
    while the current one streams) gives the same bits as every unit
    starting cold, in indexed and compact mode."""
    announce(f"attn pipelined vs cold {case}")
    g = torch.Generator().manual_seed(7 + sum(case[:5]))
    q, K, V, idx, counts = _attn_inputs(case, g)
    qd, Kd, Vd, idxd, cd = q.to(dev), K.to(dev), V.to(dev), idx.to(dev), counts.to(dev)
    ks, vs = spec.gather(Kd, Vd, idxd, cd)
    runs = {}
    for sched in ("auto", "cold"):
        if sched == "cold":
            monkeypatch.setenv("SPEC_ATTN_SCHEDULE", "cold")
        else:
            monkeypatch.delenv("SPEC_ATTN_SCHEDULE", raising=False)
        runs[sched] = (spec.sparse_decode_attn(qd, Kd, Vd, cd, idx=idxd),
                       spec.sparse_decode_attn(qd, ks, vs, cd))
    monkeypatch.delenv("SPEC_ATTN_SCHEDULE", raising=False)
    for mode in (0, 1):
        (o_a, l_a), (o_c, l_c) = runs["auto"][mode], runs["cold"][mode]
        assert torch.equal(o_a, o_c) and torch.equal(l_a, l_c), mode
    _check_attn(runs["auto"][0][0].cpu().numpy(), runs["auto"][0][1].cpu().numpy(), q, K, V, idx,
                counts, case)
    n_layers = case[0]
    if n_layers > 1:   # one layer per call: fewer units, every one cold; same plan per group
        for layer in range(n_layers):
            o_l, l_l = spec.sparse_decode_attn(qd[layer:layer + 1], Kd[layer:layer + 1],
                                               Vd[layer:layer + 1], cd, idx=idxd)
            assert torch.equal(o_l[0], runs["auto"][0][0][layer]), layer
            assert torch.equal(l_l[0], runs["auto"][0][1][layer]), layer


# Pipelined launches over ragged batches with at least two (layer, sequence,
# split) groups per workgroup on a 256-CU device (and at most 256
# sequences): the groups are dealt to the workgroups by selection size.
# Sizes repeat (ties keep the lower sequence first) and include empty ones.
SORTED_CASES = [
    # one unit per group: 4 x 130 groups
    (4, 130, 160, 32, 8, [(53 * b) % 129 if b % 7 else 64 for b in range(130)], 128),
    # split selections (3 splits of 864): 200 x 3 groups, partials merged
    (1, 200, 3000, 8, 2, [(911 * b) % 2501 if b % 5 else 1200 for b in range(200)], 2500),
]


@pytest.mark.parametrize("case", SORTED_CASES, ids=[str(c[:5]) for c in SORTED_CASES])
def test_sorted_order_equals_permuted(dev, case, monkeypatch):
    """Groups dealt by selection size give the same bits as the permuted
    order (every unit computes the same thing wherever it runs), in indexed
    and compact mode, and match the oracle on every (layer, sequence)."""
    announce(f"attn sorted vs permuted order {case[:5]}")
    g = torch.Generator().manual_seed(11 + sum(case[:5]))
    q, K, V, idx, counts = _attn_inputs(case, g)
    qd, Kd, Vd, idxd, cd = q.to(dev), K.to(dev), V.to(dev), idx.to(dev), counts.to(dev)
    ks, vs = spec.gather(Kd, Vd, idxd, cd)
    runs = {}
    for order in ("auto", "perm"):
        if order == "perm":
            monkeypatch.setenv("SPEC_ATTN_ORDER", "perm")
        else:
            monkeypatch.delenv("SPEC_ATTN_ORDER", raising=False)
        runs[order] = (spec.sparse_decode_attn(qd, Kd, Vd, cd, idx=idxd),
                       spec.sparse_decode_attn(qd, ks, vs, cd))
    monkeypatch.delenv("SPEC_ATTN_ORDER", raising=False)
    for mode in (0, 1):
        (o_a, l_a), (o_p, l_p) = runs["auto"][mode], runs["perm"][mode]
        assert torch.equal(o_a, o_p) and torch.equal(l_a, l_p), mode
    assert torch.equal(runs["auto"][0][0], runs["auto"][1][0])
    _check_attn(runs["auto"][0][0].cpu().numpy(), runs["auto"][0][1].cpu().numpy(), q, K, V, idx,
                counts, case)


@pytest.mark.parametrize("case", ATTN_CASES[:4], ids=[str(c) for c in ATTN_CASES[:4]])
def test_gather_then_compact_attention(dev, case):
    """spec_gather is a bit-exact row copy; compact-mode attention over its
    output equals the indexed result."""
    announce(f"gather+compact {case}")
    g = torch.Generator().manual_seed(3 + sum(case[:5]))
    q, K, V, idx, counts = _attn_inputs(case, g)
    Kd, Vd, idxd, cd = K.to(dev), V.to(dev), idx.to(dev), counts.to(dev)
    ks, vs = spec.gather(Kd, Vd, idxd, cd)
    ks, vs = ks.cpu(), vs.cpu()
    n_layers, B = case[0], case[1]
    for layer in range(n_layers):
        for b in range(B):
            c = int(counts[b])
            sel = idx[b, :c].long()
            assert torch.equal(ks[layer, b, :c].view(torch.int16), K[layer, b, sel].view(torch.int16))
            assert torch.equal(vs[layer, b, :c].view(torch.int16), V[layer, b, sel].view(torch.int16))
    out_c, lse_c = spec.sparse_decode_attn(q.to(dev), ks.to(dev), vs.to(dev), cd)
    out_i, lse_i = spec.sparse_decode_attn(q.to(dev), Kd, Vd, cd, idx=idxd)
    # same rows in the same order: identical arithmetic, identical bits
    assert torch.equal(out_c, out_i)
    _check_attn(out_c.cpu().numpy(), lse_c.cpu().numpy(), q, K, V, idx, counts, case)


def test_full_budget_is_dense(dev):
    """k = L selects every token: the fused step equals dense attention
    (checked against torch SDPA in fp64 on the CPU)."""
    announce("dense k=L")
    w = small_workload(B=2, L=300, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=300)
    x = generate(w, seed=5)
    r = spec.step(x["q_r"].to(dev), x["K_r"].to(dev), x["seq_lens"].to(dev), x["ks"].to(dev),
                  x["q"].to(dev), x["K"].to(dev), x["V"].to(dev), k_max=300)
    idx = r["idx"].cpu().numpy()
    assert (idx == np.arange(300)[None, :]).all()
    out = r["out"].cpu().numpy()
    qn, Kn, Vn = f64(x["q"]), f64(x["K"]), f64(x["V"])
    for layer in range(2):
        for b in range(2):
            qt = torch.tensor(qn[layer, b]).reshape(1, 32, 1, 128)
            kt = torch.tensor(Kn[layer, b]).permute(1, 0, 2).repeat_interleave(4, 0)[None].contiguous()
            vt = torch.tensor(Vn[layer, b]).permute(1, 0, 2).repeat_interleave(4, 0)[None].contiguous()
            want = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt).reshape(32, 128).numpy()
            assert np.abs(out[layer, b] - want).max() <= TOL_ATTN


# ------------------------------------------------------------------ fused step

STEP_CASES = [
    dict(B=2, L=1000, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=128, heavy_frac=0.05),
    dict(B=3, L=3000, H_r=16, d_r=64, n_layers=1, H_q=32, H_kv=8, k=256, heavy_frac=0.01,
         ragged_min=700),
    dict(B=1, L=5000, H_r=8, d_r=128, n_layers=2, H_q=64, H_kv=8, k=600, n_clusters=3,
         cluster_len=64),
    dict(B=2, L=4000, H_r=8, d_r=64, n_layers=1, H_q=32, H_kv=8, k=512, heavy_frac=0.02,
         recent=256),
    # one KV head for 32 query heads (MQA-like)
    dict(B=2, L=2000, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=1, k=256, heavy_frac=0.02),
]


@pytest.mark.parametrize("kw", STEP_CASES, ids=[str(i) for i in range(len(STEP_CASES))])
def test_step_vs_oracle(dev, kw):
    announce(f"step {kw}")
    w = small_workload(**kw)
    x = generate(w, seed=kw["B"] + kw["L"])
    r = spec.step(x["q_r"].to(dev), x["K_r"].to(dev), x["seq_lens"].to(dev), x["ks"].to(dev),
                  x["q"].to(dev), x["K"].to(dev), x["V"].to(dev), k_max=w.k, with_scores=True,
                  with_lse=True)
    idx, cnt = r["idx"].cpu().numpy(), r["counts"].cpu().numpy()
    out, sc = r["out"].cpu().numpy(), r["scores"].cpu().numpy().astype(np.float64)
    qrn, Krn = f64(x["q_r"]), f64(x["K_r"])
    qn, Kn, Vn = f64(x["q"]), f64(x["K"]), f64(x["V"])
    for b in range(w.B):
        L = int(x["seq_lens"][b])
        kb = min(int(x["ks"][b]), L)
        s64 = oracle.retrieval_scores(qrn[b], Krn[b], L)
        assert np.all(np.abs(sc[b, :L] - s64) <= SCORE_ABS + SCORE_REL * s64)
        assert cnt[b] == kb
        got = idx[b, :kb]
        ok, info = oracle.accept_index_set(s64, kb, got)
        assert ok, info
        # exact on the kernel's own fp32 scores
        assert got.tolist() == oracle.topk_indices(sc[b, :L], kb).tolist()
        # planted heavy tokens are recovered when the budget covers them
        heavy = x["heavy"][b]
        if 0 < len(heavy) <= kb:
            assert np.isin(heavy, got).mean() >= 0.99
        for layer in range(w.n_layers):
            want, _ = oracle.sparse_gqa_attention(qn[layer, b], Kn[layer, b], Vn[layer, b], got)
            assert np.abs(out[layer, b] - want).max() <= TOL_ATTN


ROW_CASES = STEP_CASES + [
    # the longest rows the row kernel takes: 8 heads x 4096 tokens, and
    # (head-level sets, one head per row) 8192 tokens; many short rows
    dict(B=2, L=4096, H_r=8, d_r=64, n_layers=1, H_q=32, H_kv=8, k=1000, heavy_frac=0.02,
         ragged_min=4000),
    dict(B=2, L=8192, H_r=8, d_r=64, n_layers=1, H_q=32, H_kv=8, k=2000, heavy_frac=0.02,
         ragged_min=8000),
    dict(B=50, L=300, H_r=8, d_r=64, n_layers=1, H_q=32, H_kv=8, k=64, ragged_min=1,
         heavy_frac=0.05),
]


@pytest.mark.parametrize("kw", ROW_CASES, ids=[str(i) for i in range(len(ROW_CASES))])
@pytest.mark.parametrize("head_level", [False, True], ids=["sets1", "setsHkv"])
def test_row_select_equals_tiles(dev, kw, head_level, monkeypatch):
    """Short rows: the one-workgroup-per-row kernel (normalisers merged in
    the softmax kernel's order, the same sum over heads) gives the tiled
    path's scores, selections and attention bit for bit, with and without
    the scores kept."""
    announce(f"row vs tiles {kw} head_level={head_level}")
    w = small_workload(**kw)
    x = generate(w, seed=kw["B"] * 7 + kw["L"], device=dev)
    args = [x[n] for n in ("q_r", "K_r", "seq_lens", "ks", "q", "K", "V")]
    runs = {}
    for path in ("auto", "tiles"):
        if path == "tiles":
            monkeypatch.setenv("SPEC_TOPK_PATH", "tiles")
        runs[path] = spec.step(*args, k_max=w.k, with_scores=True, with_lse=True,
                               head_level=head_level)
        runs[path + "-noscores"] = spec.step(*args, k_max=w.k, with_lse=True,
                                             head_level=head_level)
    monkeypatch.delenv("SPEC_TOPK_PATH", raising=False)
    for key in ("scores", "idx", "counts", "out", "lse"):
        assert torch.equal(runs["auto"][key], runs["tiles"][key]), key
    for key in ("idx", "counts", "out", "lse"):
        assert torch.equal(runs["auto-noscores"][key], runs["auto"][key]), key


def test_step_deterministic(dev):
    """Two runs of the fused step give identical bits (no atomics-order
    dependence, no uninitialised reads)."""
    announce("determinism")
    w = small_workload(B=2, L=3000, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=256,
                       heavy_frac=0.02)
    x = generate(w, seed=9)
    args = [x[n].to(dev) for n in ("q_r", "K_r", "seq_lens", "ks", "q", "K", "V")]
    r1 = spec.step(*args, k_max=w.k, with_scores=True, with_lse=True)
    r2 = spec.step(*args, k_max=w.k, with_scores=True, with_lse=True)
    for key in ("idx", "counts", "out", "lse", "scores"):
        assert torch.equal(r1[key], r2[key]), key


# ------------------------------------------------------------------ elastic loading

def test_delta_gather_vs_oracle(dev):
    """Several elastic updates with a fixed budget: slot->token maps equal
    the oracle's, every held row is a bit-exact copy, and the rows loaded
    equal |S_now - S_last|."""
    announce("delta gather")
    g = torch.Generator().manual_seed(21)
    n_layers, B, L_cap, H_kv, k_max = 2, 3, 900, 8, 200
    K = _rand_bf16((n_layers, B, L_cap, H_kv, 128), g)
    V = _rand_bf16((n_layers, B, L_cap, H_kv, 128), g)
    Kd, Vd = K.to(dev), V.to(dev)
    st = spec.ElasticState(n_layers, B, k_max, H_kv, 128, dev)
    budgets = [200, 150, 1]
    slot_ref = [np.full(k_max, -1) for _ in range(B)]
    prev = [np.sort(np.random.default_rng(b).choice(L_cap, budgets[b], replace=False)) for b in range(B)]
    for it in range(4):
        rng = np.random.default_rng(100 + it)
        now = []
        for b in range(B):
            keep = prev[b][rng.random(len(prev[b])) < 0.8]
            fresh = np.setdiff1d(np.arange(L_cap), prev[b])
            add = rng.choice(fresh, budgets[b] - len(keep), replace=False)
            now.append(np.sort(np.concatenate([keep, add])))
        idx = torch.full((B, k_max), -1, dtype=torch.int32)
        for b in range(B):
            idx[b, :len(now[b])] = torch.tensor(now[b], dtype=torch.int32)
        cnt = torch.tensor([len(s) for s in now], dtype=torch.int32)
        spec.delta_gather(idx.to(dev), cnt.to(dev), Kd, Vd, st)
        slots = st.slot_tok.cpu().numpy()
        nch = st.n_changed.cpu().numpy()
        kb, vb = st.kbuf.cpu(), st.vbuf.cpu()
        for b in range(B):
            ref, loads = oracle.elastic_update(slot_ref[b], now[b])
            slot_ref[b] = ref
            assert slots[b].tolist() == ref.tolist(), (it, b)
            assert nch[b] == len(loads)
            held = [(s, t) for s, t in enumerate(ref.tolist()) if t >= 0]
            ss = torch.tensor([s for s, _ in held])
            tt = torch.tensor([t for _, t in held])
            assert torch.equal(kb[:, b, ss].view(torch.int16), K[:, b, tt].view(torch.int16))
            assert torch.equal(vb[:, b, ss].view(torch.int16), V[:, b, tt].view(torch.int16))
        prev = now


def test_step_elastic_equals_indexed(dev):
    """The fused step with elastic loading (compact attention over the slot
    buffers) agrees with the indexed step, over a few appended tokens."""
    announce("step elastic")
    w = small_workload(B=2, L=2000, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=256,
                       heavy_frac=0.02, extra_cap=8)
    x = generate(w, seed=4)
    dev_x = {n: x[n].to(dev) for n in ("q_r", "K_r", "seq_lens", "ks", "q", "K", "V")}
    st = spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev)
    g = torch.Generator().manual_seed(5)
    for it in range(4):
        dev_x["seq_lens"] += 1                       # one appended token per step
        dev_x["q_r"] = (0.95 * dev_x["q_r"].float()
                        + 0.31 * torch.randn(dev_x["q_r"].shape, generator=g).to(dev)).to(torch.bfloat16)
        r_el = spec.step(**{k: dev_x[k] for k in ("q_r", "K_r", "seq_lens", "ks", "q")},
                         K=dev_x["K"], V=dev_x["V"], k_max=w.k, elastic=st, with_lse=True)
        r_ix = spec.step(**{k: dev_x[k] for k in ("q_r", "K_r", "seq_lens", "ks", "q")},
                         K=dev_x["K"], V=dev_x["V"], k_max=w.k, with_lse=True)
        assert torch.equal(r_el["idx"], r_ix["idx"])
        assert torch.allclose(r_el["out"], r_ix["out"], atol=1e-5, rtol=0)
        slots = st.slot_tok.cpu().numpy()
        for b in range(w.B):
            c = int(r_ix["counts"][b])
            assert sorted(slots[b, :c].tolist()) == r_ix["idx"][b, :c].cpu().tolist()
            assert np.all(slots[b, c:] == -1)


ELASTIC_FUSED_CASES = [
    # split selections (few groups), ragged lengths
    dict(B=3, L=3000, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=400, heavy_frac=0.02,
         ragged_min=900, extra_cap=8, steps=6),
    # one unit per group, several per wavefront (the pipelined schedule)
    dict(B=40, L=1500, H_r=8, d_r=64, n_layers=2, H_q=32, H_kv=8, k=256, heavy_frac=0.02,
         ragged_min=300, extra_cap=8, steps=4),
    # 32 query heads per KV head: two column groups read each row, one writes it
    dict(B=2, L=2500, H_r=8, d_r=64, n_layers=2, H_q=64, H_kv=2, k=300, heavy_frac=0.02,
         ragged_min=1000, extra_cap=8, steps=4),
]


@pytest.mark.parametrize("kw", ELASTIC_FUSED_CASES, ids=[str(i) for i in range(3)])
def test_elastic_attention_loads_equal_copy(dev, kw, monkeypatch):
    """Sec. 5.4's loads done by the attention (the rows of the slots an
    update assigned are read from the caches and written into their slots
    as they stream) against the update's copy followed by compact
    attention: the same outputs, lse, slot maps, slot sources, changed
    counts and slot buffers, bit for bit, step after step, with every
    update loaded by the attention ("fused"), with none ("copy") and with
    the step's own choice per sequence (mostly-new updates fused: the first
    step; the last step halves the budgets, which reloads sequences in
    full)."""
    announce(f"elastic fused vs copy {kw}")
    w = small_workload(**kw)
    x = generate(w, seed=kw["B"] + 17, device=dev)
    e = elastic_sequence(w, x, seed=kw["B"] + 17, device=dev)
    paths = ("auto", "fused", "copy")
    states = {p: spec.ElasticState(w.n_layers, w.B, w.k, w.H_kv, w.d, dev) for p in paths}
    for s in range(w.steps):
        ks = x["ks"] if s < w.steps - 1 else torch.clamp(x["ks"] // 2, min=1)
        r = {}
        for p in paths:
            if p == "auto":
                monkeypatch.delenv("SPEC_ELASTIC_PATH", raising=False)
            else:
                monkeypatch.setenv("SPEC_ELASTIC_PATH", p)
            r[p] = spec.step(e["q_r"][s], x["K_r"], e["seq_lens"][s], ks, e["q"][s], x["K"], x["V"],
                             k_max=w.k, elastic=states[p], with_lse=True)
        monkeypatch.delenv("SPEC_ELASTIC_PATH", raising=False)
        torch.cuda.synchronize()
        for p in ("auto", "fused"):
            for key in ("idx", "counts", "out", "lse"):
                assert torch.equal(r[p][key], r["copy"][key]), (s, p, key)
            for attr in ("slot_tok", "slot_src", "n_changed", "kbuf", "vbuf"):
                assert torch.equal(getattr(states[p], attr), getattr(states["copy"], attr)), (s, p, attr)
        assert int(states["fused"].n_changed.sum()) > 0 or s > 0
    # the standalone entry point with the last update's slot sources rewrites
    # the same rows and gives the step's output again
    st = states["fused"]
    kb, vb = st.kbuf.clone(), st.vbuf.clone()
    out, lse = spec.sparse_decode_attn_elastic(e["q"][w.steps - 1], x["K"], x["V"], st,
                                               r["fused"]["counts"])
    torch.cuda.synchronize()
    assert torch.equal(out, r["fused"]["out"]) and torch.equal(lse, r["fused"]["lse"])
    assert torch.equal(st.kbuf, kb) and torch.equal(st.vbuf, vb)


# ------------------------------------------------------- head-level selection

SET_SCORE_CASES = [
    # B, L_cap, H_r, d_r, n_sets (= H_kv), seq_lens
    (2, 700, 8, 64, 8, [700, 333]),       # one retrieval head per KV head
    (2, 1000, 16, 64, 8, [1000, 600]),    # two heads per group: their maximum
    (1, 520, 4, 128, 2, [520]),
    (3, 300, 8, 64, 4, [300, 1, 0]),
]


@pytest.mark.parametrize("case", SET_SCORE_CASES, ids=[str(c[:5]) for c in SET_SCORE_CASES])
def test_score_head_level(dev, case):
    B, L_cap, H_r, d_r, n_sets, lens = case
    announce(f"score head-level {case}")
    g = torch.Generator().manual_seed(2000 + B * L_cap + H_r)
    q_r = _rand_bf16((B, H_r, d_r), g)
    K_r = _rand_bf16((B, L_cap, H_r, d_r), g, 1.5)
    seq = torch.tensor(lens, dtype=torch.int32)
    got = spec.score(q_r.to(dev), K_r.to(dev), seq.to(dev), n_sets=n_sets)
    torch.cuda.synchronize()
    assert tuple(got.shape) == (B, n_sets, L_cap)
    got = got.cpu().numpy().astype(np.float64)
    for b in range(B):
        L = lens[b]
        want = oracle.head_level_scores(f64(q_r)[b], f64(K_r)[b], L, n_sets)
        err = np.abs(got[b, :, :L] - want)
        assert np.all(err <= SCORE_ABS + SCORE_REL * want), (b, err.max())
        assert np.all(np.isneginf(got[b, :, L:]))


def test_topk_head_level_rows(dev):
    """Every (sequence, set) row is an independent exact top-k with the
    sequence's length and budget; counts hold one value per sequence."""
    announce("topk head-level")
    g = torch.Generator().manual_seed(77)
    B, n_sets, L_max, k_max = 3, 4, 3000, 400
    sc = torch.rand((B, n_sets, L_max), generator=g)
    sc[1, 2] = torch.randint(0, 3, (L_max,), generator=g).float()   # ties in one row
    lens, ks = [3000, 2500, 200], [400, 399, 400]
    idx, cnt = spec.topk(sc.to(dev), torch.tensor(lens, dtype=torch.int32).to(dev),
                         torch.tensor(ks, dtype=torch.int32).to(dev), k_max)
    torch.cuda.synchronize()
    assert tuple(idx.shape) == (B, n_sets, k_max)
    idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
    scn = sc.numpy().astype(np.float64)
    for b in range(B):
        kb = min(ks[b], lens[b])
        assert cnt[b] == kb
        for s_ in range(n_sets):
            want = oracle.topk_indices(scn[b, s_, :lens[b]], kb)
            assert idx[b, s_, :kb].tolist() == want.tolist(), (b, s_)
            assert np.all(idx[b, s_, kb:] == -1)


def _attn_sets_inputs(n_layers, B, L_cap, H_q, H_kv, counts, k_max, g):
    q = _rand_bf16((n_layers, B, H_q, 128), g)
    K = _rand_bf16((n_layers, B, L_cap, H_kv, 128), g)
    V = _rand_bf16((n_layers, B, L_cap, H_kv, 128), g)
    idx = torch.full((B, H_kv, k_max), -1, dtype=torch.int32)
    for b in range(B):
        for h in range(H_kv):
            c = counts[b]
            idx[b, h, :c] = torch.randperm(L_cap, generator=g)[:c].sort().values.to(torch.int32)
    return q, K, V, idx, torch.tensor(counts, dtype=torch.int32)


SET_ATTN_CASES = [
    # n_layers, B, L_cap, H_q, H_kv, counts, k_max
    (2, 2, 700, 32, 8, [513, 64], 600),
    (1, 3, 400, 16, 4, [1, 0, 17], 64),
    (4, 32, 160, 32, 8, [(37 * b) % 129 for b in range(32)], 128),   # one unit per group
    (1, 1, 12000, 8, 2, [9000], 9000),                               # split selections
    (1, 2, 500, 64, 2, [300, 50], 300),                              # 32 query heads per set
]


@pytest.mark.parametrize("case", SET_ATTN_CASES, ids=[str(c[:5]) for c in SET_ATTN_CASES])
def test_attention_head_level_sets(dev, case):
    n_layers, B, L_cap, H_q, H_kv, counts, k_max = case
    announce(f"attn head-level {case}")
    g = torch.Generator().manual_seed(300 + sum(case[:5]))
    q, K, V, idx, cnt = _attn_sets_inputs(*case, g)
    out, lse = spec.sparse_decode_attn(q.to(dev), K.to(dev), V.to(dev), cnt.to(dev),
                                       idx=idx.to(dev))
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    qn, Kn, Vn = f64(q), f64(K), f64(V)
    for layer in range(n_layers):
        for b in range(B):
            sets = [idx[b, h, :counts[b]].numpy() for h in range(H_kv)]
            want, wl = oracle.sparse_gqa_attention_sets(qn[layer, b], Kn[layer, b], Vn[layer, b],
                                                        sets)
            assert np.abs(out[layer, b] - want).max() <= TOL_ATTN, (layer, b)
            if counts[b] == 0:
                assert np.all(np.isneginf(lse[layer, b]))
            else:
                assert np.abs(lse[layer, b] - wl).max() <= TOL_ATTN


def test_gather_head_level_then_compact(dev):
    """With one set per KV head, row j of the gathered buffer holds each
    head's piece of its own j-th token; compact attention over it equals the
    indexed result bit for bit."""
    announce("gather head-level + compact")
    g = torch.Generator().manual_seed(91)
    case = (2, 2, 500, 16, 4, [300, 77], 320)
    q, K, V, idx, cnt = _attn_sets_inputs(*case, g)
    Kd, Vd, idxd, cd = K.to(dev), V.to(dev), idx.to(dev), cnt.to(dev)
    ks, vs = spec.gather(Kd, Vd, idxd, cd)
    ksc, vsc = ks.cpu(), vs.cpu()
    for layer in range(2):
        for b in range(2):
            for h in range(4):
                c = int(cnt[b])
                sel = idx[b, h, :c].long()
                assert torch.equal(ksc[layer, b, :c, h].view(torch.int16),
                                   K[layer, b, sel, h].view(torch.int16))
                assert torch.equal(vsc[layer, b, :c, h].view(torch.int16),
                                   V[layer, b, sel, h].view(torch.int16))
    out_c, _ = spec.sparse_decode_attn(q.to(dev), ks, vs, cd)
    out_i, _ = spec.sparse_decode_attn(q.to(dev), Kd, Vd, cd, idx=idxd)
    assert torch.equal(out_c, out_i)


def test_step_head_level_vs_oracle(dev):
    announce("step head-level")
    w = small_workload(B=3, L=2500, H_r=16, d_r=64, n_layers=2, H_q=32, H_kv=8, k=300,
                       heavy_frac=0.02, ragged_min=800)
    x = generate(w, seed=6)
    d_x = {n: x[n].to(dev) for n in ("q_r", "K_r", "seq_lens", "ks", "q", "K", "V")}
    r = spec.step(d_x["q_r"], d_x["K_r"], d_x["seq_lens"], d_x["ks"], d_x["q"], d_x["K"],
                  d_x["V"], k_max=w.k, with_scores=True, with_lse=True, head_level=True)
    torch.cuda.synchronize()
    idx, cnt = r["idx"].cpu().numpy(), r["counts"].cpu().numpy()
    sc = r["scores"].cpu().numpy().astype(np.float64)
    lens, ks = x["seq_lens"].numpy(), x["ks"].numpy()
    for b in range(w.B):
        L, kb = int(lens[b]), min(int(ks[b]), int(lens[b]))
        assert cnt[b] == kb
        s64 = oracle.head_level_scores(f64(x["q_r"][b]), f64(x["K_r"][b]), L, w.H_kv)
        sets = []
        for h in range(w.H_kv):
            err = np.abs(sc[b, h, :L] - s64[h])
            assert np.all(err <= SCORE_ABS + SCORE_REL * s64[h]), (b, h)
            assert idx[b, h, :kb].tolist() == oracle.topk_indices(sc[b, h, :L], kb).tolist()
            ok, info = oracle.accept_index_set(s64[h], kb, idx[b, h, :kb])
            assert ok, (b, h, info)
            sets.append(idx[b, h, :kb])
        for layer in range(w.n_layers):
            want, wl = oracle.sparse_gqa_attention_sets(f64(x["q"][layer, b]), f64(x["K"][layer, b]),
                                                        f64(x["V"][layer, b]), sets)
            assert np.abs(r["out"][layer, b].cpu().numpy() - want).max() <= TOL_ATTN
            assert np.abs(r["lse"][layer, b].cpu().numpy() - wl).max() <= TOL_ATTN
