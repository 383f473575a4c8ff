"""Seeded random shapes, HIP path vs the fp64 oracle.

* Retrieval scores: any head count up to 16, d_r 64 or 128, ragged lengths
  (zero and one included), L_max below L_cap; the internal score gate.
* Top-k: the same fp32 keys on both sides, so the index sets, the -1 padding
  and the counts must match exactly.  Shapes mix short rows, rows spanning
  several classify tiles and rows past 64 tiles; lengths and budgets are
  ragged, zero or the whole row.
* Elastic delta-gather: fixed, growing and shrinking budgets per sequence,
  overlaps from none to full between consecutive selections; the slot map
  equals the oracle's pairing (from the empty state when the budget shrank
  below a kept token's slot: the documented full reload), every held row is
  a bit-exact copy, and the rows loaded equal what the pairing loads.
* Sparse GQA attention (indexed: the gather fused into the loads): every
  supported query-group size up to 64, one to three layers, one token set per
  sequence or one per KV head, ragged and empty selections, budgets up to the
  whole cache; max-abs error within the
  attention tolerance, lse included.  Batches of 64-256 ragged sequences
  (the attention's order by selection size) give the same bits as the
  permuted order.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2512_00722_amd as spec
from tests.gpu_helpers import SCORE_ABS, SCORE_REL, TOL_ATTN, announce, f64, need_gpu
from tests.test_parity_gpu import _topk_rows

pytestmark = pytest.mark.gpu

KINDS = ["random", "ties", "equal", "signed", "narrow"]


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def _ragged(rng, n, hi, p_other=0.3):
    """n values: mostly hi, some uniform in [0, hi]."""
    return [int(rng.integers(0, hi + 1)) if rng.random() < p_other else hi for _ in range(n)]


@pytest.mark.parametrize("seed", range(4))
def test_topk_random_shapes(dev, seed):
    rng = np.random.default_rng(100 + seed)
    for it in range(15):
        kind = KINDS[(seed * 15 + it) % len(KINDS)]
        B = int(rng.integers(1, 6))
        L_max = int(rng.choice([rng.integers(1, 4096), rng.integers(4096, 70000),
                                rng.integers(70000, 150001)]))
        k_max = int(rng.integers(1, min(L_max, 12000) + 1))
        lens = _ragged(rng, B, L_max)
        ks = _ragged(rng, B, k_max)
        announce(f"topk random seed={seed} it={it} kind={kind} B={B} L_max={L_max} k_max={k_max}")
        g = torch.Generator().manual_seed(10_000 * seed + it)
        sc = _topk_rows(kind, B, L_max, g).float()
        idx, cnt = spec.topk(sc.to(dev), torch.tensor(lens, dtype=torch.int32).to(dev),
                             torch.tensor(ks, dtype=torch.int32).to(dev), k_max)
        idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
        scn = sc.numpy().astype(np.float64)
        for b in range(B):
            L = min(lens[b], L_max)
            kb = max(0, min(ks[b], L, k_max))
            want = oracle.topk_indices(scn[b, :L], kb)
            assert cnt[b] == kb, (it, b)
            assert idx[b, :kb].tolist() == want.tolist(), (it, b, kind, L, kb)
            assert np.all(idx[b, kb:] == -1), (it, b)


@pytest.mark.parametrize("seed", range(4))
def test_attention_random_shapes(dev, seed):
    rng = np.random.default_rng(200 + seed)
    for it in range(8):
        n_layers = int(rng.integers(1, 4))
        B = int(rng.integers(1, 5))
        H_kv = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.choice([g for g in (1, 2, 4, 8, 16, 32, 64) if g * H_kv <= 128]))
        H_q = H_kv * G
        L_cap = int(rng.integers(64, 4001))
        k_max = int(rng.integers(1, L_cap + 1))
        counts = _ragged(rng, B, k_max, p_other=0.5)
        g = torch.Generator().manual_seed(20_000 * seed + it)
        q = torch.randn((n_layers, B, H_q, 128), generator=g).to(torch.bfloat16)
        K = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g).to(torch.bfloat16)
        V = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g).to(torch.bfloat16)
        sets = rng.random() < 0.35  # one token set per KV head (head-level selection)
        n_sets = H_kv if sets else 1
        idx = torch.full((B, n_sets, k_max), -1, dtype=torch.int32)
        for b in range(B):
            for s_ in range(n_sets):
                sel = torch.randperm(L_cap, generator=g)[:counts[b]].sort().values
                idx[b, s_, :counts[b]] = sel.to(torch.int32)
        if not sets:
            idx = idx[:, 0].contiguous()
        announce(f"attn random seed={seed} it={it} layers={n_layers} B={B} H_q={H_q} "
                 f"H_kv={H_kv} L_cap={L_cap} k_max={k_max} counts={counts} sets={sets}")
        cnt = torch.tensor(counts, dtype=torch.int32)
        out, lse = spec.sparse_decode_attn(q.to(dev), K.to(dev), V.to(dev), cnt.to(dev),
                                           idx=idx.to(dev), with_lse=True)
        out, lse = out.cpu().numpy(), lse.cpu().numpy()
        qn, Kn, Vn = f64(q), f64(K), f64(V)
        for layer in range(n_layers):
            for b in range(B):
                if sets:
                    want, want_lse = oracle.sparse_gqa_attention_sets(
                        qn[layer, b], Kn[layer, b], Vn[layer, b],
                        [idx[b, s_, :counts[b]].numpy() for s_ in range(H_kv)])
                else:
                    want, want_lse = oracle.sparse_gqa_attention(
                        qn[layer, b], Kn[layer, b], Vn[layer, b], idx[b, :counts[b]].numpy())
                if counts[b] == 0:
                    assert np.all(out[layer, b] == 0.0)
                    assert np.all(np.isneginf(lse[layer, b]))
                    continue
                err = np.abs(out[layer, b] - want).max()
                assert err <= TOL_ATTN, (it, layer, b, err)
                assert np.abs(lse[layer, b] - want_lse).max() <= TOL_ATTN, (it, layer, b)


@pytest.mark.parametrize("seed", range(3))
def test_attention_random_ragged_batches(dev, seed, monkeypatch):
    """Batches of 64-256 sequences with unequal selections, enough
    (layer, sequence) groups for the attention to deal them to its
    workgroups by selection size: the same bits as the permuted order, and
    sampled (layer, sequence) outputs against the oracle."""
    rng = np.random.default_rng(500 + seed)
    for it in range(4):
        B = int(rng.integers(64, 257))
        n_layers = int(rng.integers(-(-520 // B), -(-520 // B) + 3))
        H_kv = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.choice([g for g in (1, 2, 4, 8, 16, 32) if g * H_kv <= 128]))
        H_q = H_kv * G
        L_cap = int(rng.integers(32, 257))
        k_max = int(rng.integers(1, L_cap + 1))
        counts = _ragged(rng, B, k_max, p_other=0.7)
        announce(f"attn ragged batch seed={seed} it={it} layers={n_layers} B={B} H_q={H_q} "
                 f"H_kv={H_kv} L_cap={L_cap} k_max={k_max}")
        g = torch.Generator(device=dev).manual_seed(30_000 * seed + it)
        q = torch.randn((n_layers, B, H_q, 128), generator=g, device=dev).to(torch.bfloat16)
        K = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g, device=dev).to(torch.bfloat16)
        V = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g, device=dev).to(torch.bfloat16)
        gc = torch.Generator().manual_seed(40_000 * seed + it)
        idx = torch.full((B, k_max), -1, dtype=torch.int32)
        for b in range(B):
            idx[b, :counts[b]] = torch.randperm(L_cap, generator=gc)[:counts[b]].sort().values.int()
        cnt = torch.tensor(counts, dtype=torch.int32)
        runs = {}
        for order in ("auto", "perm"):
            if order == "perm":
                monkeypatch.setenv("SPEC_ATTN_ORDER", "perm")
            else:
                monkeypatch.delenv("SPEC_ATTN_ORDER", raising=False)
            runs[order] = spec.sparse_decode_attn(q, K, V, cnt.to(dev), idx=idx.to(dev))
        monkeypatch.delenv("SPEC_ATTN_ORDER", raising=False)
        assert torch.equal(runs["auto"][0], runs["perm"][0]), it
        assert torch.equal(runs["auto"][1], runs["perm"][1]), it
        out, lse = runs["auto"][0].cpu().numpy(), runs["auto"][1].cpu().numpy()
        assert np.all(np.isfinite(out)), it
        for _ in range(12):
            layer, b = int(rng.integers(0, n_layers)), int(rng.integers(0, B))
            want, want_lse = oracle.sparse_gqa_attention(
                f64(q[layer, b].cpu()), f64(K[layer, b].cpu()), f64(V[layer, b].cpu()),
                idx[b, :counts[b]].numpy())
            if counts[b] == 0:
                assert np.all(out[layer, b] == 0.0) and np.all(np.isneginf(lse[layer, b]))
                continue
            assert np.abs(out[layer, b] - want).max() <= TOL_ATTN, (it, layer, b)
            assert np.abs(lse[layer, b] - want_lse).max() <= TOL_ATTN, (it, layer, b)


@pytest.mark.parametrize("seed", range(3))
def test_score_random_shapes(dev, seed):
    rng = np.random.default_rng(300 + seed)
    for it in range(8):
        B = int(rng.integers(1, 5))
        H_r = int(rng.integers(1, 17))
        d_r = int(rng.choice([64, 128]))
        L_cap = int(rng.integers(1, 9000))
        L_max = int(rng.integers(1, L_cap + 1))
        lens = [int(rng.choice([0, 1, L_max, int(rng.integers(0, L_max + 1))])) for _ in range(B)]
        announce(f"score random seed={seed} it={it} B={B} H_r={H_r} d_r={d_r} L_cap={L_cap} "
                 f"L_max={L_max} lens={lens}")
        g = torch.Generator().manual_seed(30_000 * seed + it)
        q_r = torch.randn((B, H_r, d_r), generator=g).to(torch.bfloat16)
        K_r = (torch.randn((B, L_cap, H_r, d_r), generator=g) * 1.5).to(torch.bfloat16)
        got = spec.score(q_r.to(dev), K_r.to(dev), torch.tensor(lens, dtype=torch.int32).to(dev),
                         L_max=L_max).cpu().numpy().astype(np.float64)
        qn, Kn = f64(q_r), f64(K_r)
        for b in range(B):
            L = min(lens[b], L_max)
            want = oracle.retrieval_scores(qn[b], Kn[b], L)
            assert np.all(np.abs(got[b, :L] - want) <= SCORE_ABS + SCORE_REL * want), (it, b)
            assert np.all(np.isneginf(got[b, L:L_max])), (it, b)


@pytest.mark.parametrize("seed", range(5))
def test_elastic_random_shapes(dev, seed):
    rng = np.random.default_rng(400 + seed)
    n_layers = int(rng.integers(1, 3))
    B = int(rng.integers(1, 5))
    H_kv = int(rng.choice([1, 2, 4, 8]))
    L_cap = int(rng.integers(50, 3001))
    k_max = int(rng.integers(1, min(L_cap, 800) + 1))
    announce(f"elastic random seed={seed} layers={n_layers} B={B} H_kv={H_kv} L_cap={L_cap} "
             f"k_max={k_max}")
    g = torch.Generator().manual_seed(40_000 + seed)
    K = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g).to(torch.bfloat16)
    V = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g).to(torch.bfloat16)
    Kd, Vd = K.to(dev), V.to(dev)
    st = spec.ElasticState(n_layers, B, k_max, H_kv, 128, dev)
    budget = [int(rng.integers(0, k_max + 1)) for _ in range(B)]
    slot_ref = [np.full(k_max, -1) for _ in range(B)]
    prev = [np.zeros(0, dtype=np.int64) for _ in range(B)]
    n_reload = 0
    for it in range(8):
        keep_p = float(rng.choice([0.0, 0.5, 0.8, 0.95, 1.0]))
        now = []
        for b in range(B):
            r = rng.random()
            if r < 0.25:  # the budget grows
                budget[b] = int(rng.integers(budget[b], k_max + 1))
            elif r < 0.45:  # the budget shrinks
                budget[b] = int(rng.integers(0, budget[b] + 1))
            keep = prev[b][rng.random(len(prev[b])) < keep_p][:budget[b]]
            pool = np.setdiff1d(np.arange(L_cap), keep)  # may return dropped tokens
            add = rng.choice(pool, budget[b] - len(keep), replace=False)
            now.append(np.sort(np.concatenate([keep, add]).astype(np.int64)))
        idx = torch.full((B, k_max), -1, dtype=torch.int32)
        for b in range(B):
            idx[b, :len(now[b])] = torch.tensor(now[b], dtype=torch.int32)
        cnt = torch.tensor([len(x) for x in now], dtype=torch.int32)
        spec.delta_gather(idx.to(dev), cnt.to(dev), Kd, Vd, st)
        slots = st.slot_tok.cpu().numpy()
        nch = st.n_changed.cpu().numpy()
        kb, vb = st.kbuf.cpu(), st.vbuf.cpu()
        for b in range(B):
            # a token of S_now held at a slot >= |S_now| forces a full reload
            in_now = np.isin(slot_ref[b], now[b]) & (slot_ref[b] >= 0)
            reload = bool(np.any(in_now[len(now[b]):]))
            n_reload += reload
            start = np.full(k_max, -1) if reload else slot_ref[b]
            ref, loads = oracle.elastic_update(start, now[b])
            slot_ref[b] = ref
            assert slots[b].tolist() == ref.tolist(), (it, b, reload)
            assert nch[b] == len(loads), (it, b, reload)
            if not reload:
                assert len(loads) == len(np.setdiff1d(now[b], prev[b])), (it, b)
            held = [(sl, t) for sl, t in enumerate(ref.tolist()) if t >= 0]
            if held:
                ss = torch.tensor([sl for sl, _ in held])
                tt = torch.tensor([t for _, t in held])
                assert torch.equal(kb[:, b, ss].view(torch.int16), K[:, b, tt].view(torch.int16))
                assert torch.equal(vb[:, b, ss].view(torch.int16), V[:, b, tt].view(torch.int16))
        prev = now
    print(f"[elastic] seed={seed}: {n_reload} full reloads", flush=True)


@pytest.mark.parametrize("seed", range(4))
def test_elastic_attention_random_shapes(dev, seed):
    """Sec. 5.4's loads done by the attention, on random shapes (query-group
    sizes up to 64, so that some KV heads are read by several column groups,
    one of which writes) and random update sequences: after each update
    (spec_delta_gather, which records the slot sources) the slots it loaded
    are overwritten with garbage; the elastic attention must read those rows
    from the caches, give the compact attention's output over the clean
    slots bit for bit, and leave the slots exactly as the copy had."""
    rng = np.random.default_rng(500 + seed)
    n_layers = int(rng.integers(1, 4))
    B = int(rng.integers(1, 5))
    H_kv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([g for g in (1, 2, 4, 8, 16, 32, 64) if g * H_kv <= 128]))
    H_q = H_kv * G
    L_cap = int(rng.integers(64, 3001))
    k_max = int(rng.integers(1, min(L_cap, 1500) + 1))
    announce(f"elastic attention random seed={seed} layers={n_layers} B={B} H_q={H_q} "
             f"H_kv={H_kv} L_cap={L_cap} k_max={k_max}")
    g = torch.Generator().manual_seed(50_000 + seed)
    Kd = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g).to(torch.bfloat16).to(dev)
    Vd = torch.randn((n_layers, B, L_cap, H_kv, 128), generator=g).to(torch.bfloat16).to(dev)
    st = spec.ElasticState(n_layers, B, k_max, H_kv, 128, dev)
    prev = [np.zeros(0, dtype=np.int64) for _ in range(B)]
    for it in range(6):
        keep_p = float(rng.choice([0.0, 0.5, 0.8, 1.0]))
        now = []
        for b in range(B):
            budget = int(rng.integers(0, k_max + 1))
            keep = prev[b][rng.random(len(prev[b])) < keep_p][:budget]
            pool = np.setdiff1d(np.arange(L_cap), keep)
            add = rng.choice(pool, budget - len(keep), replace=False)
            now.append(np.sort(np.concatenate([keep, add]).astype(np.int64)))
        idx = torch.full((B, k_max), -1, dtype=torch.int32)
        for b in range(B):
            idx[b, :len(now[b])] = torch.tensor(now[b], dtype=torch.int32)
        cnt = torch.tensor([len(x) for x in now], dtype=torch.int32).to(dev)
        spec.delta_gather(idx.to(dev), cnt, Kd, Vd, st)
        q = torch.randn((n_layers, B, H_q, 128), generator=g).to(torch.bfloat16).to(dev)
        ref_out, ref_lse = spec.sparse_decode_attn(q, st.kbuf, st.vbuf, cnt)
        torch.cuda.synchronize()
        clean_k, clean_v = st.kbuf.clone(), st.vbuf.clone()
        loaded = st.slot_src >= 0                       # [B, k_max]
        assert int(loaded.sum()) == int(st.n_changed.sum()), it
        st.kbuf[:, loaded] = 7.0                        # garbage in every loaded slot
        st.vbuf[:, loaded] = -3.0
        out, lse = spec.sparse_decode_attn_elastic(q, Kd, Vd, st, cnt)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse), it
        assert torch.equal(st.kbuf, clean_k) and torch.equal(st.vbuf, clean_v), it
        prev = now
