"""MLA sparse decode attention on the GPU against the fp64 oracle (Sec. 4.3,
"Support for MLA"): selected latent rows, per-head keys and values raised by
W_UK / W_UV (the oracle forms them explicitly; the kernels use the absorbed
form), softmax over the selection, all layers in one call.

Tolerance: max |out - out64| <= 2e-3 and the same on lse, the bound of the
other attention path.  The absorbed query is rounded to bf16 once for the
matrix cores (the latent output enters them as a bf16 high + low pair,
~2^-16 relative, the softmax weights as a truncated pair, 2^-14); the test
prints the measured error.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2512_00722_amd as spec
from tests.gpu_helpers import TOL_ATTN, announce, f64, need_gpu
from workloads import WORKLOADS, generate_mla, small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return need_gpu()


def _oracle(x, layer, b, idx_b, heads=None):
    """fp64 oracle of one (layer, sequence), optionally on a subset of heads."""
    hs = slice(None) if heads is None else heads
    q = f64(x["q_mla"][layer, b])[hs]
    ckv = f64(x["ckv"][layer, b])
    return oracle.mla_sparse_attention(q[:, :128], q[:, 128:], ckv[:, :512], ckv[:, 512:],
                                       f64(x["w_uk"][layer])[hs], f64(x["w_uv"][layer])[hs],
                                       idx_b)


def _random_idx(rng, B, k_max, L, counts):
    idx = np.full((B, k_max), -1, dtype=np.int32)
    for b in range(B):
        sel = np.sort(rng.choice(L, counts[b], replace=False))
        idx[b, :counts[b]] = sel
    return idx


# (B, L, k_max, n_layers, H, counts): one split per unit, many splits
# (merge of 12 partial results), empty and single-token selections, more
# than 16 sequences (the output kernel's second group), 64 heads
CASES = [
    (2, 300, 64, 2, 64, [64, 37]),
    (1, 5000, 3000, 2, 128, [2999]),
    (3, 200, 40, 1, 128, [40, 0, 1]),
    (20, 180, 100, 1, 64, [100 - 3 * i for i in range(20)]),
    (4, 2100, 2048, 1, 128, [2048, 1500, 700, 33]),
]


@pytest.mark.parametrize("case", CASES, ids=[f"B{c[0]}_L{c[1]}_k{c[2]}_l{c[3]}_H{c[4]}"
                                             for c in CASES])
def test_mla_cases(dev, case):
    B, L, k_max, n_layers, H, counts = case
    announce(f"mla {case}")
    w = small_workload(B=B, L=L, k=k_max, n_layers=n_layers, H_q=H, H_kv=1, mla=True)
    x = generate_mla(w, seed=7, device=dev)
    rng = np.random.default_rng(11)
    idx = _random_idx(rng, B, k_max, L, counts)
    idx_t = torch.as_tensor(idx, device=dev)
    cnt_t = torch.as_tensor(np.array(counts, dtype=np.int32), device=dev)
    out, lse = spec.mla_sparse_decode_attn(x["q_mla"], x["ckv"], x["w_uk"], x["w_uv"], idx_t,
                                           cnt_t)
    torch.cuda.synchronize()
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    # the oracle raises every selected latent for every head: keep it to a
    # few seconds by checking a spread of heads on the long selections
    heads = (np.arange(H) if max(counts) * H <= 20000
             else np.array([0, 5, 15, 16, 31, 32, 63, H - 1]))
    worst = 0.0
    for layer in range(n_layers):
        for b in range(B):
            if counts[b] == 0:
                assert np.all(out[layer, b] == 0) and np.all(np.isneginf(lse[layer, b]))
                continue
            want, wl = _oracle(x, layer, b, idx[b, :counts[b]], heads=heads)
            err = np.abs(out[layer, b][heads] - want).max()
            worst = max(worst, err)
            assert err <= TOL_ATTN, (layer, b, err)
            assert np.abs(lse[layer, b][heads] - wl).max() <= TOL_ATTN, (layer, b)
    print(f"max |out - oracle| = {worst:.2e}")


def test_mla_strided_cache_and_repeat(dev):
    """A cache with padding between sequences and layers (strides from the
    tensor view) gives the same result as a packed one, bit for bit, and a
    second call repeats the first."""
    announce("mla strided cache")
    w = small_workload(B=2, L=96, k=50, n_layers=2, H_q=64, H_kv=1, mla=True)
    x = generate_mla(w, seed=3, device=dev)
    big = torch.zeros((2, 2, 128, 576), dtype=torch.bfloat16, device=dev)
    big[:, :, :96] = x["ckv"]
    idx = torch.as_tensor(_random_idx(np.random.default_rng(2), 2, 50, 96, [50, 41]), device=dev)
    cnt = torch.tensor([50, 41], dtype=torch.int32, device=dev)
    o1, l1 = spec.mla_sparse_decode_attn(x["q_mla"], x["ckv"], x["w_uk"], x["w_uv"], idx, cnt)
    o2, l2 = spec.mla_sparse_decode_attn(x["q_mla"], big[:, :, :96], x["w_uk"], x["w_uv"], idx,
                                         cnt)
    o3, _ = spec.mla_sparse_decode_attn(x["q_mla"], x["ckv"], x["w_uk"], x["w_uv"], idx, cnt)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2) and torch.equal(o1, o3)


def test_mla_full_size_step(dev):
    """The 61-layer, 128-head MLA workload at full size: retrieval scores,
    top-k, then MLA attention over the selected latent rows of every layer;
    sampled (layer, sequence) pairs against the oracle on a subset of heads."""
    w = WORKLOADS["b8_l32768_k2048_mla"]
    announce(f"mla full size {w.name}")
    x = generate_mla(w, seed=0, device=dev)
    scores = spec.score(x["q_r"], x["K_r"], x["seq_lens"])
    idx, counts = spec.topk(scores, x["seq_lens"], x["ks"], w.k)
    out, lse = spec.mla_sparse_decode_attn(x["q_mla"], x["ckv"], x["w_uk"], x["w_uv"], idx,
                                           counts)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all() and torch.isfinite(lse).all()
    idx_h = idx.cpu().numpy()
    heads = np.array([0, 1, 63, 64, 100, 127])
    worst = 0.0
    for layer, b in [(0, 0), (30, 3), (60, 7)]:
        want, wl = _oracle(x, layer, b, idx_h[b, :w.k], heads=heads)
        got = out[layer, b].cpu().numpy()[heads]
        err = np.abs(got - want).max()
        worst = max(worst, err)
        assert err <= TOL_ATTN, (layer, b, err)
        assert np.abs(lse[layer, b].cpu().numpy()[heads] - wl).max() <= TOL_ATTN
    print(f"max |out - oracle| = {worst:.2e}")
    del x
    torch.cuda.empty_cache()


@pytest.mark.parametrize("seed", range(3))
def test_mla_random_shapes(dev, seed):
    """Seeded random shapes: sequences, layers, 64 or 128 heads, ragged and
    empty selections up to the whole cache; eight random heads of every
    (layer, sequence) against the oracle."""
    rng = np.random.default_rng(500 + seed)
    for it in range(3):
        B = int(rng.integers(1, 7))
        n_layers = int(rng.integers(1, 3))
        H = int(rng.choice([64, 128]))
        L = int(rng.integers(16, 1500))
        k_max = int(rng.integers(1, L + 1))
        counts = [int(rng.integers(0, k_max + 1)) if rng.random() < 0.5 else k_max
                  for _ in range(B)]
        announce(f"mla random seed={seed} it={it} B={B} layers={n_layers} H={H} L={L} "
                 f"k_max={k_max} counts={counts}")
        w = small_workload(B=B, L=L, k=k_max, n_layers=n_layers, H_q=H, H_kv=1, mla=True)
        x = generate_mla(w, seed=100 * seed + it, device=dev)
        idx = _random_idx(rng, B, k_max, L, counts)
        out, lse = spec.mla_sparse_decode_attn(
            x["q_mla"], x["ckv"], x["w_uk"], x["w_uv"], torch.as_tensor(idx, device=dev),
            torch.as_tensor(np.array(counts, dtype=np.int32), device=dev))
        out, lse = out.cpu().numpy(), lse.cpu().numpy()
        heads = np.sort(rng.choice(H, 8, replace=False))
        for layer in range(n_layers):
            for b in range(B):
                if counts[b] == 0:
                    assert np.all(out[layer, b] == 0) and np.all(np.isneginf(lse[layer, b]))
                    continue
                want, wl = _oracle(x, layer, b, idx[b, :counts[b]], heads=heads)
                assert np.abs(out[layer, b][heads] - want).max() <= TOL_ATTN, (it, layer, b)
                assert np.abs(lse[layer, b][heads] - wl).max() <= TOL_ATTN, (it, layer, b)
