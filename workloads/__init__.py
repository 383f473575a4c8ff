"""Seeded synthetic decode-step workloads (input generation only).

This package builds the inputs that both the HIP path and the CPU oracle
consume.  It holds none of the method's arithmetic: it draws Gaussian
tensors, plants structure into the retrieval key cache, rounds to bf16 and
places the tensors on a device.  The paper measures on LongBench/LongWriter
with 8B models; these workloads stand in for their decode-step shapes
(32 layers, 32 query / 8 KV heads, head dim 128, contexts 4K-128K, budgets
512-4096).  No benchmark item is used.

Structure recipe (all tensors drawn N(0,1) in fp32, planted, then rounded to
bf16 with round-to-nearest-even):

* heavy tokens: K_r[b, t, h, :] += heavy_gain * q_r[b, h] / |q_r[b, h]| in
  every retrieval head, for a seeded set of positions;
* recency bias: the last `recent` tokens get += recent_gain * q_r/|q_r|;
* clusters: `n_clusters` runs of `cluster_len` contiguous heavy tokens.

Positions and ragged lengths come from numpy's PCG64 (portable); tensor
values come from a torch generator on the target device, seeded per tensor
from (seed, tensor name).
"""

from __future__ import annotations

import dataclasses
import zlib
from typing import Optional

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "BENCH_WORKLOAD", "tensor_seed",
           "generate", "elastic_sequence", "algorithmic_bytes", "small_workload",
           "frontend_inputs", "frontend_bytes", "generate_mla", "mla_bytes", "mla_attn_bytes"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    L: int                 # context length (upper bound for ragged)
    H_r: int
    d_r: int
    n_layers: int
    H_q: int
    H_kv: int
    d: int
    k: int
    heavy_frac: float = 0.0
    recent: int = 0        # length of the recency-biased tail
    recent_gain: float = 1.0
    heavy_gain: float = 2.0
    n_clusters: int = 0
    cluster_len: int = 0
    ragged_min: int = 0    # >0: L_b uniform integer in [ragged_min, L]
    k_frac_den: int = 0    # >0: k_b = min(k, L_b // k_frac_den)
    extra_cap: int = 0     # spare capacity for appended tokens
    steps: int = 1         # decode steps simulated (elastic workload)
    drift: float = 0.95    # AR(1) coefficient of q_r across steps
    # retrieval-head front end (synthetic weights; an 8B-class model's
    # embedding table and width, its rotary base, and the 2K training context
    # of the distilled model that YaRN extends to L_cap)
    hidden: int = 4096
    vocab: int = 128256
    rope_base: float = 500000.0
    orig_ctx: int = 2048
    # MLA models (DeepSeek-V3 / Kimi-K2 shapes): H_q query heads attend over
    # a latent cache of d_c + d_rope per token (H_kv and d are unused)
    mla: bool = False
    d_c: int = 512
    d_rope: int = 64
    d_nope: int = 128
    d_v: int = 128

    @property
    def L_cap(self) -> int:
        return self.L + self.extra_cap

    @property
    def G(self) -> int:
        return self.H_q // self.H_kv

    @property
    def yarn_scale(self) -> float:
        """Context-extension factor from the training context to L_cap."""
        return max(1.0, self.L_cap / self.orig_ctx)


# The five decode-step workloads (shapes of the paper's cloud/edge settings).
WORKLOADS = {
    "b1_l4096_k512_1layer": Workload(
        "b1_l4096_k512_1layer", B=1, L=4096, H_r=8, d_r=64, n_layers=1,
        H_q=32, H_kv=8, d=128, k=512, heavy_frac=0.05),
    "b8_l32768_k2048_32layers": Workload(
        "b8_l32768_k2048_32layers", B=8, L=32768, H_r=8, d_r=64, n_layers=32,
        H_q=32, H_kv=8, d=128, k=2048, heavy_frac=0.02, recent=256),
    "b32_l16384_k1024_hr16": Workload(
        "b32_l16384_k1024_hr16", B=32, L=16384, H_r=16, d_r=64, n_layers=32,
        H_q=32, H_kv=8, d=128, k=1024, heavy_frac=0.01),
    "b1_l131072_k4096_g8": Workload(
        "b1_l131072_k4096_g8", B=1, L=131072, H_r=8, d_r=128, n_layers=32,
        H_q=64, H_kv=8, d=128, k=4096, n_clusters=3, cluster_len=512, hidden=8192),
    "b8_l32768_k2048_mla": Workload(
        "b8_l32768_k2048_mla", B=8, L=32768, H_r=8, d_r=64, n_layers=61,
        H_q=128, H_kv=1, d=128, k=2048, heavy_frac=0.02, recent=256, mla=True),
    "b64_ragged_l2k_16k_elastic": Workload(
        "b64_ragged_l2k_16k_elastic", B=64, L=16384, H_r=8, d_r=64,
        n_layers=32, H_q=32, H_kv=8, d=128, k=2048, heavy_frac=0.02,
        ragged_min=2048, k_frac_den=4, extra_cap=16, steps=16),
}

# The workload the throughput metric is quoted on.
BENCH_WORKLOAD = "b8_l32768_k2048_32layers"


def small_workload(**kw) -> Workload:
    """A custom (usually tiny) workload for tests."""
    base = dict(name="custom", B=1, L=64, H_r=2, d_r=64, n_layers=1, H_q=4,
                H_kv=1, d=128, k=8)
    base.update(kw)
    return Workload(**base)


def tensor_seed(seed: int, name: str) -> int:
    return zlib.crc32(f"{int(seed)}:{name}".encode()) & 0x7FFFFFFF


def _gen(device, seed, name) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(tensor_seed(seed, name))
    return g


def _lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    if w.ragged_min > 0:
        return rng.integers(w.ragged_min, w.L, size=w.B, endpoint=True)
    return np.full(w.B, w.L, dtype=np.int64)


def _budgets(w: Workload, lens: np.ndarray) -> np.ndarray:
    if w.k_frac_den > 0:
        return np.minimum(w.k, lens // w.k_frac_den)
    return np.full(w.B, w.k, dtype=np.int64)


def _heavy_positions(w: Workload, L_b: int, rng: np.random.Generator) -> np.ndarray:
    """Planted heavy positions for one sequence (sorted, distinct)."""
    if w.n_clusters > 0:
        starts = []
        span = L_b - w.cluster_len
        while len(starts) < w.n_clusters:
            s = int(rng.integers(0, span + 1))
            if all(abs(s - o) >= w.cluster_len for o in starts):
                starts.append(s)
        pos = np.concatenate([np.arange(s, s + w.cluster_len) for s in sorted(starts)])
        return pos
    n_heavy = int(round(w.heavy_frac * L_b))
    if n_heavy == 0:
        return np.zeros((0,), dtype=np.int64)
    hi = L_b - w.recent if w.recent > 0 else L_b
    return np.sort(rng.choice(hi, size=n_heavy, replace=False))


def generate(w: Workload, seed: int = 0, device="cpu", with_kv: bool = True,
             layers: Optional[range] = None):
    """Draw one decode step's inputs for workload `w`.

    Returns a dict of tensors on `device`:
      q_r [B, H_r, d_r] bf16, K_r [B, L_cap, H_r, d_r] bf16,
      seq_lens [B] int32, ks [B] int32,
      q [n_layers, B, H_q, d] bf16,
      K, V [n_layers, B, L_cap, H_kv, d] bf16 (if with_kv),
      heavy: list of numpy arrays of planted positions per sequence.
    Rows at or beyond a sequence's length hold random values too; they must
    never be read by the method.
    """
    device = torch.device(device)
    rng = np.random.default_rng(seed)
    lens = _lengths(w, rng)
    ks = _budgets(w, lens)
    heavy = [_heavy_positions(w, int(lens[b]), rng) for b in range(w.B)]

    q_r = torch.randn((w.B, w.H_r, w.d_r), generator=_gen(device, seed, "q_r"),
                      device=device, dtype=torch.float32).to(torch.bfloat16)
    qf = q_r.float()
    qhat = qf / qf.norm(dim=-1, keepdim=True)             # [B, H_r, d_r]

    K_r = torch.empty((w.B, w.L_cap, w.H_r, w.d_r), dtype=torch.bfloat16, device=device)
    for b in range(w.B):
        row = torch.randn((w.L_cap, w.H_r, w.d_r), generator=_gen(device, seed, f"K_r.{b}"),
                          device=device, dtype=torch.float32)
        if len(heavy[b]):
            pos = torch.as_tensor(heavy[b], device=device, dtype=torch.long)
            row[pos] += w.heavy_gain * qhat[b]
        if w.recent > 0:
            L_b = int(lens[b])
            row[L_b - w.recent:L_b] += w.recent_gain * qhat[b]
        K_r[b] = row.to(torch.bfloat16)
        del row

    q = torch.randn((w.n_layers, w.B, w.H_q, w.d), generator=_gen(device, seed, "q"),
                    device=device, dtype=torch.float32).to(torch.bfloat16)
    out = {
        "q_r": q_r, "K_r": K_r,
        "seq_lens": torch.as_tensor(lens, dtype=torch.int32, device=device),
        "ks": torch.as_tensor(ks, dtype=torch.int32, device=device),
        "q": q, "heavy": heavy,
    }
    if with_kv:
        rng_layers = layers if layers is not None else range(w.n_layers)
        shape = (len(rng_layers), w.B, w.L_cap, w.H_kv, w.d)
        K = torch.empty(shape, dtype=torch.bfloat16, device=device)
        V = torch.empty(shape, dtype=torch.bfloat16, device=device)
        for i, layer in enumerate(rng_layers):
            K[i].normal_(generator=_gen(device, seed, f"K.{layer}"))
            V[i].normal_(generator=_gen(device, seed, f"V.{layer}"))
        out["K"], out["V"] = K, V
    return out


def elastic_sequence(w: Workload, x: dict, seed: int = 0, device=None):
    """Per-step inputs of a run of `w.steps` decode steps on the inputs `x`
    drawn by `generate` (one appended token per step).

    Step s sees seq_lens + s tokens: the rows past the initial lengths were
    drawn N(0,1) and unplanted by `generate`, so appending a token only moves
    the length.  The retrieval query drifts as an AR(1) process,
    q_r(s+1) = drift * q_r(s) + sqrt(1 - drift^2) * xi_s with xi_s ~ N(0,1),
    carried in fp32 and rounded to bf16 per step; the LLM queries are fresh
    N(0,1) draws each step.  The budgets stay those of the initial lengths.

    Returns q_r [S, B, H_r, d_r] bf16, q [S, n_layers, B, H_q, d] bf16 and
    seq_lens [S, B] int32 (S = w.steps).
    """
    device = torch.device(device if device is not None else x["q_r"].device)
    S = w.steps
    lens0 = x["seq_lens"].to(device=device, dtype=torch.int64)
    if int((lens0 + S - 1).max()) > w.L_cap:
        raise ValueError("the appended tokens do not fit the capacity")
    qr = x["q_r"].to(device).float()
    c = float(np.sqrt(1.0 - w.drift * w.drift))
    q_r_steps = torch.empty((S,) + tuple(qr.shape), dtype=torch.bfloat16, device=device)
    q_steps = torch.empty((S, w.n_layers, w.B, w.H_q, w.d), dtype=torch.bfloat16, device=device)
    for s in range(S):
        if s > 0:
            xi = torch.randn(qr.shape, generator=_gen(device, seed, f"q_r.drift.{s}"),
                             device=device, dtype=torch.float32)
            qr = w.drift * qr + c * xi
        q_r_steps[s] = qr.to(torch.bfloat16)
        q_steps[s] = torch.randn((w.n_layers, w.B, w.H_q, w.d),
                                 generator=_gen(device, seed, f"q.step.{s}"), device=device,
                                 dtype=torch.float32).to(torch.bfloat16)
    lens = (lens0[None, :] + torch.arange(S, device=device)[:, None]).to(torch.int32)
    return {"q_r": q_r_steps, "q": q_steps, "seq_lens": lens}


def frontend_inputs(w: Workload, seq_lens, seed: int = 0, device="cpu", vocab=None):
    """Inputs of the retrieval head's front end for the new token of every
    sequence: token ids uniform over the vocabulary (numpy PCG64), the
    embedding table N(0,1), the Q/K projection weights N(0, 1/hidden) (so
    that the projected vectors have unit variance), all rounded to bf16, and
    each new token's position = seq_lens - 1 (its key is the last cached row).
    `vocab` overrides the workload's (tests use small tables).

    Returns tokens [B] int32, pos [B] int32, emb [vocab, hidden],
    w_q, w_k [H_r * d_r, hidden] (bf16).
    """
    device = torch.device(device)
    V = int(vocab) if vocab is not None else w.vocab
    rng = np.random.default_rng(tensor_seed(seed, "tokens"))
    tokens = rng.integers(0, V, size=w.B)
    emb = torch.empty((V, w.hidden), dtype=torch.bfloat16, device=device)
    step = max(1, (1 << 26) // w.hidden)            # rows per fp32 chunk (256 MiB)
    g = _gen(device, seed, "emb")
    for r0 in range(0, V, step):
        r1 = min(V, r0 + step)
        emb[r0:r1] = torch.randn((r1 - r0, w.hidden), generator=g, device=device,
                                 dtype=torch.float32).to(torch.bfloat16)
    sd = 1.0 / float(np.sqrt(w.hidden))
    wq = (torch.randn((w.H_r * w.d_r, w.hidden), generator=_gen(device, seed, "w_q"),
                      device=device, dtype=torch.float32) * sd).to(torch.bfloat16)
    wk = (torch.randn((w.H_r * w.d_r, w.hidden), generator=_gen(device, seed, "w_k"),
                      device=device, dtype=torch.float32) * sd).to(torch.bfloat16)
    lens = torch.as_tensor(seq_lens).to(device=device, dtype=torch.int64)
    return {"tokens": torch.as_tensor(tokens, dtype=torch.int32, device=device),
            "pos": (lens - 1).to(torch.int32), "emb": emb, "w_q": wq, "w_k": wk}


def frontend_bytes(w: Workload) -> int:
    """Bytes the front end must move: both projection matrices, one
    embedding row per sequence, and q_r and the new K_r row written."""
    return (2 * w.H_r * w.d_r * w.hidden * 2 + w.B * w.hidden * 2
            + 2 * w.B * w.H_r * w.d_r * 2)


def generate_mla(w: Workload, seed: int = 0, device="cpu", layers: Optional[range] = None):
    """Inputs of an MLA decode step: the retrieval inputs of `generate`
    (q_r, K_r, seq_lens, ks, heavy; same seeds) and, per layer, the queries
    q_mla [n_layers, B, H, d_nope + d_rope] N(0,1), the latent cache ckv
    [n_layers, B, L_cap, d_c + d_rope] N(0,1) (the latent after its RMS norm,
    then the rotary key), and the up-projections w_uk [n_layers, H, d_nope,
    d_c], w_uv [n_layers, H, d_v, d_c] N(0, 1/d_c); all bf16."""
    device = torch.device(device)
    x = generate(w, seed=seed, device=device, with_kv=False)
    del x["q"]
    rng_layers = layers if layers is not None else range(w.n_layers)
    nl = len(rng_layers)
    dk = w.d_c + w.d_rope
    sd = 1.0 / float(np.sqrt(w.d_c))
    q = torch.empty((nl, w.B, w.H_q, w.d_nope + w.d_rope), dtype=torch.bfloat16, device=device)
    ckv = torch.empty((nl, w.B, w.L_cap, dk), dtype=torch.bfloat16, device=device)
    w_uk = torch.empty((nl, w.H_q, w.d_nope, w.d_c), dtype=torch.bfloat16, device=device)
    w_uv = torch.empty((nl, w.H_q, w.d_v, w.d_c), dtype=torch.bfloat16, device=device)
    for i, layer in enumerate(rng_layers):
        q[i] = torch.randn(q.shape[1:], generator=_gen(device, seed, f"mla.q.{layer}"),
                           device=device, dtype=torch.float32).to(torch.bfloat16)
        for b in range(w.B):
            ckv[i, b] = torch.randn((w.L_cap, dk), generator=_gen(device, seed, f"mla.ckv.{layer}.{b}"),
                                    device=device, dtype=torch.float32).to(torch.bfloat16)
        w_uk[i] = (torch.randn(w_uk.shape[1:], generator=_gen(device, seed, f"mla.w_uk.{layer}"),
                               device=device, dtype=torch.float32) * sd).to(torch.bfloat16)
        w_uv[i] = (torch.randn(w_uv.shape[1:], generator=_gen(device, seed, f"mla.w_uv.{layer}"),
                               device=device, dtype=torch.float32) * sd).to(torch.bfloat16)
    x.update({"q_mla": q, "ckv": ckv, "w_uk": w_uk, "w_uv": w_uv})
    return x


def mla_attn_bytes(w: Workload, seq_lens, ks) -> int:
    """Bytes an MLA sparse attention must move: every selected latent row of
    every layer, the queries and up-projection weights of every layer, and
    the fp32 outputs."""
    kb = sum(min(int(k), int(L)) for k, L in zip(ks, seq_lens))
    dk = w.d_c + w.d_rope
    per_layer = (kb * dk * 2 + w.B * w.H_q * (w.d_nope + w.d_rope) * 2
                 + w.H_q * (w.d_nope + w.d_v) * w.d_c * 2 + w.B * w.H_q * w.d_v * 4)
    return w.n_layers * per_layer


def mla_bytes(w: Workload, seq_lens, ks) -> int:
    """Bytes of an MLA decode step: the retrieval head's K_r rows and q_r,
    then the MLA sparse attention."""
    kr = sum(int(L) for L in seq_lens) * w.H_r * w.d_r * 2 + w.B * w.H_r * w.d_r * 2
    return kr + mla_attn_bytes(w, seq_lens, ks)


def algorithmic_bytes(w: Workload, seq_lens, ks, delta_rows: int = 0) -> int:
    """Bytes the method must move for one decode step.

    K_r rows of every cached token, q_r, and per layer the selected K and V
    rows, the query and the fp32 output; plus, for elastic loading, a write
    of every changed K/V row in every layer into its slot (delta_rows =
    total changed indices over the batch; the changed rows are among the
    selected rows, read once).  Scratch (logits, scores, indices, partials)
    is implementation traffic and is not counted.
    """
    seq_lens = [int(x) for x in seq_lens]
    ks = [int(x) for x in ks]
    kb = [min(k, L) for k, L in zip(ks, seq_lens)]
    kr = sum(seq_lens) * w.H_r * w.d_r * 2 + w.B * w.H_r * w.d_r * 2
    per_layer = (sum(kb) * w.H_kv * w.d * 2 * 2 + w.B * w.H_q * w.d * 2
                 + w.B * w.H_q * w.d * 4)
    delta = delta_rows * w.H_kv * w.d * 2 * 2 * w.n_layers
    return kr + w.n_layers * per_layer + delta
