"""Plain fp64 CPU oracle of the SpeContext per-decode-step hot path.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct
definition that the HIP path is checked against.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product library never does, and nothing here is shared with the HIP sources.

What it computes (SpeContext, arXiv 2512.00722):

* retrieval scoring (Sec. 4.3 "Implementation Details", Eq. 1): the
  lightweight retrieval head keeps a full key cache K_r and, for the current
  query q_r, forms attention weights softmax(q_r K_r^T / sqrt(d_r)) per head;
  the per-head weights are summed over heads into one importance score per
  cached token (batch-level mapping of Sec. 4.2: one token set shared by every
  head and, per Sec. 7.2.1, by every layer);
* token selection (Sec. 4.3): the k tokens with the largest score;
* sparse attention (Sec. 4.3 "Support for MHA" / "Support for GQA", Eq. 1):
  the LLM's K/V rows at the selected indices are gathered per KV head and
  decode attention runs over them only; the G = H_q / H_kv query heads of a
  group share one KV head;
* elastic loading (Sec. 5.4): with S_last the set held on the device and
  S_now the new selection, only S_now - S_last is loaded, into the places freed
  by S_last - S_now (equal in size because the budget is fixed);
* the retrieval head's front end (Sec. 4.3): the new token's embedding row,
  the Q/K projection and the rotary embedding with YaRN scaling (Peng et al.)
  that extends the distilled model's 2K context;
* MLA (Sec. 4.3 "Support for MLA"): the cache holds a latent per token and
  only the selected latents are raised to per-head keys and values.

Everything is computed in float64 from the bf16-rounded inputs (bf16 embeds
exactly in float64).  Readings of points the paper leaves open:

* scale: Eq. 1 divides by sqrt(d) without naming d; the retrieval head uses
  1/sqrt(d_r) and the LLM attention 1/sqrt(d) (head dimensions);
* k_b = min(k, L_b): a budget above the context takes every token, so sparse
  attention with k = L_b is dense attention;
* ties: equal scores are ordered by lower token index; the returned index set
  is sorted ascending (attention is permutation invariant, so order only
  fixes the rounding order);
* no token is forced into the set (no sink or recent window: those are prior
  work in Sec. 2.2, not the method);
* the slot pairing of elastic loading (which freed slot receives which new
  token) is not stated; the oracle pairs the i-th smallest freed slot with the
  i-th smallest new token.  Only the resulting slot->token map is compared.
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "retrieval_logits",
    "head_softmax",
    "head_sum",
    "retrieval_scores",
    "topk_indices",
    "group_max_scores",
    "head_level_scores",
    "sparse_gqa_attention",
    "sparse_gqa_attention_sets",
    "dense_gqa_attention",
    "elastic_update",
    "decode_step",
    "accept_index_set",
    "bf16_to_f64",
    "yarn_frequencies",
    "rope_rotate",
    "retrieval_qk",
    "mla_sparse_attention",
]


def bf16_to_f64(x_u16: np.ndarray) -> np.ndarray:
    """Decode raw bf16 bit patterns (uint16) to float64 exactly.

    bf16 is the upper half of an IEEE binary32, so shifting the 16 bits into
    the high half of a uint32 gives the float32 with the same value.
    """
    u = np.asarray(x_u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Retrieval head (Sec. 4.3, Eq. 1)
# ---------------------------------------------------------------------------

def retrieval_logits(q_r: np.ndarray, K_r: np.ndarray, L: int,
                     scale: float | None = None) -> np.ndarray:
    """Per-head attention logits of the retrieval head, Eq. 1 before softmax.

    q_r: [H_r, d_r] query of the current token for each retrieval head.
    K_r: [L_cap, H_r, d_r] full retrieval key cache (token-major).
    L:   number of cached tokens (only t < L are scored).
    Returns logits l[h, t] = (q_r[h] . K_r[t, h]) * scale, shape [H_r, L].
    """
    q_r = np.asarray(q_r, dtype=np.float64)
    K_r = np.asarray(K_r, dtype=np.float64)
    H_r, d_r = q_r.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d_r)
    out = np.empty((H_r, L), dtype=np.float64)
    for h in range(H_r):
        # one matrix-vector product per head: K_r[:L, h, :] @ q_r[h]
        out[h] = (K_r[:L, h, :] @ q_r[h]) * scale
    return out


def head_softmax(logits: np.ndarray) -> np.ndarray:
    """Softmax over the token axis, separately for each head (Eq. 1).

    In decode every cached token precedes the query, so no causal mask is
    applied beyond the context length.  The maximum is subtracted first so
    that exp never overflows; this does not change the result.
    """
    logits = np.asarray(logits, dtype=np.float64)
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    return e / e.sum(axis=1, keepdims=True)


def head_sum(p: np.ndarray) -> np.ndarray:
    """Importance score of each token: the per-head weights summed over heads."""
    return np.asarray(p, dtype=np.float64).sum(axis=0)


def retrieval_scores(q_r, K_r, L: int, scale: float | None = None) -> np.ndarray:
    """score[t] for t < L: softmax per retrieval head, then sum over heads."""
    if L == 0:
        return np.zeros((0,), dtype=np.float64)
    return head_sum(head_softmax(retrieval_logits(q_r, K_r, L, scale)))


def group_max_scores(p: np.ndarray, n_groups: int) -> np.ndarray:
    """GQA group-level weights (Sec. 4.3 "Support for GQA").

    The heads of each group are reduced by an element-wise maximum, per
    token, giving one weight row per group.  p: [H, L] -> [n_groups, L], with
    group g holding heads g*H/n_groups ... (g+1)*H/n_groups - 1.  This is the
    head-level selection the paper prefers; the decode step below uses the
    summed (batch-level) score instead.
    """
    p = np.asarray(p, dtype=np.float64)
    H = p.shape[0]
    assert H % n_groups == 0
    per = H // n_groups
    return np.stack([p[g * per:(g + 1) * per].max(axis=0) for g in range(n_groups)])


def head_level_scores(q_r, K_r, L: int, n_sets: int, scale: float | None = None) -> np.ndarray:
    """Head-level importance (Sec. 4.2 head-level mapping; Sec. 4.3 "Support
    for GQA"): the per-head softmax weights of the retrieval head, reduced by
    an element-wise maximum within each group of heads that shares one KV
    head.  Returns [n_sets, L]: one row of weights per KV head, from which
    that KV head's tokens are chosen.
    """
    H_r = np.asarray(q_r).shape[0]
    if L == 0:
        return np.zeros((n_sets, 0), dtype=np.float64)
    assert H_r % n_sets == 0
    return group_max_scores(head_softmax(retrieval_logits(q_r, K_r, L, scale)), n_sets)


# ---------------------------------------------------------------------------
# Token selection
# ---------------------------------------------------------------------------

def topk_indices(score: np.ndarray, k: int) -> np.ndarray:
    """The min(k, L) tokens with the largest score, ascending by token index.

    Order by descending score, equal scores by ascending token index, keep
    the first k_b, and return them sorted by token index.
    """
    score = np.asarray(score)
    L = score.shape[0]
    kb = max(0, min(int(k), L))
    t = np.arange(L)
    # np.lexsort sorts by the last key first: primary -score, secondary t.
    order = np.lexsort((t, -score))
    return np.sort(order[:kb]).astype(np.int64)


# ---------------------------------------------------------------------------
# Sparse GQA decode attention (Eq. 1 over the selected rows)
# ---------------------------------------------------------------------------

def sparse_gqa_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray,
                         idx: np.ndarray, scale: float | None = None):
    """Decode attention of one sequence and one layer over selected tokens.

    q: [H_q, d] query; K, V: [L_cap, H_kv, d] layer KV cache (token-major).
    idx: selected token indices (any order, distinct).
    Query head h reads KV head g = h // G with G = H_q / H_kv (the heads of
    one group share a KV head; G = 1 is MHA, H_kv = 1 is MQA).
    Returns (out [H_q, d], lse [H_q]) with lse = log sum_j exp(s_j) of the
    scaled logits; with no selected token out is 0 and lse is -inf.
    """
    q = np.asarray(q, dtype=np.float64)
    H_q, d = q.shape
    H_kv = K.shape[1]
    assert H_q % H_kv == 0
    G = H_q // H_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    idx = np.asarray(idx, dtype=np.int64)
    out = np.zeros((H_q, d), dtype=np.float64)
    lse = np.full((H_q,), -np.inf, dtype=np.float64)
    if idx.size == 0:
        return out, lse
    Ks = np.asarray(K[idx], dtype=np.float64)  # [k, H_kv, d]   (gather)
    Vs = np.asarray(V[idx], dtype=np.float64)
    for h in range(H_q):
        g = h // G
        s = (Ks[:, g, :] @ q[h]) * scale       # [k]
        m = s.max()
        w = np.exp(s - m)
        z = w.sum()
        out[h] = (w / z) @ Vs[:, g, :]
        lse[h] = m + math.log(z)
    return out, lse


def sparse_gqa_attention_sets(q: np.ndarray, K: np.ndarray, V: np.ndarray, idx_sets,
                              scale: float | None = None):
    """Decode attention with one token set per KV head (head-level selection,
    Sec. 4.3): the query heads of group g attend over KV head g's rows at
    idx_sets[g] only.  Same shapes and returns as sparse_gqa_attention.
    """
    q = np.asarray(q, dtype=np.float64)
    H_q, d = q.shape
    H_kv = K.shape[1]
    assert len(idx_sets) == H_kv and H_q % H_kv == 0
    G = H_q // H_kv
    out = np.zeros((H_q, d), dtype=np.float64)
    lse = np.full((H_q,), -np.inf, dtype=np.float64)
    for g in range(H_kv):
        # group g alone, as an MHA/GQA problem with one KV head
        o, l_ = sparse_gqa_attention(q[g * G:(g + 1) * G], K[:, g:g + 1], V[:, g:g + 1],
                                     idx_sets[g], scale)
        out[g * G:(g + 1) * G] = o
        lse[g * G:(g + 1) * G] = l_
    return out, lse


def dense_gqa_attention(q, K, V, L: int, scale: float | None = None):
    """Dense decode attention over all L cached tokens (for the k = L pin)."""
    return sparse_gqa_attention(q, K, V, np.arange(L), scale)


# ---------------------------------------------------------------------------
# The retrieval head's front end for the new token (Sec. 4.3 "Implementation
# Details": the head keeps the draft model's embedding and Q/K projection
# weights and extends its context with YaRN)
# ---------------------------------------------------------------------------

def mla_sparse_attention(q_nope: np.ndarray, q_rope: np.ndarray, c: np.ndarray,
                         k_rope: np.ndarray, w_uk: np.ndarray, w_uv: np.ndarray,
                         idx: np.ndarray, scale: float | None = None):
    """Decode attention of one sequence and one layer of an MLA model over
    the selected tokens (Sec. 4.3, "Support for MLA").

    The cache holds, per token, the latent c_t [d_c] and the rotary key
    k_rope_t [d_rope] that all heads share.  Only the selected latents are
    raised to per-head keys and values:
        key of head h at token j   = [W_UK[h] c_j ; k_rope_j]     (d_nope + d_rope)
        value of head h at token j = W_UV[h] c_j                  (d_v)
    and head h attends over them as in Eq. 1, its query being
    [q_nope[h] ; q_rope[h]] and the scale 1/sqrt(d_nope + d_rope).

    q_nope [H, d_nope], q_rope [H, d_rope]; c [L_cap, d_c]; k_rope
    [L_cap, d_rope]; w_uk [H, d_nope, d_c], w_uv [H, d_v, d_c] (each maps a
    latent to one head's part, as a linear layer stores [out, in]).
    Returns (out [H, d_v], lse [H]); with no selected token out is 0 and lse
    is -inf.
    """
    q_nope = np.asarray(q_nope, dtype=np.float64)
    q_rope = np.asarray(q_rope, dtype=np.float64)
    H, d_nope = q_nope.shape
    d_rope = q_rope.shape[1]
    d_v = w_uv.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d_nope + d_rope)
    idx = np.asarray(idx, dtype=np.int64)
    out = np.zeros((H, d_v), dtype=np.float64)
    lse = np.full((H,), -np.inf, dtype=np.float64)
    if idx.size == 0:
        return out, lse
    cs = np.asarray(c[idx], dtype=np.float64)          # the selected latents only
    krs = np.asarray(k_rope[idx], dtype=np.float64)
    for h in range(H):
        k_nope = cs @ np.asarray(w_uk[h], dtype=np.float64).T   # [k, d_nope]
        v = cs @ np.asarray(w_uv[h], dtype=np.float64).T        # [k, d_v]
        s = (k_nope @ q_nope[h] + krs @ q_rope[h]) * scale
        m = s.max()
        w = np.exp(s - m)
        z = w.sum()
        out[h] = (w / z) @ v
        lse[h] = math.log(z) + m
    return out, lse


def yarn_frequencies(d_r: int, base: float, scale: float, orig_ctx: int,
                     alpha: float = 1.0, beta: float = 32.0):
    """Rotary frequencies of the d_r/2 dimension pairs after YaRN scaling
    (Peng et al., YaRN: the published method, written out here), and the
    magnitude factor applied to q and k.

    theta_i = base^(-2i/d_r).  A pair whose wavelength 2*pi/theta_i fits r_i =
    orig_ctx * theta_i / (2*pi) times into the original context is
    interpolated by gamma(r_i): gamma = 0 below alpha (the frequency is
    divided by `scale`), 1 above beta (kept), linear in between:
        theta'_i = (1 - gamma) * theta_i / scale + gamma * theta_i.
    Both q and k are multiplied by m = 0.1 * ln(scale) + 1 (so that the
    logits carry m^2); scale <= 1 leaves the frequencies and m = 1 unchanged.
    Returns (theta' [d_r/2], m).
    """
    i = np.arange(d_r // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / d_r)
    if scale <= 1.0:
        return theta, 1.0
    r = orig_ctx * theta / (2.0 * math.pi)
    gamma = np.clip((r - alpha) / (beta - alpha), 0.0, 1.0)
    theta_s = (1.0 - gamma) * theta / scale + gamma * theta
    return theta_s, 0.1 * math.log(scale) + 1.0


def rope_rotate(v: np.ndarray, pos: int, theta: np.ndarray, m: float = 1.0) -> np.ndarray:
    """Rotate one head vector v [d_r] to position `pos`: dimension pair
    (i, i + d_r/2) turns by the angle pos * theta[i] (the half-split pairing),
    and the result is scaled by m."""
    v = np.asarray(v, dtype=np.float64)
    h = v.shape[-1] // 2
    ang = pos * np.asarray(theta, dtype=np.float64)
    c, s_ = np.cos(ang), np.sin(ang)
    x, y = v[..., :h], v[..., h:]
    return m * np.concatenate([x * c - y * s_, x * s_ + y * c], axis=-1)


def retrieval_qk(token: int, pos: int, emb: np.ndarray, w_q: np.ndarray, w_k: np.ndarray,
                 H_r: int, theta: np.ndarray, m: float):
    """The new token's retrieval query and key: its embedding row, the Q and
    K projections (no bias; weights [H_r*d_r, hidden] as a linear layer
    stores them), then each head's vector rotated to position `pos`.
    Returns (q_r [H_r, d_r], k_r [H_r, d_r]); k_r is what the token appends
    to the retrieval key cache."""
    x = np.asarray(emb[token], dtype=np.float64)
    q = (np.asarray(w_q, dtype=np.float64) @ x).reshape(H_r, -1)
    k = (np.asarray(w_k, dtype=np.float64) @ x).reshape(H_r, -1)
    return (np.stack([rope_rotate(q[h], pos, theta, m) for h in range(H_r)]),
            np.stack([rope_rotate(k[h], pos, theta, m) for h in range(H_r)]))


# ---------------------------------------------------------------------------
# Elastic loading (Sec. 5.4)
# ---------------------------------------------------------------------------

def elastic_update(slot_tok: np.ndarray, s_now: np.ndarray):
    """One elastic-loading update of a fixed-budget slot array.

    slot_tok: [n_slots] token held by each device slot (-1 = empty); its
              valid entries form S_last.
    s_now:    the new selection S_now (distinct tokens), |S_now| <= n_slots.
    Slots whose token is not in S_now are freed (S_last - S_now, plus empty
    slots); the tokens S_now - S_last are loaded into freed slots, the i-th
    smallest freed slot receiving the i-th smallest new token.  Slots beyond
    |S_now| that stay free are marked -1 so that the slot multiset is S_now.

    Returns (new_slot_tok, loads) where loads is a list of (slot, token)
    copies in slot order.  With a fixed budget, |S_last - S_now| equals
    |S_now - S_last| whenever |S_last| = |S_now|.
    """
    slot_tok = np.asarray(slot_tok, dtype=np.int64).copy()
    now = set(int(t) for t in np.asarray(s_now).tolist())
    held = set(int(t) for t in slot_tok.tolist() if t >= 0)
    d_in = sorted(now - held)                    # S_now - S_last
    free = [i for i, t in enumerate(slot_tok.tolist()) if t < 0 or t not in now]
    assert len(free) >= len(d_in)
    loads = list(zip(free[:len(d_in)], d_in))
    for slot, tok in loads:
        slot_tok[slot] = tok
    for slot in free[len(d_in):]:
        slot_tok[slot] = -1
    return slot_tok, loads


# ---------------------------------------------------------------------------
# One decode step (batched), and the acceptance predicate
# ---------------------------------------------------------------------------

def decode_step(q_r, K_r, seq_lens, ks, q, K_layers, V_layers,
                scale_r: float | None = None, scale: float | None = None):
    """Retrieve + select + sparse attention for every sequence and layer.

    q_r [B, H_r, d_r]; K_r [B, L_cap, H_r, d_r]; seq_lens [B]; ks [B];
    q [n_layers, B, H_q, d]; K_layers/V_layers [n_layers, B, L_cap, H_kv, d].
    One selection per sequence serves every layer and every KV head.
    Returns (idx list of arrays, scores list, out [n_layers, B, H_q, d],
    lse [n_layers, B, H_q]).
    """
    B = len(seq_lens)
    n_layers = len(q)
    H_q, d = np.asarray(q[0][0]).shape
    idxs, scores = [], []
    out = np.zeros((n_layers, B, H_q, d))
    lse = np.full((n_layers, B, H_q), -np.inf)
    for b in range(B):
        L = int(seq_lens[b])
        s = retrieval_scores(q_r[b], K_r[b], L, scale_r)
        idx = topk_indices(s, int(ks[b]))
        idxs.append(idx)
        scores.append(s)
        for layer in range(n_layers):
            o, l_ = sparse_gqa_attention(q[layer][b], K_layers[layer][b],
                                         V_layers[layer][b], idx, scale)
            out[layer, b] = o
            lse[layer, b] = l_
    return idxs, scores, out, lse


def accept_index_set(score: np.ndarray, k: int, cand: np.ndarray,
                     band: float = 1e-6):
    """Is `cand` an acceptable top-k set for the oracle scores `score`?

    Let s_k be the k_b-th largest oracle score.  The candidate must hold k_b
    distinct in-range tokens, contain every token scoring above s_k + band,
    and hold no token scoring below s_k - band.  Outside the band around the
    k-th score the set is therefore unique; inside it any choice is allowed
    (the oracle itself breaks exact ties by lower index).
    Returns (ok, info) where info reports the band population and the
    symmetric difference to the oracle's own set.
    """
    score = np.asarray(score, dtype=np.float64)
    L = score.shape[0]
    kb = max(0, min(int(k), L))
    cand = np.asarray(cand, dtype=np.int64)
    ref = topk_indices(score, kb)
    info = {"k_b": kb, "band_pop": 0, "sym_diff": 0, "reason": ""}
    if cand.shape[0] != kb:
        info["reason"] = f"size {cand.shape[0]} != {kb}"
        return False, info
    if kb == 0:
        return True, info
    if len(np.unique(cand)) != kb or cand.min() < 0 or cand.max() >= L:
        info["reason"] = "duplicate or out-of-range index"
        return False, info
    s_k = np.sort(score)[::-1][kb - 1]
    info["band_pop"] = int(np.sum(np.abs(score - s_k) <= band))
    info["sym_diff"] = int(len(set(cand.tolist()) ^ set(ref.tolist())))
    inset = np.zeros(L, dtype=bool)
    inset[cand] = True
    must = score > s_k + band
    if np.any(must & ~inset):
        info["reason"] = "missed a token above the band"
        return False, info
    if np.any(inset & (score < s_k - band)):
        info["reason"] = "took a token below the band"
        return False, info
    return True, info
