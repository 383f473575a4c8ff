"""SpeContext decode-step hot path on MI355X: thin Python binding of libspecctx.

Every step runs in the HIP kernels of libspecctx.so (gfx950); this module
only marshals torch tensors (device memory, the current HIP stream) into the
C ABI declared in include/spec.h.  There is no fallback: if the library is
missing, importing the ops raises.

    import paper_2512_00722_amd as spec
    scores = spec.score(q_r, K_r, seq_lens)
    idx, counts = spec.topk(scores, seq_lens, ks, k_max)
    out, lse = spec.sparse_decode_attn(q, K, V, counts, idx=idx)
    res = spec.step(q_r, K_r, seq_lens, ks, q, K, V, k_max)
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = [
    "SpecError", "load_library", "lib_path", "Dims", "workspace_size", "score", "topk",
    "gather", "sparse_decode_attn", "delta_gather", "ElasticState", "step", "step_noalloc",
    "step_noalloc_max_bytes", "Frontend",
    "retrieval_qk", "MlaDims", "mla_workspace_size", "mla_sparse_decode_attn",
    "OP_SCORE", "OP_TOPK", "OP_GATHER", "OP_ATTN", "OP_DELTA", "OP_STEP", "OP_FRONTEND",
    "OP_OFFLOAD", "HostKv", "OffloadEvents", "offload_load", "step_offload",
    "EXPORTED_SYMBOLS",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
lib_path = os.path.join(_PKG, "libspecctx.so")

OP_SCORE, OP_TOPK, OP_GATHER, OP_ATTN, OP_DELTA, OP_STEP, OP_FRONTEND, OP_OFFLOAD = range(8)
STATUS = {0: "SPEC_OK", 1: "SPEC_ERR_INVALID", 2: "SPEC_ERR_UNSUPPORTED",
          3: "SPEC_ERR_WORKSPACE", 4: "SPEC_ERR_HIP", 5: "SPEC_ERR_TOO_LARGE"}

EXPORTED_SYMBOLS = ["spec_score", "spec_topk", "spec_gather", "spec_sparse_decode_attn",
                    "spec_sparse_decode_attn_elastic", "spec_delta_gather", "spec_step", "spec_step_noalloc",
                    "spec_step_noalloc_max_bytes", "spec_offload_load", "spec_step_offload",
                    "spec_retrieval_qk",
                    "spec_mla_sparse_decode_attn", "spec_mla_workspace_size", "spec_workspace_size",
                    "spec_status_string", "spec_last_hip_error", "spec_version"]


class SpecError(RuntimeError):
    def __init__(self, status: int, where: str, lib=None):
        self.status = status
        msg = STATUS.get(status, str(status))
        if lib is not None:
            msg += ": " + lib.spec_status_string(status).decode()
            if status == 4:
                msg += f" (hip error {lib.spec_last_hip_error()})"
        super().__init__(f"{where}: {msg}")


class Dims(ctypes.Structure):
    """Mirror of `spec_dims` (include/spec.h)."""
    _fields_ = [
        ("B", ctypes.c_int32), ("L_cap", ctypes.c_int32), ("L_max", ctypes.c_int32),
        ("k_max", ctypes.c_int32), ("H_r", ctypes.c_int32), ("d_r", ctypes.c_int32),
        ("n_layers", ctypes.c_int32), ("H_q", ctypes.c_int32), ("H_kv", ctypes.c_int32),
        ("d", ctypes.c_int32),
        ("kr_stride_b", ctypes.c_int64), ("kv_stride_layer", ctypes.c_int64),
        ("kv_stride_b", ctypes.c_int64),
        ("scale_r", ctypes.c_float), ("scale", ctypes.c_float),
        ("n_sets", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]

    @classmethod
    def make(cls, B, L_cap, L_max, k_max, H_r=8, d_r=64, n_layers=1, H_q=8, H_kv=8, d=128,
             kr_stride_b=0, kv_stride_layer=0, kv_stride_b=0, scale_r=0.0, scale=0.0,
             n_sets=1):
        return cls(B, L_cap, L_max, k_max, H_r, d_r, n_layers, H_q, H_kv, d, kr_stride_b,
                   kv_stride_layer, kv_stride_b, scale_r, scale, n_sets, 0)


class Elastic(ctypes.Structure):
    """Mirror of `spec_elastic`."""
    _fields_ = [("slot_tok", ctypes.c_void_p), ("kbuf", ctypes.c_void_p),
                ("vbuf", ctypes.c_void_p), ("n_changed", ctypes.c_void_p),
                ("slot_src", ctypes.c_void_p)]


class HostKv(ctypes.Structure):
    """Mirror of `spec_host_kv`."""
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("stride_layer", ctypes.c_int64), ("stride_b", ctypes.c_int64)]


class Frontend(ctypes.Structure):
    """Mirror of `spec_frontend`."""
    _fields_ = [("vocab", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("rope_base", ctypes.c_float), ("yarn_scale", ctypes.c_float),
                ("yarn_orig_ctx", ctypes.c_int32), ("yarn_alpha", ctypes.c_float),
                ("yarn_beta", ctypes.c_float), ("reserved", ctypes.c_int32)]


class MlaDims(ctypes.Structure):
    """Mirror of `spec_mla_dims`."""
    _fields_ = [("B", ctypes.c_int32), ("L_cap", ctypes.c_int32), ("k_max", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("H", ctypes.c_int32), ("d_c", ctypes.c_int32),
                ("d_rope", ctypes.c_int32), ("d_nope", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("ckv_stride_layer", ctypes.c_int64),
                ("ckv_stride_b", ctypes.c_int64), ("scale", ctypes.c_float),
                ("reserved2", ctypes.c_int32)]

    @classmethod
    def make(cls, B, L_cap, k_max, n_layers, H, d_c=512, d_rope=64, d_nope=128, d_v=128,
             ckv_stride_layer=0, ckv_stride_b=0, scale=0.0):
        return cls(B, L_cap, k_max, n_layers, H, d_c, d_rope, d_nope, d_v, 0, ckv_stride_layer,
                   ckv_stride_b, scale, 0)


_lib = None


def load_library(path: Optional[str] = None):
    """Load libspecctx.so (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or lib_path
    if not os.path.exists(p):
        raise ImportError(f"{p} not found: build it with `python -m paper_2512_00722_amd.build` "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(p)
    P, I, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    D = ctypes.POINTER(Dims)
    E = ctypes.POINTER(Elastic)
    F = ctypes.POINTER(Frontend)
    M = ctypes.POINTER(MlaDims)
    sig = {
        "spec_score": [D, P, P, P, P, P, S, P],
        "spec_topk": [D, P, P, P, P, P, P, S, P],
        "spec_gather": [D, P, P, P, P, P, P, P],
        "spec_sparse_decode_attn": [D, P, P, P, P, P, P, P, P, S, P],
        "spec_sparse_decode_attn_elastic": [D, P, P, P, E, P, P, P, P, S, P],
        "spec_delta_gather": [D, P, P, P, P, E, P, S, P],
        "spec_step": [D, P, P, P, P, P, P, P, P, P, P, P, P, E, P, S, P],
        "spec_step_noalloc": [D, P, P, P, P, P, P, P, P, P, P, P, P, E, P],
        "spec_offload_load": [D, P, P, ctypes.POINTER(HostKv), E, P, S, P, P, P],
        "spec_step_offload": [D, P, P, P, P, P, P, P, ctypes.c_int32, ctypes.POINTER(HostKv),
                              P, P, P, P, P, E, P, S, P, P, P],
        "spec_retrieval_qk": [D, F, P, P, P, P, P, P, P, P, S, P],
        "spec_mla_sparse_decode_attn": [M, P, P, P, P, P, P, P, P, P, S, P],
        "spec_mla_workspace_size": [M, ctypes.POINTER(S)],
        "spec_workspace_size": [D, I, ctypes.POINTER(S)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.spec_status_string.argtypes = [ctypes.c_int]
    lib.spec_status_string.restype = ctypes.c_char_p
    lib.spec_last_hip_error.argtypes = []
    lib.spec_last_hip_error.restype = ctypes.c_int
    lib.spec_version.argtypes = []
    lib.spec_version.restype = ctypes.c_char_p
    lib.spec_step_noalloc_max_bytes.argtypes = []
    lib.spec_step_noalloc_max_bytes.restype = ctypes.c_size_t
    if path is None:
        _lib = lib
    return lib


# ------------------------------------------------------------------ helpers

def _check(st: int, where: str):
    if st != 0:
        raise SpecError(st, where, _lib)


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _need(t: torch.Tensor, name: str, dtype, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")


def _inner_contig(t: torch.Tensor, name: str, n_inner: int):
    """The last n_inner dims must be densely packed (row-major)."""
    exp = 1
    for dim in range(t.dim() - 1, t.dim() - 1 - n_inner, -1):
        if t.shape[dim] != 1 and t.stride(dim) != exp:
            raise ValueError(f"{name}: inner {n_inner} dims must be contiguous")
        exp *= t.shape[dim]


def _i32(t: torch.Tensor, name: str, n: int):
    _need(t, name, torch.int32, 1)
    if t.shape[0] != n or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous int32 [{n}] tensor")


def workspace_size(dims: Dims, op: int) -> int:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check(lib.spec_workspace_size(ctypes.byref(dims), op, ctypes.byref(n)), "spec_workspace_size")
    return int(n.value)


def _workspace(dims: Dims, op: int, device, ws: Optional[torch.Tensor]):
    need = workspace_size(dims, op)
    if ws is not None:
        if ws.numel() * ws.element_size() < need:
            raise ValueError(f"workspace too small: {need} bytes needed")
        return ws, need
    return torch.empty(max(need, 16), dtype=torch.uint8, device=device), need


def _dims_retrieval(K_r: torch.Tensor, L_max: int, k_max: int, scale_r: float, **llm):
    B, L_cap, H_r, d_r = K_r.shape
    base = dict(n_layers=1, H_q=1, H_kv=1, d=128)
    base.update(llm)
    return Dims.make(B=B, L_cap=L_cap, L_max=L_max, k_max=k_max, H_r=H_r, d_r=d_r,
                     kr_stride_b=K_r.stride(0), scale_r=scale_r, **base)


# ------------------------------------------------------------------ ops

def score(q_r: torch.Tensor, K_r: torch.Tensor, seq_lens: torch.Tensor,
          L_max: Optional[int] = None, scale_r: float = 0.0,
          out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
          n_sets: int = 1) -> torch.Tensor:
    """Retrieval scores fp32: softmax per head over the cached tokens of
    q_r.K_r^T * scale_r, then summed over heads ([B, L_max], n_sets = 1) or,
    with n_sets > 1 sets (one per KV head), the maximum over each group of
    H_r / n_sets heads ([B, n_sets, L_max]); -inf beyond seq_lens."""
    lib = load_library()
    _need(q_r, "q_r", torch.bfloat16, 3)
    _need(K_r, "K_r", torch.bfloat16, 4)
    B, L_cap, H_r, d_r = K_r.shape
    if tuple(q_r.shape) != (B, H_r, d_r) or not q_r.is_contiguous():
        raise ValueError("q_r must be contiguous [B, H_r, d_r]")
    _inner_contig(K_r, "K_r", 3)
    _i32(seq_lens, "seq_lens", B)
    L_max = L_cap if L_max is None else int(L_max)
    dims = _dims_retrieval(K_r, L_max, 1, scale_r, H_q=n_sets, H_kv=n_sets, n_sets=n_sets)
    ws, nws = _workspace(dims, OP_SCORE, K_r.device, ws)
    shape = (B, L_max) if n_sets == 1 else (B, n_sets, L_max)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=K_r.device)
    elif tuple(out.shape) != shape or not out.is_contiguous() or out.dtype != torch.float32:
        raise ValueError(f"out must be contiguous fp32 {shape}")
    _check(lib.spec_score(ctypes.byref(dims), _p(q_r), _p(K_r), _p(seq_lens), _p(out), _p(ws),
                          nws, _stream(K_r)), "spec_score")
    return out


def topk(scores: torch.Tensor, seq_lens: torch.Tensor, ks: torch.Tensor, k_max: int,
         idx: Optional[torch.Tensor] = None, counts: Optional[torch.Tensor] = None,
         ws: Optional[torch.Tensor] = None):
    """Exact top-k of each score row (ties to the lower index): scores
    [B, L_max] (one set per sequence) or [B, n_sets, L_max]; ascending
    indices of the same leading shape [.., k_max] int32 padded with -1, and
    counts [B] int32."""
    lib = load_library()
    if scores.dim() == 3:
        _need(scores, "scores", torch.float32, 3)
        B, n_sets, L_max = scores.shape
    else:
        _need(scores, "scores", torch.float32, 2)
        (B, L_max), n_sets = scores.shape, 1
    if not scores.is_contiguous():
        raise ValueError("scores must be contiguous")
    _i32(seq_lens, "seq_lens", B)
    _i32(ks, "ks", B)
    dims = Dims.make(B=B, L_cap=L_max, L_max=L_max, k_max=int(k_max), H_q=n_sets, H_kv=n_sets,
                     n_sets=n_sets)
    ws, nws = _workspace(dims, OP_TOPK, scores.device, ws)
    if idx is None:
        shape = (B, int(k_max)) if n_sets == 1 else (B, n_sets, int(k_max))
        idx = torch.empty(shape, dtype=torch.int32, device=scores.device)
    if counts is None:
        counts = torch.empty((B,), dtype=torch.int32, device=scores.device)
    _check(lib.spec_topk(ctypes.byref(dims), _p(scores), _p(seq_lens), _p(ks), _p(idx),
                         _p(counts), _p(ws), nws, _stream(scores)), "spec_topk")
    return idx, counts


def _dims_llm(q: torch.Tensor, K: torch.Tensor, k_max: int, scale: float, L_max=None, **extra):
    n_layers, B, L_cap, H_kv, d = K.shape
    _, _, H_q, _ = q.shape
    return Dims.make(B=B, L_cap=L_cap, L_max=L_cap if L_max is None else L_max, k_max=k_max,
                     n_layers=n_layers, H_q=H_q, H_kv=H_kv, d=d,
                     kv_stride_layer=K.stride(0), kv_stride_b=K.stride(1), scale=scale, **extra)


def _check_cache(K: torch.Tensor, V: torch.Tensor):
    _need(K, "K", torch.bfloat16, 5)
    _need(V, "V", torch.bfloat16, 5)
    if K.shape != V.shape or K.stride() != V.stride():
        raise ValueError("K and V must have the same shape and strides")
    _inner_contig(K, "K", 3)


def _sets_of(idx: torch.Tensor, H_kv: int) -> int:
    """Token sets per sequence of an index tensor: [B, k_max] -> 1,
    [B, H_kv, k_max] -> H_kv (one set per KV head)."""
    if idx.dim() == 3:
        _need(idx, "idx", torch.int32, 3)
        if idx.shape[1] != H_kv:
            raise ValueError("idx with one set per KV head must be [B, H_kv, k_max]")
        return H_kv
    _need(idx, "idx", torch.int32, 2)
    return 1


def gather(K: torch.Tensor, V: torch.Tensor, idx: torch.Tensor, counts: torch.Tensor,
           out: Optional[tuple] = None):
    """Materialised gather: (K_sel, V_sel) [n_layers, B, k_max, H_kv, d] with
    rows j < counts[b] = K/V[layer, b, idx[b, j]].  Rows beyond counts[b]
    are left as they are (zero when the outputs are allocated here); `out`
    takes preallocated contiguous outputs."""
    lib = load_library()
    _check_cache(K, V)
    n_layers, B, L_cap, H_kv, d = K.shape
    n_sets = _sets_of(idx, H_kv)
    k_max = idx.shape[-1]
    _i32(counts, "counts", B)
    dims = Dims.make(B=B, L_cap=L_cap, L_max=L_cap, k_max=k_max, n_layers=n_layers, H_q=H_kv,
                     H_kv=H_kv, d=d, kv_stride_layer=K.stride(0), kv_stride_b=K.stride(1),
                     n_sets=n_sets)
    if out is None:
        ks = torch.zeros((n_layers, B, k_max, H_kv, d), dtype=torch.bfloat16, device=K.device)
        vs = torch.zeros_like(ks)
    else:
        ks, vs = out
        for t, nm in ((ks, "K_sel"), (vs, "V_sel")):
            _need(t, nm, torch.bfloat16, 5)
            if tuple(t.shape) != (n_layers, B, k_max, H_kv, d) or not t.is_contiguous():
                raise ValueError(f"{nm} must be contiguous [n_layers, B, k_max, H_kv, d]")
    _check(lib.spec_gather(ctypes.byref(dims), _p(K), _p(V), _p(idx.contiguous()), _p(counts),
                           _p(ks), _p(vs), _stream(K)), "spec_gather")
    return ks, vs


def sparse_decode_attn(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, counts: torch.Tensor,
                       idx: Optional[torch.Tensor] = None, scale: float = 0.0,
                       out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                       with_lse: bool = True, ws: Optional[torch.Tensor] = None):
    """GQA decode attention over the selected rows.  Indexed mode (idx given):
    K/V are caches [n_layers, B, L_cap, H_kv, d].  Compact mode (idx None):
    K/V are [n_layers, B, k_max, H_kv, d] and rows [0, counts[b]) are used.
    Returns (out fp32 [n_layers, B, H_q, d], lse fp32 [n_layers, B, H_q] or None)."""
    lib = load_library()
    _need(q, "q", torch.bfloat16, 4)
    _check_cache(K, V)
    n_layers, B, L_cap, H_kv, d = K.shape
    if q.shape[0] != n_layers or q.shape[1] != B or q.shape[3] != d or not q.is_contiguous():
        raise ValueError("q must be contiguous [n_layers, B, H_q, d]")
    _i32(counts, "counts", B)
    if idx is not None:
        n_sets = _sets_of(idx, H_kv)
        idx = idx.contiguous()
        k_max = idx.shape[-1]
        dims = _dims_llm(q, K, k_max, scale, n_sets=n_sets)
    else:
        k_max = L_cap
        if not K.is_contiguous():
            raise ValueError("compact K/V must be contiguous")
        dims = _dims_llm(q, K, k_max, scale)
    ws, nws = _workspace(dims, OP_ATTN, q.device, ws)
    if out is None:
        out = torch.empty((n_layers, B, q.shape[2], d), dtype=torch.float32, device=q.device)
    if lse is None and with_lse:
        lse = torch.empty((n_layers, B, q.shape[2]), dtype=torch.float32, device=q.device)
    _check(lib.spec_sparse_decode_attn(ctypes.byref(dims), _p(q), _p(K), _p(V), _p(idx),
                                       _p(counts), _p(out), _p(lse), _p(ws), nws, _stream(q)),
           "spec_sparse_decode_attn")
    return out, lse


class ElasticState:
    """Device-resident elastic-loading state: the slot->token map (S_last) and
    the compact K/V rows it holds for every layer."""

    def __init__(self, n_layers: int, B: int, k_max: int, H_kv: int, d: int, device):
        self.slot_tok = torch.full((B, k_max), -1, dtype=torch.int32, device=device)
        self.kbuf = torch.zeros((n_layers, B, k_max, H_kv, d), dtype=torch.bfloat16, device=device)
        self.vbuf = torch.zeros_like(self.kbuf)
        self.n_changed = torch.zeros((B,), dtype=torch.int32, device=device)
        # per slot, the token the last update loaded into it (-1: kept or empty)
        self.slot_src = torch.full((B, k_max), -1, dtype=torch.int32, device=device)

    def reset(self):
        self.slot_tok.fill_(-1)

    def c_struct(self) -> Elastic:
        return Elastic(self.slot_tok.data_ptr(), self.kbuf.data_ptr(), self.vbuf.data_ptr(),
                       self.n_changed.data_ptr(), self.slot_src.data_ptr())


def sparse_decode_attn_elastic(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                               state: ElasticState, counts: torch.Tensor, scale: float = 0.0,
                               out: Optional[torch.Tensor] = None,
                               lse: Optional[torch.Tensor] = None, with_lse: bool = True,
                               ws: Optional[torch.Tensor] = None):
    """Attention over the slots of `state` after an update whose rows have
    not been copied: slots with state.slot_src >= 0 are read from the caches
    K/V [n_layers, B, L_cap, H_kv, d] at that token and written into the slot
    on the way; the others are read from the slot.  Returns (out, lse)."""
    lib = load_library()
    _need(q, "q", torch.bfloat16, 4)
    _check_cache(K, V)
    n_layers, B, L_cap, H_kv, d = K.shape
    if q.shape[0] != n_layers or q.shape[1] != B or q.shape[3] != d or not q.is_contiguous():
        raise ValueError("q must be contiguous [n_layers, B, H_q, d]")
    _i32(counts, "counts", B)
    k_max = state.slot_tok.shape[1]
    if tuple(state.kbuf.shape) != (n_layers, B, k_max, H_kv, d):
        raise ValueError("elastic state shape does not match")
    dims = _dims_llm(q, K, k_max, scale)
    ws, nws = _workspace(dims, OP_ATTN, q.device, ws)
    if out is None:
        out = torch.empty((n_layers, B, q.shape[2], d), dtype=torch.float32, device=q.device)
    if lse is None and with_lse:
        lse = torch.empty((n_layers, B, q.shape[2]), dtype=torch.float32, device=q.device)
    el = state.c_struct()
    _check(lib.spec_sparse_decode_attn_elastic(ctypes.byref(dims), _p(q), _p(K), _p(V),
                                               ctypes.byref(el), _p(counts), _p(out), _p(lse),
                                               _p(ws), nws, _stream(q)),
           "spec_sparse_decode_attn_elastic")
    return out, lse


def delta_gather(idx_now: torch.Tensor, counts: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                 state: ElasticState, L_max: Optional[int] = None,
                 ws: Optional[torch.Tensor] = None):
    """Elastic loading: copy only S_now - S_last rows into freed slots."""
    lib = load_library()
    _check_cache(K, V)
    n_layers, B, L_cap, H_kv, d = K.shape
    _need(idx_now, "idx_now", torch.int32, 2)
    k_max = idx_now.shape[1]
    _i32(counts, "counts", B)
    if tuple(state.kbuf.shape) != (n_layers, B, k_max, H_kv, d):
        raise ValueError("elastic state shape does not match")
    dims = Dims.make(B=B, L_cap=L_cap, L_max=L_cap if L_max is None else L_max, k_max=k_max,
                     n_layers=n_layers, H_q=H_kv, H_kv=H_kv, d=d,
                     kv_stride_layer=K.stride(0), kv_stride_b=K.stride(1))
    ws, nws = _workspace(dims, OP_DELTA, K.device, ws)
    el = state.c_struct()
    _check(lib.spec_delta_gather(ctypes.byref(dims), _p(idx_now.contiguous()), _p(counts),
                                 _p(K), _p(V), ctypes.byref(el), _p(ws), nws, _stream(K)),
           "spec_delta_gather")
    return state


def _step_args(q_r, K_r, seq_lens, ks, q, K, V, k_max, L_max, scale_r, scale, with_scores,
               with_lse, outputs, head_level):
    """Checks and dims of a fused step; the outputs dict (allocated if absent)."""
    _need(q_r, "q_r", torch.bfloat16, 3)
    _need(K_r, "K_r", torch.bfloat16, 4)
    _need(q, "q", torch.bfloat16, 4)
    _check_cache(K, V)
    _inner_contig(K_r, "K_r", 3)
    n_layers, B, L_cap_kv, H_kv, d = K.shape
    _, L_cap_r, H_r, d_r = K_r.shape
    if K_r.shape[0] != B or tuple(q_r.shape) != (B, H_r, d_r) or not q_r.is_contiguous():
        raise ValueError("q_r / K_r shapes do not match")
    if q.shape[0] != n_layers or q.shape[1] != B or q.shape[3] != d or not q.is_contiguous():
        raise ValueError("q must be contiguous [n_layers, B, H_q, d]")
    _i32(seq_lens, "seq_lens", B)
    _i32(ks, "ks", B)
    L_cap = min(L_cap_r, L_cap_kv)
    L_max = L_cap if L_max is None else int(L_max)
    dims = Dims.make(B=B, L_cap=L_cap, L_max=L_max, k_max=int(k_max), H_r=H_r, d_r=d_r,
                     n_layers=n_layers, H_q=q.shape[2], H_kv=H_kv, d=d,
                     kr_stride_b=K_r.stride(0), kv_stride_layer=K.stride(0),
                     kv_stride_b=K.stride(1), scale_r=scale_r, scale=scale,
                     n_sets=H_kv if head_level else 1)
    dev = q.device
    sets = (H_kv,) if head_level else ()
    o = outputs if outputs is not None else {}
    if "idx" not in o:
        o["idx"] = torch.empty((B,) + sets + (int(k_max),), dtype=torch.int32, device=dev)
        o["counts"] = torch.empty((B,), dtype=torch.int32, device=dev)
        o["out"] = torch.empty((n_layers, B, q.shape[2], d), dtype=torch.float32, device=dev)
        o["lse"] = (torch.empty((n_layers, B, q.shape[2]), dtype=torch.float32, device=dev)
                    if with_lse else None)
        o["scores"] = (torch.empty((B,) + sets + (L_max,), dtype=torch.float32, device=dev)
                       if with_scores else None)
    elif tuple(o["idx"].shape) != (B,) + sets + (int(k_max),):
        raise ValueError("outputs do not match the selection layout")
    return dims, o


def step(q_r, K_r, seq_lens, ks, q, K, V, k_max: int, L_max: Optional[int] = None,
         scale_r: float = 0.0, scale: float = 0.0, elastic: Optional[ElasticState] = None,
         with_scores: bool = False, with_lse: bool = False, ws: Optional[torch.Tensor] = None,
         outputs: Optional[dict] = None, head_level: bool = False):
    """One fused decode step (score -> top-k -> [elastic load] -> attention).
    Returns a dict with idx, counts, out and optionally lse and scores.
    head_level selects one token set per KV head (idx [B, H_kv, k_max],
    scores [B, H_kv, L_max]) instead of one per sequence."""
    lib = load_library()
    dims, o = _step_args(q_r, K_r, seq_lens, ks, q, K, V, k_max, L_max, scale_r, scale,
                         with_scores, with_lse, outputs, head_level)
    ws, nws = _workspace(dims, OP_STEP, q.device, ws)
    el = elastic.c_struct() if elastic is not None else None
    _check(lib.spec_step(ctypes.byref(dims), _p(q_r), _p(K_r), _p(seq_lens), _p(ks), _p(q),
                         _p(K), _p(V), _p(o["idx"]), _p(o["counts"]), _p(o["out"]),
                         _p(o.get("lse")), _p(o.get("scores")),
                         ctypes.byref(el) if el is not None else None, _p(ws), nws,
                         _stream(q)), "spec_step")
    return o


def step_noalloc(q_r, K_r, seq_lens, ks, q, K, V, k_max: int, L_max: Optional[int] = None,
                 scale_r: float = 0.0, scale: float = 0.0,
                 elastic: Optional[ElasticState] = None, with_scores: bool = False,
                 with_lse: bool = False, outputs: Optional[dict] = None,
                 head_level: bool = False):
    """spec_step_noalloc: the fused step on the library's static per-GPU
    scratch instead of a caller workspace (the library allocates nothing;
    pass `outputs` to allocate nothing here either).  Calls that overlap on
    one GPU race on that scratch."""
    lib = load_library()
    dims, o = _step_args(q_r, K_r, seq_lens, ks, q, K, V, k_max, L_max, scale_r, scale,
                         with_scores, with_lse, outputs, head_level)
    el = elastic.c_struct() if elastic is not None else None
    _check(lib.spec_step_noalloc(ctypes.byref(dims), _p(q_r), _p(K_r), _p(seq_lens), _p(ks),
                                 _p(q), _p(K), _p(V), _p(o["idx"]), _p(o["counts"]),
                                 _p(o["out"]), _p(o.get("lse")), _p(o.get("scores")),
                                 ctypes.byref(el) if el is not None else None, _stream(q)),
           "spec_step_noalloc")
    return o


class OffloadEvents:
    """The n_layers + 1 HIP events of the host-offload dataflow (caller-owned,
    as the C ABI wants them): event l marks layer l's rows loaded, the last
    one the fork after the slot plan."""

    def __init__(self, n: int, device):
        self.events = [torch.cuda.Event() for _ in range(n + 1)]
        with torch.cuda.device(device):
            for e in self.events:        # torch creates its events on first record
                e.record()
        self._arr = (ctypes.c_void_p * (n + 1))(*[e.cuda_event for e in self.events])

    def c_array(self):
        return self._arr


def _host_kv(Kh: torch.Tensor, Vh: torch.Tensor) -> HostKv:
    for t, nm in ((Kh, "K_host"), (Vh, "V_host")):
        _need_host = t.dtype == torch.bfloat16 and t.dim() == 5 and t.device.type == "cpu"
        if not _need_host or not t.is_pinned():
            raise ValueError(f"{nm} must be a pinned host bf16 tensor [n_off, B, L_cap, H_kv, d]")
    if Kh.shape != Vh.shape or Kh.stride() != Vh.stride():
        raise ValueError("K_host and V_host must have the same shape and strides")
    _inner_contig(Kh, "K_host", 3)
    return HostKv(Kh.data_ptr(), Vh.data_ptr(), Kh.stride(0), Kh.stride(1))


def offload_load(idx_now: torch.Tensor, counts: torch.Tensor, K_host: torch.Tensor,
                 V_host: torch.Tensor, state: ElasticState, copy_stream=None,
                 events: Optional[OffloadEvents] = None, L_max: Optional[int] = None,
                 ws: Optional[torch.Tensor] = None):
    """spec_offload_load: elastic loading of the offloaded layers from pinned
    host memory.  The slot plan runs on the current stream; with copy_stream
    (a torch.cuda.Stream) the per-layer host->device copies run there and
    events.events[l] marks layer l loaded.  Returns the events (or None)."""
    lib = load_library()
    n_off, B, L_cap, H_kv, d = K_host.shape
    _need(idx_now, "idx_now", torch.int32, 2)
    k_max = idx_now.shape[1]
    _i32(counts, "counts", B)
    if tuple(state.kbuf.shape) != (n_off, B, k_max, H_kv, d):
        raise ValueError("elastic state shape does not match")
    dims = Dims.make(B=B, L_cap=L_cap, L_max=L_cap if L_max is None else L_max, k_max=k_max,
                     n_layers=n_off, H_q=H_kv, H_kv=H_kv, d=d)
    ws, nws = _workspace(dims, OP_DELTA, idx_now.device, ws)
    host = _host_kv(K_host, V_host)
    if copy_stream is not None and events is None:
        events = OffloadEvents(n_off, idx_now.device)
    el = state.c_struct()
    _check(lib.spec_offload_load(ctypes.byref(dims), _p(idx_now.contiguous()), _p(counts),
                                 ctypes.byref(host), ctypes.byref(el), _p(ws), nws,
                                 _stream(idx_now),
                                 ctypes.c_void_p(copy_stream.cuda_stream) if copy_stream else None,
                                 events.c_array() if events is not None else None),
           "spec_offload_load")
    return events


def step_offload(q_r, K_r, seq_lens, ks, q, K, V, K_host, V_host, k_max: int,
                 state: ElasticState, copy_stream=None, events: Optional[OffloadEvents] = None,
                 L_max: Optional[int] = None, with_scores: bool = False, with_lse: bool = False,
                 ws: Optional[torch.Tensor] = None, outputs: Optional[dict] = None):
    """spec_step_offload: one decode step whose last n_off layers live in
    pinned host memory (K_host/V_host [n_off, B, L_cap, H_kv, d]) and whose
    first n_dev layers are the device caches K/V ([n_dev, ...]; with n_dev =
    0 pass None for both).  q is [n_dev + n_off, B, H_q, d].  The offloaded
    layers' rows are loaded elastically into `state` (slot buffers [n_off,
    B, k_max, H_kv, d]) on copy_stream (a torch.cuda.Stream, or None: all on
    the current stream), each layer's attention waiting for its own rows.
    Returns the outputs dict as step(), plus "events"."""
    lib = load_library()
    _need(q_r, "q_r", torch.bfloat16, 3)
    _need(K_r, "K_r", torch.bfloat16, 4)
    _need(q, "q", torch.bfloat16, 4)
    _inner_contig(K_r, "K_r", 3)
    n_off, B, L_cap, H_kv, d = K_host.shape
    host = _host_kv(K_host, V_host)
    n_dev = 0
    if K is not None:
        _check_cache(K, V)
        n_dev = K.shape[0]
        if tuple(K.shape[1:]) != (B, L_cap, H_kv, d):
            raise ValueError("device and host caches must have the same [B, L_cap, H_kv, d]")
    n_layers = n_dev + n_off
    _, L_cap_r, H_r, d_r = K_r.shape
    if K_r.shape[0] != B or tuple(q_r.shape) != (B, H_r, d_r) or not q_r.is_contiguous():
        raise ValueError("q_r / K_r shapes do not match")
    if tuple(q.shape[:2]) != (n_layers, B) or q.shape[3] != d or not q.is_contiguous():
        raise ValueError("q must be contiguous [n_dev + n_off, B, H_q, d]")
    _i32(seq_lens, "seq_lens", B)
    _i32(ks, "ks", B)
    if tuple(state.kbuf.shape) != (n_off, B, int(k_max), H_kv, d):
        raise ValueError("elastic state shape does not match")
    L = min(L_cap_r, L_cap)
    L_max = L if L_max is None else int(L_max)
    dims = Dims.make(B=B, L_cap=L, L_max=L_max, k_max=int(k_max), H_r=H_r, d_r=d_r,
                     n_layers=n_layers, H_q=q.shape[2], H_kv=H_kv, d=d,
                     kr_stride_b=K_r.stride(0),
                     kv_stride_layer=K.stride(0) if n_dev else 0,
                     kv_stride_b=K.stride(1) if n_dev else 0)
    ws, nws = _workspace(dims, OP_OFFLOAD, q.device, ws)
    dev = q.device
    o = outputs if outputs is not None else {}
    if "idx" not in o:
        o["idx"] = torch.empty((B, int(k_max)), dtype=torch.int32, device=dev)
        o["counts"] = torch.empty((B,), dtype=torch.int32, device=dev)
        o["out"] = torch.empty((n_layers, B, q.shape[2], d), dtype=torch.float32, device=dev)
        o["lse"] = (torch.empty((n_layers, B, q.shape[2]), dtype=torch.float32, device=dev)
                    if with_lse else None)
        o["scores"] = (torch.empty((B, L_max), dtype=torch.float32, device=dev)
                       if with_scores else None)
    if copy_stream is not None and events is None:
        events = OffloadEvents(n_off, dev)
    el = state.c_struct()
    _check(lib.spec_step_offload(ctypes.byref(dims), _p(q_r), _p(K_r), _p(seq_lens), _p(ks),
                                 _p(q), _p(K) if n_dev else None, _p(V) if n_dev else None,
                                 n_dev, ctypes.byref(host), _p(o["idx"]), _p(o["counts"]),
                                 _p(o["out"]), _p(o.get("lse")), _p(o.get("scores")),
                                 ctypes.byref(el), _p(ws), nws, _stream(q),
                                 ctypes.c_void_p(copy_stream.cuda_stream) if copy_stream else None,
                                 events.c_array() if events is not None else None),
           "spec_step_offload")
    o["events"] = events
    return o


def step_noalloc_max_bytes() -> int:
    """Bytes of spec_step_noalloc's static scratch (per GPU)."""
    return int(load_library().spec_step_noalloc_max_bytes())


def retrieval_qk(tokens: torch.Tensor, pos: torch.Tensor, emb: torch.Tensor, w_q: torch.Tensor,
                 w_k: torch.Tensor, K_r: torch.Tensor, rope_base: float = 500000.0,
                 yarn_scale: float = 1.0, yarn_orig_ctx: int = 2048, yarn_alpha: float = 0.0,
                 yarn_beta: float = 0.0, q_r: Optional[torch.Tensor] = None,
                 ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Retrieval-head front end of the new token of every sequence: embedding
    row, Q/K projection, rotary embedding with YaRN scaling.  Returns q_r
    [B, H_r, d_r] bf16 and writes each new key into K_r[b, pos[b]] in place
    (nothing for positions outside [0, L_cap)).  tokens, pos: int32 [B];
    emb [vocab, hidden]; w_q, w_k [H_r * d_r, hidden] (bf16)."""
    lib = load_library()
    _need(emb, "emb", torch.bfloat16, 2)
    _need(w_q, "w_q", torch.bfloat16, 2)
    _need(w_k, "w_k", torch.bfloat16, 2)
    _need(K_r, "K_r", torch.bfloat16, 4)
    _inner_contig(K_r, "K_r", 3)
    B = tokens.shape[0]
    _i32(tokens, "tokens", B)
    _i32(pos, "pos", B)
    if K_r.shape[0] != B:
        raise ValueError("K_r must hold B sequences")
    _, L_cap, H_r, d_r = K_r.shape
    vocab, hidden = emb.shape
    for t, nm in ((emb, "emb"), (w_q, "w_q"), (w_k, "w_k")):
        if not t.is_contiguous():
            raise ValueError(f"{nm} must be contiguous")
    if tuple(w_q.shape) != (H_r * d_r, hidden) or tuple(w_k.shape) != (H_r * d_r, hidden):
        raise ValueError("w_q / w_k must be [H_r * d_r, hidden]")
    if q_r is None:
        q_r = torch.empty((B, H_r, d_r), dtype=torch.bfloat16, device=K_r.device)
    elif tuple(q_r.shape) != (B, H_r, d_r) or not q_r.is_contiguous() or q_r.dtype != torch.bfloat16:
        raise ValueError("q_r must be contiguous bf16 [B, H_r, d_r]")
    dims = _dims_retrieval(K_r, L_cap, 1, 0.0)
    ws, nws = _workspace(dims, OP_FRONTEND, K_r.device, ws)
    fe = Frontend(vocab, hidden, rope_base, yarn_scale, yarn_orig_ctx, yarn_alpha, yarn_beta, 0)
    _check(lib.spec_retrieval_qk(ctypes.byref(dims), ctypes.byref(fe), _p(tokens), _p(pos),
                                 _p(emb), _p(w_q), _p(w_k), _p(q_r), _p(K_r), _p(ws), nws,
                                 _stream(K_r)), "spec_retrieval_qk")
    return q_r


def mla_workspace_size(dims: MlaDims) -> int:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check(lib.spec_mla_workspace_size(ctypes.byref(dims), ctypes.byref(n)),
           "spec_mla_workspace_size")
    return int(n.value)


def mla_sparse_decode_attn(q: torch.Tensor, ckv: torch.Tensor, w_uk: torch.Tensor,
                           w_uv: torch.Tensor, idx: torch.Tensor, counts: torch.Tensor,
                           scale: float = 0.0, out: Optional[torch.Tensor] = None,
                           lse: Optional[torch.Tensor] = None, with_lse: bool = True,
                           ws: Optional[torch.Tensor] = None):
    """Sparse decode attention of an MLA model over the selected tokens.
    q [n_layers, B, H, d_nope + d_rope]; ckv [n_layers, B, L_cap, d_c + d_rope]
    (latent, then rotary key; the last two dims packed); w_uk [n_layers, H,
    d_nope, d_c]; w_uv [n_layers, H, d_v, d_c] (bf16); idx [B, k_max] and
    counts [B] int32.  Returns (out fp32 [n_layers, B, H, d_v], lse fp32
    [n_layers, B, H] or None)."""
    lib = load_library()
    _need(q, "q", torch.bfloat16, 4)
    _need(ckv, "ckv", torch.bfloat16, 4)
    _need(w_uk, "w_uk", torch.bfloat16, 4)
    _need(w_uv, "w_uv", torch.bfloat16, 4)
    _need(idx, "idx", torch.int32, 2)
    n_layers, B, L_cap, dk = ckv.shape
    H = q.shape[2]
    d_nope = w_uk.shape[2]
    d_c = w_uk.shape[3]
    d_rope = dk - d_c
    d_v = w_uv.shape[2]
    if tuple(q.shape) != (n_layers, B, H, d_nope + d_rope) or not q.is_contiguous():
        raise ValueError("q must be contiguous [n_layers, B, H, d_nope + d_rope]")
    if tuple(w_uk.shape) != (n_layers, H, d_nope, d_c) or not w_uk.is_contiguous():
        raise ValueError("w_uk must be contiguous [n_layers, H, d_nope, d_c]")
    if tuple(w_uv.shape) != (n_layers, H, d_v, d_c) or not w_uv.is_contiguous():
        raise ValueError("w_uv must be contiguous [n_layers, H, d_v, d_c]")
    _inner_contig(ckv, "ckv", 2)
    if idx.shape[0] != B or not idx.is_contiguous():
        raise ValueError("idx must be contiguous [B, k_max]")
    _i32(counts, "counts", B)
    dims = MlaDims.make(B=B, L_cap=L_cap, k_max=idx.shape[1], n_layers=n_layers, H=H, d_c=d_c,
                        d_rope=d_rope, d_nope=d_nope, d_v=d_v, ckv_stride_layer=ckv.stride(0),
                        ckv_stride_b=ckv.stride(1), scale=scale)
    need = mla_workspace_size(dims)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    elif ws.numel() * ws.element_size() < need:
        raise ValueError(f"workspace too small: {need} bytes needed")
    if out is None:
        out = torch.empty((n_layers, B, H, d_v), dtype=torch.float32, device=q.device)
    if lse is None and with_lse:
        lse = torch.empty((n_layers, B, H), dtype=torch.float32, device=q.device)
    _check(lib.spec_mla_sparse_decode_attn(ctypes.byref(dims), _p(q), _p(ckv), _p(w_uk),
                                           _p(w_uv), _p(idx), _p(counts), _p(out), _p(lse),
                                           _p(ws), need, _stream(q)),
           "spec_mla_sparse_decode_attn")
    return out, lse
