"""Shared glue for the GPU parity tests (no method arithmetic here)."""
import os
import sys

import numpy as np
import pytest
import torch

TOL_ATTN = 2e-3          # max-abs on attention outputs (bf16 in, fp32 accumulate)
SCORE_ABS, SCORE_REL = 1e-7, 1e-5   # internal gate on retrieval scores


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU on this host")
    import paper_2512_00722_amd as spec
    spec.load_library()   # raises if the HIP library is missing: no fallback exists
    return torch.device("cuda:0")


def f64(t: torch.Tensor) -> np.ndarray:
    """Exact float64 copy of a (bf16 / fp32) tensor."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def announce(msg: str):
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()
