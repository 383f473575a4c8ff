"""The C ABI on a host without a GPU: the library loads, exports every symbol
include/spec.h declares, and rejects bad arguments before any HIP call
(fake pointers are never dereferenced because validation fails first)."""
import ctypes
import os
import re

import pytest

import paper_2512_00722_amd as spec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    # SPEC_TEST_LIB names another build of the same library (the host
    # sanitizer variant, run by test_host_sanitizers in a child process)
    other = os.environ.get("SPEC_TEST_LIB")
    if other:
        return spec.load_library(other)
    if not os.path.exists(spec.lib_path):
        pytest.fail("libspecctx.so is not built (run __graft_entry__.build())")
    return spec.load_library()


def header_functions():
    txt = open(os.path.join(ROOT, "include", "spec.h")).read()
    return re.findall(r"SPEC_API\s+[\w\s\*]+?\b(spec_\w+)\s*\(", txt)


def test_exports_every_declared_symbol(lib):
    declared = header_functions()
    assert len(declared) >= 10
    assert sorted(declared) == sorted(spec.EXPORTED_SYMBOLS)
    for name in declared:
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert b"gfx950" in lib.spec_version()
    for s in range(5):
        assert lib.spec_status_string(s)
    assert lib.spec_status_string(99) == b"unknown status"
    assert lib.spec_last_hip_error() == 0


FAKE = ctypes.c_void_p(0x7000_0000_0000)     # 16-byte aligned, never dereferenced
FAKE_ODD = ctypes.c_void_p(0x7000_0000_0008)  # 8-byte aligned only


def good_dims(**kw):
    # k_max above 4 x 2048 makes the attention split its selection across
    # workgroups, so that its workspace is not empty
    base = dict(B=2, L_cap=16384, L_max=16384, k_max=12288, H_r=8, d_r=64, n_layers=2, H_q=32,
                H_kv=8, d=128)
    base.update(kw)
    return spec.Dims.make(**base)


def ws_size(lib, dims, op):
    n = ctypes.c_size_t(0)
    st = lib.spec_workspace_size(ctypes.byref(dims), op, ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("field,value,status", [
    ("B", 0, 1), ("L_cap", -1, 1), ("k_max", 0, 1), ("H_r", 0, 1), ("d", 0, 1),
    ("L_max", 16385, 1),        # L_max > L_cap
    ("k_max", 16385, 1),        # k_max > L_max
    ("H_q", 30, 1),             # H_q % H_kv != 0
    ("d", 64, 2), ("d_r", 32, 2), ("H_r", 17, 2), ("H_kv", 32, 2),
    ("H_q", 24, 2),             # G = 3
    ("n_sets", 4, 2),           # neither 1 nor H_kv
    ("n_sets", 0, 2),
    ("reserved", 1, 1),
    ("kv_stride_b", 12, 1),     # smaller than a sequence's block
    ("kr_stride_b", 16384 * 8 * 64 + 3, 1),  # not a multiple of 8
    ("scale", -1.0, 1),
])
def test_dims_validation(lib, field, value, status):
    d = good_dims()
    setattr(d, field, value)
    for op in range(7):
        st, _ = ws_size(lib, d, op)
        assert st == status, (field, op, st)


def test_large_query_groups(lib):
    """More than 16 query heads per KV head (MQA-like) run as 16-head column
    groups: powers of two up to 128 are accepted; the attention workspace
    still holds one partial row per query head."""
    for H_q, H_kv in [(32, 1), (64, 1), (128, 1), (64, 2), (128, 4)]:
        d = good_dims(H_q=H_q, H_kv=H_kv)
        for op in range(7):
            assert ws_size(lib, d, op)[0] == 0, (H_q, H_kv, op)
    assert ws_size(lib, good_dims(H_q=256, H_kv=1), spec.OP_ATTN)[0] == 2   # G = 256
    assert ws_size(lib, good_dims(H_q=48, H_kv=1), spec.OP_ATTN)[0] == 2    # G = 48
    # with fewer KV heads the groups split further: a workspace is still sized
    _, n = ws_size(lib, good_dims(H_q=64, H_kv=1), spec.OP_ATTN)
    assert n == 0 or n >= 2 * 2 * 64 * 128 * 4


def test_head_level_sets(lib):
    # one set per KV head: valid when H_r is a multiple of H_kv
    d = good_dims(n_sets=8)
    for op in range(7):
        assert ws_size(lib, d, op)[0] == 0
    st1, n1 = ws_size(lib, good_dims(), spec.OP_STEP)
    st8, n8 = ws_size(lib, d, spec.OP_STEP)
    assert n8 > n1                       # per-set scores, histograms and lists
    assert ws_size(lib, good_dims(n_sets=8, H_r=12), spec.OP_SCORE)[0] == 2
    assert ws_size(lib, good_dims(n_sets=8, B=9000), spec.OP_TOPK)[0] == 2   # B*n_sets rows
    # elastic loading keeps one token per slot for every head: not with sets
    el = spec.Elastic(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    _, nws = ws_size(lib, d, spec.OP_STEP)
    assert lib.spec_delta_gather(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, ctypes.byref(el), FAKE,
                                 nws, None) == 2
    assert lib.spec_step(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                         FAKE, None, None, ctypes.byref(el), FAKE, nws, None) == 2
    assert lib.spec_sparse_decode_attn_elastic(ctypes.byref(d), FAKE, FAKE, FAKE,
                                               ctypes.byref(el), FAKE, FAKE, None, FAKE, nws,
                                               None) == 2
    assert lib.spec_last_hip_error() == 0


def test_workspace_sizes(lib):
    d = good_dims()
    sizes = {op: ws_size(lib, d, op) for op in range(7)}
    assert all(st == 0 for st, _ in sizes.values())
    assert sizes[spec.OP_GATHER][1] == 0
    assert sizes[spec.OP_SCORE][1] >= 2 * 16384 * 8 * 4      # the logits
    assert sizes[spec.OP_STEP][1] >= sizes[spec.OP_SCORE][1] + sizes[spec.OP_ATTN][1]
    assert lib.spec_workspace_size(None, 0, ctypes.byref(ctypes.c_size_t())) == 1
    assert lib.spec_workspace_size(ctypes.byref(d), 9, ctypes.byref(ctypes.c_size_t())) == 1
    # the front end's fp32 partial sums: up to 16 slices of [B][2 * H_r * d_r]
    assert sizes[spec.OP_FRONTEND][1] >= 16 * 2 * 2 * 8 * 64 * 4


def test_entry_points_reject_before_hip(lib):
    d = good_dims()
    _, nws = ws_size(lib, d, spec.OP_STEP)
    byref = ctypes.byref
    # null pointers
    assert lib.spec_score(byref(d), None, FAKE, FAKE, FAKE, FAKE, nws, None) == 1
    assert lib.spec_topk(byref(d), FAKE, FAKE, None, FAKE, None, FAKE, nws, None) == 1
    assert lib.spec_gather(byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == 1
    assert lib.spec_sparse_decode_attn(byref(d), FAKE, FAKE, FAKE, None, None, FAKE, None,
                                       FAKE, nws, None) == 1
    # misaligned bf16 tensor
    assert lib.spec_score(byref(d), FAKE_ODD, FAKE, FAKE, FAKE, FAKE, nws, None) == 1
    assert lib.spec_sparse_decode_attn(byref(d), FAKE, FAKE_ODD, FAKE, FAKE, FAKE, FAKE, None,
                                       FAKE, nws, None) == 1
    # workspace missing or too small (the sizes used must really be too small:
    # a call that passed validation would launch a kernel on fake pointers)
    _, n_attn = ws_size(lib, d, spec.OP_ATTN)
    _, n_score = ws_size(lib, d, spec.OP_SCORE)
    assert n_attn > 16 and n_score > 0
    assert lib.spec_score(byref(d), FAKE, FAKE, FAKE, FAKE, None, 0, None) == 3
    assert lib.spec_sparse_decode_attn(byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                       FAKE, 16, None) == 3
    assert lib.spec_step(byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                         None, None, None, FAKE, 64, None) == 3
    # unsupported dims on every entry point
    bad = good_dims(d=96)
    assert lib.spec_score(byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, nws, None) == 2
    assert lib.spec_step(byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                         None, None, None, FAKE, nws, None) == 2
    # elastic state with a null member
    el = spec.Elastic(FAKE.value, FAKE.value, None, FAKE.value, FAKE.value)
    assert lib.spec_delta_gather(byref(d), FAKE, FAKE, FAKE, FAKE, byref(el), FAKE, nws,
                                 None) == 1
    assert lib.spec_sparse_decode_attn_elastic(byref(d), FAKE, FAKE, FAKE, byref(el), FAKE,
                                               FAKE, None, FAKE, nws, None) == 1
    assert lib.spec_sparse_decode_attn_elastic(byref(d), FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                               None, FAKE, nws, None) == 1
    # the elastic attention needs the slot sources and its workspace
    el = spec.Elastic(FAKE.value, FAKE.value, FAKE.value, FAKE.value, None)
    assert lib.spec_sparse_decode_attn_elastic(byref(d), FAKE, FAKE, FAKE, byref(el), FAKE,
                                               FAKE, None, FAKE, nws, None) == 1
    assert lib.spec_step(byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                         None, None, byref(el), FAKE, nws, None) == 1
    el = spec.Elastic(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value + 2)
    assert lib.spec_sparse_decode_attn_elastic(byref(d), FAKE, FAKE, FAKE, byref(el), FAKE,
                                               FAKE, None, FAKE, nws, None) == 1
    el = spec.Elastic(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    assert lib.spec_sparse_decode_attn_elastic(byref(d), FAKE, FAKE, FAKE, byref(el), FAKE,
                                               FAKE, None, FAKE, 16, None) == 3
    assert lib.spec_sparse_decode_attn_elastic(byref(d), FAKE_ODD, FAKE, FAKE, byref(el), FAKE,
                                               FAKE, None, FAKE, nws, None) == 1
    # elastic loading caps L_cap
    big = good_dims(L_cap=300000, L_max=300000)
    el = spec.Elastic(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    assert lib.spec_delta_gather(byref(big), FAKE, FAKE, FAKE, FAKE, byref(el), FAKE, 1 << 40,
                                 None) == 2
    assert lib.spec_last_hip_error() == 0


def good_frontend(**kw):
    base = dict(vocab=128256, hidden=4096, rope_base=500000.0, yarn_scale=16.0,
                yarn_orig_ctx=2048, yarn_alpha=0.0, yarn_beta=0.0, reserved=0)
    base.update(kw)
    return spec.Frontend(**base)


@pytest.mark.parametrize("field,value,status", [
    ("vocab", 0, 1), ("hidden", -128, 1), ("hidden", 4000, 2),   # not a multiple of 128
    ("rope_base", 0.0, 1), ("rope_base", float("inf"), 1), ("yarn_scale", float("nan"), 1),
    ("yarn_orig_ctx", 0, 1),                                      # needed when scaling
    ("yarn_alpha", 40.0, 1),                                      # alpha >= beta = 32
    ("reserved", 3, 1),
])
def test_frontend_validation(lib, field, value, status):
    """Every rejection of spec_retrieval_qk happens on the host."""
    d = good_dims()
    fe = good_frontend()
    setattr(fe, field, value)
    if field == "yarn_alpha":
        fe.yarn_beta = 32.0
    args = (FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30)
    assert lib.spec_retrieval_qk(ctypes.byref(d), ctypes.byref(fe), *args, None) == status
    assert lib.spec_last_hip_error() == 0


def test_frontend_rejects_before_hip(lib):
    d = good_dims()
    fe = good_frontend()
    byref = ctypes.byref
    _, nws = ws_size(lib, d, spec.OP_FRONTEND)
    ws = (FAKE, nws)
    assert lib.spec_retrieval_qk(byref(d), None, *(FAKE,) * 7, *ws, None) == 1
    assert lib.spec_retrieval_qk(None, byref(fe), *(FAKE,) * 7, *ws, None) == 1
    for i in range(7):              # each tensor null in turn, then misaligned
        args = [FAKE] * 7
        args[i] = None
        assert lib.spec_retrieval_qk(byref(d), byref(fe), *args, *ws, None) == 1, i
        args[i] = ctypes.c_void_p(FAKE.value + (2 if i < 2 else 8))
        assert lib.spec_retrieval_qk(byref(d), byref(fe), *args, *ws, None) == 1, i
    # workspace missing, too small, misaligned
    assert lib.spec_retrieval_qk(byref(d), byref(fe), *(FAKE,) * 7, None, nws, None) == 3
    assert lib.spec_retrieval_qk(byref(d), byref(fe), *(FAKE,) * 7, FAKE, nws - 1, None) == 3
    assert lib.spec_retrieval_qk(byref(d), byref(fe), *(FAKE,) * 7, FAKE_ODD, nws, None) == 1
    # the retrieval dimensions are validated as for every entry point
    assert lib.spec_retrieval_qk(byref(good_dims(d_r=96)), byref(fe), *(FAKE,) * 7, *ws,
                                 None) == 2
    assert lib.spec_retrieval_qk(byref(good_dims(kr_stride_b=12)), byref(fe), *(FAKE,) * 7,
                                 *ws, None) == 1
    assert lib.spec_last_hip_error() == 0


def good_mla(**kw):
    base = dict(B=8, L_cap=32768, k_max=2048, n_layers=61, H=128)
    base.update(kw)
    return spec.MlaDims.make(**base)


@pytest.mark.parametrize("field,value,status", [
    ("B", 0, 1), ("k_max", 40000, 1), ("n_layers", -1, 1), ("reserved", 1, 1), ("reserved2", 2, 1),
    ("scale", -1.0, 1), ("scale", float("nan"), 1), ("ckv_stride_b", 100, 1),
    ("ckv_stride_b", 32768 * 576 + 4, 1),
    ("d_c", 256, 2), ("d_rope", 32, 2), ("d_nope", 64, 2), ("d_v", 64, 2), ("H", 32, 2),
    ("H", 96, 2), ("B", 70000, 2),
])
def test_mla_validation(lib, field, value, status):
    d = good_mla()
    if field == "k_max" and value > 32768:
        d.L_cap = 65536   # k_max within L_cap, above the supported 32768
        status = 2
    setattr(d, field, value)
    n = ctypes.c_size_t(0)
    assert lib.spec_mla_workspace_size(ctypes.byref(d), ctypes.byref(n)) == status
    assert lib.spec_mla_sparse_decode_attn(ctypes.byref(d), *(FAKE,) * 6, FAKE, None, FAKE,
                                           1 << 40, None) == status
    assert lib.spec_last_hip_error() == 0


def test_mla_rejects_before_hip(lib):
    d = good_mla()
    n = ctypes.c_size_t(0)
    assert lib.spec_mla_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    # absorbed queries of every (layer, sequence, head) and one split of partials
    assert n.value >= 61 * 8 * 128 * (576 * 2 + 512 * 4)
    byref = ctypes.byref
    for i in range(7):              # q, ckv, w_uk, w_uv, idx, counts, out: null, then misaligned
        args = [FAKE] * 7
        args[i] = None
        assert lib.spec_mla_sparse_decode_attn(byref(d), *args, None, FAKE, n.value, None) == 1
        args[i] = ctypes.c_void_p(FAKE.value + (2 if i in (4, 5) else 8))
        assert lib.spec_mla_sparse_decode_attn(byref(d), *args, None, FAKE, n.value, None) == 1
    args = [FAKE] * 7
    assert lib.spec_mla_sparse_decode_attn(byref(d), *args, None, None, n.value, None) == 3
    assert lib.spec_mla_sparse_decode_attn(byref(d), *args, None, FAKE, n.value - 1, None) == 3
    assert lib.spec_mla_sparse_decode_attn(byref(d), *args, ctypes.c_void_p(FAKE.value + 2),
                                           FAKE, n.value, None) == 1     # misaligned lse
    assert lib.spec_mla_workspace_size(None, byref(n)) == 1
    assert lib.spec_mla_workspace_size(byref(d), None) == 1
    assert lib.spec_last_hip_error() == 0


def test_python_wrappers_refuse_cpu_tensors(lib):
    import torch
    q_r = torch.zeros((1, 8, 64), dtype=torch.bfloat16)
    K_r = torch.zeros((1, 64, 8, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        spec.score(q_r, K_r, torch.zeros(1, dtype=torch.int32))
    with pytest.raises(TypeError):
        spec.score(q_r.float(), K_r, torch.zeros(1, dtype=torch.int32))


def test_host_sanitizers():
    """Every ABI test above, again in a child process against the host
    sanitizer build (spec_api.cpp under AddressSanitizer and
    UndefinedBehaviorSanitizer): any out-of-bounds access, use of freed
    memory or undefined behaviour in the host-side validation and
    workspace carve-up aborts the child."""
    import subprocess
    import sys

    from paper_2512_00722_amd import build as b

    if os.environ.get("SPEC_TEST_LIB"):
        pytest.skip("already the sanitized child")
    path = b.build_sanitized()
    nm = subprocess.run(["nm", "-D", path], capture_output=True, text=True).stdout
    assert "__asan_report_load" in nm and "__ubsan_handle" in nm   # really instrumented
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    env = dict(os.environ, SPEC_TEST_LIB=path, LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py"),
                        "-k", "not host_sanitizers"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out, out[-2000:]


def test_step_noalloc_rejects_before_hip(lib):
    """The allocation-free step validates as spec_step does and rejects a
    step whose workspace exceeds its static scratch, all before any HIP
    call (fake pointers are never touched)."""
    assert lib.spec_step_noalloc_max_bytes() == 64 << 20
    assert lib.spec_status_string(5) and lib.spec_status_string(5) != b"unknown status"
    byref = ctypes.byref
    args = lambda: [FAKE] * 10 + [None, None, None]   # q_r .. out; lse, scores, elastic
    d = good_dims()
    a = args()
    a[0] = None
    assert lib.spec_step_noalloc(byref(d), *a, None) == 1                 # null q_r
    a = args()
    a[5] = FAKE_ODD
    assert lib.spec_step_noalloc(byref(d), *a, None) == 1                 # misaligned K
    assert lib.spec_step_noalloc(byref(good_dims(d=96)), *args(), None) == 2
    # a step that needs more than 64 MiB of workspace (logits and lists of
    # 64 sequences of 128K tokens)
    big = good_dims(B=64, L_cap=131072, L_max=131072, k_max=2048)
    _, need = ws_size(lib, big, spec.OP_STEP)
    assert need > 64 << 20
    assert lib.spec_step_noalloc(byref(big), *args(), None) == 5
    assert lib.spec_last_hip_error() == 0


def test_offload_rejects_before_launch(lib):
    """The host-offload entry points validate everything before any launch:
    a host pointer that is not pinned host memory (here a fake address the
    runtime does not know) is rejected, as are a copy stream without events,
    device-layer counts out of range, head-level sets and small workspaces."""
    byref = ctypes.byref
    d = good_dims(n_layers=4)
    st_off, n_off = ws_size(lib, d, spec.OP_OFFLOAD)
    st_step, n_step = ws_size(lib, d, spec.OP_STEP)
    assert st_off == 0 and n_off >= n_step - ws_size(lib, d, spec.OP_ATTN)[1]
    host = spec.HostKv(FAKE.value, FAKE.value, 0, 0)
    el = spec.Elastic(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value)
    _, nd = ws_size(lib, d, spec.OP_DELTA)
    ev = (ctypes.c_void_p * 5)()
    # spec_offload_load
    assert lib.spec_offload_load(byref(d), FAKE, FAKE, byref(host), byref(el), FAKE, nd, None,
                                 None, None) == 1          # not pinned host memory
    assert lib.spec_offload_load(byref(d), FAKE, FAKE, byref(host), byref(el), FAKE, nd, None,
                                 FAKE, None) == 1          # copy stream without events
    assert lib.spec_offload_load(byref(d), FAKE, FAKE, None, byref(el), FAKE, nd, None, None,
                                 None) == 1
    assert lib.spec_offload_load(byref(d), FAKE, FAKE, byref(host), byref(el), None, 0, None,
                                 None, None) == 3
    assert lib.spec_offload_load(byref(good_dims(n_sets=8)), FAKE, FAKE, byref(host), byref(el),
                                 FAKE, 1 << 40, None, None, None) == 2
    # spec_step_offload
    args = lambda n_dev: [FAKE] * 7 + [n_dev, byref(host)] + [FAKE] * 3 + [None, None]
    for n_dev in (-1, 4, 5):
        assert lib.spec_step_offload(byref(d), *args(n_dev), byref(el), FAKE, n_off, None, None,
                                     None) == 1, n_dev
    assert lib.spec_step_offload(byref(d), *args(2), None, FAKE, n_off, None, None, None) == 1
    assert lib.spec_step_offload(byref(d), *args(2), byref(el), FAKE, n_off, None, FAKE,
                                 None) == 1              # copy stream without events
    assert lib.spec_step_offload(byref(d), *args(2), byref(el), FAKE, 64, None, None, None) == 3
    assert lib.spec_step_offload(byref(d), *args(2), byref(el), FAKE, n_off, None, None,
                                 None) == 1              # fake host memory
    assert lib.spec_step_offload(byref(good_dims(n_layers=4, d=96)), *args(2), byref(el), FAKE,
                                 n_off, None, None, None) == 2
    assert lib.spec_last_hip_error() == 0
