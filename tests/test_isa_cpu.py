"""Checks on the gfx950 assembly of every HIP source, compiled here (no GPU):

* no packed fp32 instructions: the sources are built with packed fp32 code
  generation disabled, and none are written by hand;
* no writes through the scalar data cache (scalar memory stores or atomics,
  the cache's write-back or discard): every kernel writes with vector stores;
* in mla.hip, M0 -- named as clobbered by the inline global-to-LDS copies,
  although the compiler reserves it -- is written only by those copies, each
  write directly followed by its load, and no other instruction touches it.

The flags are the build's own (paper_2512_00722_amd.build.flags_for).
"""
import concurrent.futures
import os
import re
import shutil
import subprocess

import pytest

from paper_2512_00722_amd import build as B

HIP_SOURCES = [s for s in B.sources() if s.endswith(".hip")]

pytestmark = pytest.mark.skipif(not os.path.exists(B.HIPCC), reason="hipcc not found")


def _instructions(asm_text):
    """(kernel, instruction) pairs: comments, directives and labels dropped."""
    out, kernel = [], None
    for line in asm_text.splitlines():
        code = line.split(";")[0].strip()
        if not code:
            continue
        if code.endswith(":") and not code.startswith("."):
            if not code.startswith(".L"):
                kernel = code[:-1]
            continue
        if code.startswith(".") or code.endswith(":"):
            continue
        out.append((kernel, code))
    return out


@pytest.fixture(scope="module")
def assembly(tmp_path_factory):
    d = tmp_path_factory.mktemp("isa")

    def one(src):
        dst = d / (os.path.basename(src) + ".s")
        cmd = [B.HIPCC, *B.flags_for(src), "-x", "hip", "--cuda-device-only", "-S", "-o",
               str(dst), src]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return os.path.basename(src), _instructions(dst.read_text())

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(HIP_SOURCES))) as ex:
        res = dict(ex.map(one, HIP_SOURCES))
    shutil.rmtree(d, ignore_errors=True)
    return res


def test_every_source_compiled(assembly):
    assert set(assembly) == {os.path.basename(s) for s in HIP_SOURCES}
    for name, ins in assembly.items():
        assert ins, name


def test_no_packed_fp32(assembly):
    pat = re.compile(r"^v_pk_(fma|mul|add|mov)_f32\b")
    bad = [(n, k, i) for n, ins in assembly.items() for k, i in ins if pat.match(i)]
    assert not bad, bad[:5]


def test_no_scalar_cache_writes(assembly):
    pat = re.compile(r"^s_(store|buffer_store|scratch_store|atomic|buffer_atomic|dcache_wb"
                     r"|dcache_discard)")
    bad = [(n, k, i) for n, ins in assembly.items() for k, i in ins if pat.match(i)]
    assert not bad, bad[:5]


def test_m0_only_in_the_global_to_lds_copies(assembly):
    ins = assembly["mla.hip"]
    uses = [j for j, (_, i) in enumerate(ins) if re.search(r"\bm0\b", i)]
    assert uses, "the global-to-LDS copies are expected in mla.hip"
    for j in uses:
        kernel, i = ins[j]
        assert re.match(r"^s_mov_b32 m0, s\d+$", i), (kernel, i)
        nxt = ins[j + 1][1]
        assert nxt.startswith("global_load_lds_dwordx4"), (kernel, i, nxt)
    # the copies are the only users of the LDS-direct load
    copies = [j for j, (_, i) in enumerate(ins) if i.startswith("global_load_lds")]
    assert copies == [j + 1 for j in uses]
