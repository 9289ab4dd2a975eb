"""Host-side checks of the generated gfx950 code (no GPU needed).

The matrix-core kernel writes M0 and issues direct-to-LDS buffer loads from
inline assembly; its correctness rests on properties of the generated code
that the compiler does not guarantee by itself, so they are checked here:
  * M0 is touched only inside the kernel's own inline-assembly blocks;
  * every direct-to-LDS load takes its offset from a scalar register;
  * no packed fp32 add/mul/fma instruction is emitted anywhere;
  * the main kernels keep their scratch (spill) use small.
"""
import os
import re
import shutil

import pytest

from paper_2607_05708_amd import build

HIPCC_OK = os.path.exists(build.HIPCC) or shutil.which("hipcc") is not None
pytestmark = pytest.mark.skipif(not HIPCC_OK, reason="hipcc not available")

SOURCES = ["csrc/api.cpp", "csrc/topk_valu.hip", "csrc/topk_mfma.hip", "csrc/gather_append.hip", "csrc/compact.hip"]


@pytest.fixture(scope="module")
def asm():
    return {src: build.device_asm(src) for src in SOURCES}


def _code_lines_outside_inline_asm(text):
    inside = False
    for line in text.splitlines():
        if ";;#ASMSTART" in line:
            inside = True
            continue
        if ";;#ASMEND" in line:
            inside = False
            continue
        if not inside:
            yield line


def _strip_comment(line):
    return line.split(";", 1)[0]


def test_m0_only_in_inline_asm(asm):
    for src, text in asm.items():
        bad = [l for l in _code_lines_outside_inline_asm(text)
               if re.search(r"\bm0\b", _strip_comment(l)) and not l.lstrip().startswith(".")]
        assert not bad, f"{src}: compiler-generated code uses M0: {bad[:5]}"


def test_lds_dma_offsets_are_scalar(asm):
    text = asm["csrc/topk_mfma.hip"]
    loads = [l.strip() for l in text.splitlines() if re.search(r"offen (nt )?lds", l)]
    assert loads, "no direct-to-LDS loads found"
    pat = re.compile(r"^buffer_load_dwordx4 v\d+, s\[\d+:\d+\], s\d+ offen (nt )?lds$")
    bad = [l for l in loads if not pat.match(l)]
    assert not bad, f"direct-to-LDS loads with non-scalar operands: {bad[:5]}"


def test_non_temporal_loads_only_in_narrow_dense_shape(asm):
    # Only the full pass of the 64-query shape (no other workgroup reads its
    # bank lines), and not its grouped form, marks lines for early eviction.
    bodies = _kernel_bodies(asm["csrc/topk_mfma.hip"], "topk_mfma_kernel")
    seen = 0
    for name, body in bodies.items():
        m = re.search(r"topk_mfma_kernelILi\d+ELb([01])ELi(\d)ELb[01]ELb([01])E", name)
        assert m, name
        narrow_full = m.group(1) == "0" and m.group(2) == "1" and m.group(3) == "0"
        has_nt = "offen nt lds" in body
        assert has_nt == narrow_full, name
        seen += narrow_full
    assert seen == 6   # 3 list sizes x (dense, scoped)


def test_no_packed_fp32(asm):
    for src, text in asm.items():
        hits = re.findall(r"\bv_pk_(?:add|mul|fma)_f32\b", text)
        assert not hits, f"{src}: packed fp32 instructions emitted"


def test_main_kernel_no_scratch(asm):
    # A spill reload is a vector-memory load: waiting for it also waits for
    # every staging load in flight, which drains the load pipeline.
    text = asm["csrc/topk_mfma.hip"]
    kernels = re.findall(r"\.name:\s+(\S+)", text)
    spills = [int(x) for x in re.findall(r"\.vgpr_spill_count:\s+(\d+)", text)]
    priv = [int(x) for x in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", text)]
    assert len(kernels) == len(spills) == len(priv)
    for name, sp, pv in zip(kernels, spills, priv):
        assert sp == 0 and pv == 0, f"{name}: {sp} spilled VGPRs, {pv} B scratch"


def test_main_loop_waits(asm):
    # Inside the stage loop the only vector-memory wait is the stage barrier's.
    text = asm["csrc/topk_mfma.hip"]
    for m in re.finditer(r"^(_Z\S*topk_mfma_kernel\S*):\s*$(.*?)s_endpgm", text, re.S | re.M):
        body = m.group(2)
        waits = re.findall(r"s_waitcnt[^\n]*vmcnt\((\d+)\)[^\n]*\n\s*s_barrier", body)
        assert waits, f"{m.group(1)}: no stage barrier found"


def _kernel_bodies(text, pattern):
    out = {}
    for m in re.finditer(r"^(_Z\S*" + pattern + r"\S*):\s*(?:;.*)?$", text, re.M):
        end = text.find(".Lfunc_end", m.end())
        out[m.group(1)] = text[m.end():end]
    return out


def test_scoped_namespaces_use_scalar_loads(asm):
    # The scoped epilogue reads each half block's 16 row namespaces with
    # scalar loads; a vector load there would wait behind the staging loads.
    # Scoped instances may add only the one vector load of the key's own
    # namespace, made before the staging loads start.
    bodies = _kernel_bodies(asm["csrc/topk_mfma.hip"], "topk_mfma_kernel")
    count = lambda body, pat: len(re.findall(pat, body))  # noqa: E731
    pairs = 0
    for name, body in bodies.items():
        if "Lb1ELb0EEEv" not in name:   # scoped (and not grouped) instances
            continue
        plain = bodies[name.replace("Lb1ELb0EEEv", "Lb0ELb0EEEv")]
        assert count(body, r"\tglobal_load") <= count(plain, r"\tglobal_load") + 1, name
        assert count(body, r"\ts_load_dwordx16") >= 1, name
        pairs += 1
    assert pairs == 18   # 3 list sizes x 3 shapes x (sample, full)
