"""Machine-code checks of the inline assembly in the kernels that issue
global->LDS loads (the wide prefill kernel and the wide GEMM; host only: the
kernels are compiled to gfx950 assembly, nothing runs).

Their tile requests are inline assembly that writes M0 with an SALU
instruction and then issues a global->LDS load.  Two properties keep them
correct:

* an SALU add into M0 sets SCC, so no SCC value of compiler code may be
  live across such a request: an SCC consumer (s_addc_u32 finishing a 64-bit address, a
  conditional select or branch) after a request must see SCC written again by
  compiler code first (without that, a carry was lost and the high half of a
  cache-block address came out 4 GiB low);
* a load that reads M0 needs one wait state after an SALU write of M0.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_04875_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SCC_READ = re.compile(r"^(s_addc_u32|s_subb_u32|s_cselect_b(32|64)|s_cbranch_scc[01]|s_cmov_b(32|64))\b")
SCC_WRITE = re.compile(
    r"^(s_(add|sub)_[ui]32|s_addc_u32|s_subb_u32|s_cmp_\w+|s_(and|or|xor|andn2|orn2|nand|nor|xnor|not)_b(32|64)"
    r"|s_(lshl|lshr)_b(32|64)|s_ashr_i(32|64)|s_bfe_\w+|s_(min|max)_[ui]32|s_abs_i32|s_bcnt\w+"
    r"|s_lshl\d_add_u32|s_(and|or)_saveexec_b64)\b")


KERNELS = {"attn": ("attn_bf16_wide.hip", "attn_bf16_wide_kernel", 24),
           "gemm": ("gemm_bf16_wide.hip", "gemm_bf16_wide_kernel", 32)}


@pytest.fixture(scope="module", params=sorted(KERNELS))
def wide_asm(request, tmp_path_factory):
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    src, kernel, min_requests = KERNELS[request.param]
    out = tmp_path_factory.mktemp("isa") / (request.param + ".s")
    cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", "-x", "hip",
           "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    lines = [ln.split(";")[0].strip() if not ln.strip().startswith(";;#ASM") else ln.strip()
             for ln in out.read_text().splitlines()]
    start = next(i for i, ln in enumerate(lines) if re.match(rf"^_Z\w*{kernel}\w*:", ln))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith("s_endpgm"))
    return lines[start:end + 1], min_requests


def _asm_blocks(lines):
    """(first, last) line indexes of each inline-assembly block."""
    blocks, open_at = [], None
    for i, ln in enumerate(lines):
        if ln.startswith(";;#ASMSTART"):
            open_at = i
        elif ln.startswith(";;#ASMEND"):
            blocks.append((open_at, i))
    return blocks


def test_requests_present(wide_asm):
    lines, min_requests = wide_asm
    n = sum(1 for ln in lines if ln.startswith("global_load_lds_dwordx4"))
    assert n >= min_requests, f"expected the prologue's and the loop's tile requests, found {n}"


def test_no_compiler_scc_value_across_a_request(wide_asm):
    wide_asm, _ = wide_asm
    bad = []
    for a, b in _asm_blocks(wide_asm):
        if not any(SCC_WRITE.match(ln) for ln in wide_asm[a + 1:b]):
            continue
        for i in range(b + 1, len(wide_asm)):
            ln = wide_asm[i]
            if ln.startswith(";;#ASMSTART") or ln.endswith(":"):
                break                                # another block or a label: checked on its own
            if SCC_READ.match(ln):
                bad.append(f"{ln!r} reads SCC set by the inline assembly ending {i - b} lines above")
                break
            if SCC_WRITE.match(ln):
                break
    assert not bad, "\n".join(bad[:5])


def test_wait_state_between_m0_write_and_lds_load(wide_asm):
    wide_asm, _ = wide_asm
    bad = []
    for a, b in _asm_blocks(wide_asm):
        body = [ln for ln in wide_asm[a + 1:b] if ln]
        for j, ln in enumerate(body):
            if ln.startswith("global_load_lds") and j > 0 and re.match(r"^s_\w+ m0\b", body[j - 1]):
                bad.append(" / ".join(body))
    assert not bad, "\n".join(bad[:3])
