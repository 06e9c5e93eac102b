"""Checks of the gfx950 assembly of the 4-wave 256 x 256 kernels (CPU only: hipcc
cross-compiles the kernel source).

Their K loop issues its MFMAs from assembly statements, so the compiler neither
sees the MFMAs' latency nor provides the wait states that another instruction
touching their accumulators would need.  Two code-generation outcomes would go
unnoticed by the compiler and give wrong or slow results on the GPU, and are
checked here on the code the build produces:
* an instruction other than the MFMAs reading or writing accumulator registers
  within a few dozen cycles of an MFMA that writes them (register copies the
  allocator inserts when it runs short);
* spill traffic, accumulator copies or a full drain of the vector-memory counter
  inside the K loop (a spilled value reloaded there waits for every load in
  flight).
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2511_12500_amd import build as B

HIPCC = B.HIPCC
SRC = os.path.join(B.CSRC, "gemm_all_scatter.hip")

pytestmark = pytest.mark.skipif(not (os.path.exists(HIPCC) or shutil.which("hipcc")),
                                reason="hipcc not installed")

# gas_kernel<256, 256, BF16, 4 waves, MF = 32, no copy wave, not the reduction kernel>
KERNELS = {
    "bf16": "_ZN12_GLOBAL__N_110gas_kernelILi256ELi256ELb1ELi4ELi32ELb0ELb0EEEvNS_9GasParamsE",
    "f16": "_ZN12_GLOBAL__N_110gas_kernelILi256ELi256ELb0ELi4ELi32ELb0ELb0EEEvNS_9GasParamsE",
}


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("asm") / "gas.s")
    cmd = [HIPCC, *B.CXXFLAGS, "-S", "--cuda-device-only", SRC, "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        return f.read().splitlines()


def function_body(lines, name):
    start = next(i for i, l in enumerate(lines) if l.startswith(name + ":"))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
    return [l.strip() for l in lines[start:end]]


def instructions(body):
    return [l for l in body if l and not l.startswith((";", "."))]


def k_loop(body):
    """The innermost loop holding at least 64 MFMAs (the K loop)."""
    for i, l in enumerate(body):
        m = re.match(r"s_cbranch_\w+ (\.LBB\d+_\d+)", l)
        if not m:
            continue
        j = next(k for k, x in enumerate(body) if x.startswith(m.group(1) + ":"))
        if j < i and sum(x.startswith("v_mfma") for x in body[j:i]) >= 64:
            return body[j:i + 1]
    raise AssertionError("no K loop found")


def accumulator_hazards(body, window=40):
    """Instructions touching an accumulator register that an MFMA wrote fewer
    than `window` issue cycles before (s_nop n counts n + 1), along straight-line
    code (an unconditional branch or the end of the program clears the history)."""
    recent, pos, bad = [], 0, []
    for l in instructions(body):
        if l.startswith("s_nop"):
            pos += int(l.split()[1]) + 1
            continue
        pos += 1
        if re.match(r"s_(branch|setpc|endpgm)\b", l):
            recent = []
            continue
        m = re.match(r"v_mfma\S+ a\[(\d+):(\d+)\]", l)
        if m:
            recent = (recent + [(pos, int(m.group(1)), int(m.group(2)))])[-64:]
            continue
        regs = {int(a) for a in re.findall(r"\ba(\d+)\b", l)}
        for a, b in re.findall(r"a\[(\d+):(\d+)\]", l):
            regs.update(range(int(a), int(b) + 1))
        if any(lo <= r <= hi and pos - p < window for p, lo, hi in recent for r in regs):
            bad.append(l)
    return bad


@pytest.mark.parametrize("dtype", sorted(KERNELS))
def test_no_accumulator_access_next_to_the_mfmas(asm, dtype):
    body = function_body(asm, KERNELS[dtype])
    assert sum(l.startswith("v_mfma") for l in body) >= 64
    assert accumulator_hazards(body) == []


@pytest.mark.parametrize("dtype", sorted(KERNELS))
def test_k_loop_has_no_spills_copies_or_drains(asm, dtype):
    loop = instructions(k_loop(function_body(asm, KERNELS[dtype])))
    ops = [l.split()[0] for l in loop]
    assert sum(o.startswith("v_mfma") for o in ops) == 128        # two 64-k stages
    assert not [o for o in ops if o.startswith(("scratch_", "v_accvgpr", "v_readlane",
                                                  "v_writelane"))]
    waits = [l for l in loop if l.startswith("s_waitcnt")]
    assert not [w for w in waits if re.search(r"vmcnt\(0\)", w)]
    # every staging register goes to LDS only after its own load: exact waits
    assert any(re.search(r"vmcnt\((1[0-9]|[1-9])\)", w) for w in waits)
