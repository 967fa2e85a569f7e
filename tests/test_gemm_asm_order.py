"""Register-safety checks of the 4-wave GEMM main loop, on its gfx950 assembly.

The 4-wave GEMM kernels (`gemm_f16_kernel<256, 256, 2, 2, ...>`) issue their
fragment reads, MFMAs and counter waits as ordered asm statements while the
compiler still allocates the registers.  Two things the compiler cannot see
are checked here on the assembly it generates for this build (no GPU needed):

  * an LDS read issued by asm is, to the compiler, complete at once: no other
    instruction may read, write or copy one of its destination registers
    before an `s_waitcnt lgkmcnt(0)` covers it (only MFMAs consume them);
  * MFMAs issued by asm are outside the compiler's hazard checks: no
    instruction other than an MFMA may touch an accumulator register (AGPR) on
    any control-flow path from an MFMA until the wait-state statement (a run
    of at least four `s_nop 7`).

A check that fails means a compiler change moved code into one of these
windows: the kernels would then read registers whose values have not landed.
"""

import collections
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_10415_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
KERNEL = "gemm_f16_kernelILi256ELi256ELi2ELi2E"   # the 4-wave instantiations


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("asm") / "gemm_f16.s")
    subprocess.run([HIPCC, "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "--cuda-device-only", "-S",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-Wno-unused-command-line-argument", "-x", "hip", os.path.join(CSRC, "gemm_f16.hip"),
                    "-o", out], check=True, capture_output=True)
    lines = open(out).read().split("\n")
    found = {}
    for i, line in enumerate(lines):
        if line.startswith("_Z") and KERNEL in line and line.split()[0].endswith(":"):
            end = next(j for j in range(i, len(lines)) if lines[j].startswith(".Lfunc_end"))
            found[line.split(":")[0]] = lines[i + 1:end]
    return found


def _regs(tok, kind="v"):
    m = re.match(kind + r"\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(kind + r"(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def _instructions(body):
    return [x.strip() for x in body if x.strip() and not x.strip().startswith((";", "."))]


def _blocks(body):
    blocks = collections.OrderedDict()
    cur = "entry"
    blocks[cur] = []
    for x in body:
        m = re.match(r"^(\.LBB\d+_\d+):", x)
        if m:
            cur = m.group(1)
            blocks[cur] = []
            continue
        t = x.strip()
        if t and not t.startswith((";", ".")):
            blocks[cur].append(t)
    return blocks


def test_all_four_wave_instantiations_present(kernels):
    # forward, data and weight gradients, the two fused epilogues and the
    # split-K partial tiles
    tags = {"Lb0ELb1ELi0E", "Lb0ELb0ELi0E", "Lb1ELb0ELi0E", "Lb0ELb1ELi1E", "Lb0ELb0ELi2E", "Lb1ELb0ELi3E"}
    names = " ".join(kernels)
    missing = [t for t in tags if t not in names]
    assert not missing, missing


def test_no_instruction_touches_a_pending_lds_read_register(kernels):
    bad = []
    for name, body in kernels.items():
        # program order, the whole kernel, then its loop bodies once more
        # (a loop's reads land in its next iteration)
        ins = _instructions(body)
        loops = [b for b in _blocks(body).values() if sum(t.startswith("v_mfma") for t in b) >= 64]
        for seq in [ins] + [b + b for b in loops]:
            pending = set()
            for t in seq:
                op = t.split()[0]
                if op == "s_waitcnt" and "lgkmcnt(0)" in t:
                    pending = set()
                    continue
                if op.startswith("ds_read"):
                    pending |= _regs(t.split()[1].rstrip(","))
                    continue
                if op.startswith(("v_mfma", "s_", "buffer_")):
                    continue
                for tok in t.split()[1:]:
                    if _regs(tok.rstrip(",")) & pending:
                        bad.append((name[-60:], t))
    assert not bad, bad[:5]


def test_no_accumulator_read_between_an_mfma_and_the_wait_states(kernels):
    bad = []
    for name, body in kernels.items():
        blocks = _blocks(body)
        names = list(blocks)
        succ = {}
        for k, b in enumerate(names):
            ins = blocks[b]
            s = [t.split()[1] for t in ins if t.startswith(("s_cbranch", "s_branch"))]
            if not ins or not ins[-1].startswith("s_branch"):
                if k + 1 < len(names):
                    s.append(names[k + 1])
            succ[b] = s
        for b in names:
            ins = blocks[b]
            mf = [k for k, t in enumerate(ins) if t.startswith("v_mfma")]
            if not mf:
                continue
            work, seen = [(b, mf[-1] + 1)], set()
            while work:
                blk, start = work.pop()
                stop, nops = False, 0
                for t in blocks[blk][start:]:
                    if t.startswith("v_mfma"):
                        stop = True
                        break
                    if t.startswith("s_nop 7"):
                        nops += 1
                        if nops >= 4:
                            stop = True
                            break
                    elif re.search(r"\ba\[?\d", t):
                        bad.append((name[-60:], blk, t))
                if stop:
                    continue
                for n in succ[blk]:
                    if n not in seen:
                        seen.add(n)
                        work.append((n, 0))
    assert not bad, bad[:5]
