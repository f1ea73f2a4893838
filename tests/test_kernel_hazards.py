"""Wait states after the attention kernel's MFMAs, read from its gfx950 assembly.

The attention kernel issues its MFMAs as inline asm (explicit AGPR / VGPR
operands), so the compiler does not insert the wait states that an MFMA result
needs before another instruction may read or overwrite it.  The kernel relies
on its own s_nop fences and on the distance its schedule puts between an MFMA
and the first use of its result.  This test compiles the kernel to assembly and
follows every control-flow path from each MFMA (branches, fall-through, loop
back-edges) to the first non-MFMA instruction that touches one of the result
registers, counting one wait state per instruction and N+1 per `s_nop N`.
The bar is the length of the kernel's own fence (21 wait states), above what
CDNA3 requires after the longest (16-pass) XDL operation.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2605_16839_amd", "csrc", "attention.hip")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
NEED = 21


def _regs(text: str, kind: str) -> set:
    out = set()
    for m in re.finditer(r"\b%s\[(\d+):(\d+)\]" % kind, text):
        out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\b%s(\d+)\b" % kind, text):
        out.add(int(m.group(1)))
    return out


def _kernels(asm: str):
    for name in sorted(set(re.findall(r"^(_ZN2ca22paged_attention_kernel\w+):", asm, re.M))):
        body = asm[asm.index(name + ":"):asm.index(".Lfunc_end", asm.index(name + ":"))]
        lines, labels = [], {}
        for raw in body.split("\n")[1:]:
            t = raw.split(";")[0].strip()
            if not t:
                continue
            m = re.match(r"^(\.LBB\d+_\d+):", t)
            if m:
                labels[m.group(1)] = len(lines)
            elif not t.startswith("."):
                lines.append(t)
        yield name, lines, labels


def _successors(lines, labels, k):
    t = lines[k]
    op = t.split()[0]
    if op == "s_branch":
        return [labels[t.split()[-1]]]
    if op.startswith("s_cbranch"):
        return [labels[t.split()[-1]], k + 1]
    if op == "s_endpgm":
        return []
    return [k + 1]


def _shortest_use(lines, labels, k):
    """Fewest wait states from MFMA k to a non-MFMA access of its result."""
    dst_text = lines[k].split(None, 1)[1].split(",")[0]
    kind = "a" if dst_text.strip().startswith("a") else "v"
    dst = _regs(dst_text, kind)
    best = None
    stack = [(q, 0) for q in _successors(lines, labels, k)]
    seen = {}
    while stack:
        p, d = stack.pop()
        if p >= len(lines) or d >= NEED or seen.get(p, 1 << 30) <= d:
            continue
        seen[p] = d
        u = lines[p]
        op = u.split()[0]
        if op.startswith("v_mfma"):
            ops = u.split(None, 1)[1].split(",")
            # a later MFMA that reads the result as its A/B operand also waits
            if _regs(",".join(ops[1:3]), kind) & dst:
                best = d if best is None else min(best, d)
                continue
            if _regs(ops[0], kind) >= dst:   # overwritten by an MFMA: chain ends
                continue
        elif op.startswith(("v_", "ds_", "buffer_", "global_", "flat_")) and _regs(u, kind) & dst:
            best = d if best is None else min(best, d)
            continue
        m = re.match(r"s_nop\s+(\d+)", u)
        w = int(m.group(1)) + 1 if m else 1
        for q in _successors(lines, labels, p):
            stack.append((q, d + w))
    return best


@pytest.fixture(scope="module", params=[2, 4])
def attention_asm(request, tmp_path_factory):
    """The kernel's gfx950 assembly as built (two waves per SIMD, 2 column tiles
    per wave) and in its one-wave form (CA_COL_TILES=4)."""
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "attention.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S",
           f"-DCA_COL_TILES={request.param}",
           "-I", os.path.join(ROOT, "include"), "-o", str(out), SRC]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def test_mfma_results_wait_before_use(attention_asm):
    kernels = list(_kernels(attention_asm))
    # D in {64, 128} x {per-group, block-sparse} workgroups x {selected, dense} x
    # V layout in {token-major, transposed}
    assert len(kernels) == 16
    for name, lines, labels in kernels:
        n_mfma = 0
        for k, t in enumerate(lines):
            if not t.startswith("v_mfma"):
                continue
            n_mfma += 1
            d = _shortest_use(lines, labels, k)
            assert d is None, f"{name}: {t} is used after {d} wait states (< {NEED})"
        assert n_mfma >= 64, name


def test_checker_flags_a_missing_fence(tmp_path):
    """The check itself: a copy of the kernel without the fence between the
    masked-page QK MFMAs and the mask that reads their scores (compiled only,
    never run) must be reported, in every instantiation."""
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    src = open(SRC).read()
    fenced = "    qk_page(SA, k_s0);\n    fence_s<NCT>(SA);\n"
    assert src.count(fenced) == 1
    bad = tmp_path / "attention.hip"
    bad.write_text(src.replace(fenced, "    qk_page(SA, k_s0);\n"))
    for f in ("common.hpp", "kernels.hpp"):
        shutil.copy(os.path.join(os.path.dirname(SRC), f), tmp_path / f)
    out = tmp_path / "attention.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S",
           "-I", os.path.join(ROOT, "include"), "-o", str(out), str(bad)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    flagged = {name for name, lines, labels in _kernels(out.read_text())
               for k, t in enumerate(lines) if t.startswith("v_mfma")
               and _shortest_use(lines, labels, k) is not None}
    assert len(flagged) == 16, flagged
