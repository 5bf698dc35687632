"""Generated-code checks of the large-group GEMM core (CPU: hipcc cross-compiles).

The core issues its MFMAs as inline asm (so that its accumulators stay in
AGPRs), which hides their write latency from the compiler: the code must not
read, copy or overwrite an accumulator register before the MFMA that writes
it has finished, and the hand-ordered slice loop must not spill.  Both are
properties of the code the compiler emits, so this test compiles gemm.hip for
gfx950 with the library's flags and checks the assembly of the large-group
kernels (and, for the LDS reads and spills, the first core's kernels, whose
fragment reads are inline asm with explicit waits as well):

* no scratch access inside the slice loops (the innermost loops that issue
  MFMAs);
* along every control-flow path from an MFMA, no instruction other than
  another MFMA touches its destination AGPRs within 19 wait states (the
  most a 16-pass XDL MFMA asks of a following VALU access; `s_nop N`
  counts N + 1, every other instruction 1);
* along every path from an LDS read, its destination registers are neither
  read nor written before an lgkmcnt wait shows it landed (the explicit
  waits of the hand-ordered loop are checked this way too).
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_00573_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
KERNELS = {
    "k_ffn_big<0>": "_ZN7trimmoe9k_ffn_bigILi0EEEvNS_7FfnArgsE",
    "k_ffn_big<1>": "_ZN7trimmoe9k_ffn_bigILi1EEEvNS_7FfnArgsE",
    "k_ffn_big<2>": "_ZN7trimmoe9k_ffn_bigILi2EEEvNS_7FfnArgsE",
    "k_exit_big": "_ZN7trimmoe10k_exit_bigENS_8ExitArgsE",
}
WAIT_STATES = 19

pytestmark = pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC),
                                reason="hipcc not available")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    out = tmp_path_factory.mktemp("gemm_asm") / "gemm.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "--cuda-device-only", "-S", os.path.join(CSRC, "gemm.hip"), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def _function(text, name):
    start = text.index(f"\n{name}:") + 1
    end = text.index(".Lfunc_end", start)
    body = []
    for line in text[start:end].splitlines()[1:]:
        line = line.split(";")[0].strip()
        if line and not line.startswith("."):
            body.append(line)
        elif re.match(r"^\.LBB\d+_\d+:", line):
            body.append(line)
    return body


def _agprs(ins):
    regs = set()
    for lo, hi in re.findall(r"\ba\[(\d+):(\d+)\]", ins):
        regs.update(range(int(lo), int(hi) + 1))
    for r in re.findall(r"\ba(\d+)\b", ins):
        regs.add(int(r))
    return regs


def _cfg(body):
    labels = {l[:-1]: i for i, l in enumerate(body) if l.endswith(":")}

    def succ(i):
        ins = body[i]
        op = ins.split()[0] if not ins.endswith(":") else ""
        out = []
        if op.startswith("s_branch") or op.startswith("s_cbranch"):
            out.append(labels[ins.split()[-1]])
        if not (op.startswith("s_branch") or op.startswith("s_endpgm") or
                op.startswith("s_setpc")):
            if i + 1 < len(body):
                out.append(i + 1)
        return out
    return succ


def _hazards(body):
    succ = _cfg(body)
    found = []
    for i, ins in enumerate(body):
        if not ins.startswith("v_mfma"):
            continue
        dst = _agprs(ins.split(",")[0])
        # bounded search over paths: (position, wait states left)
        stack = [(j, WAIT_STATES) for j in succ(i)]
        seen = set()
        while stack:
            j, left = stack.pop()
            if left <= 0 or (j, left) in seen:
                continue
            seen.add((j, left))
            cur = body[j]
            cost = 0
            if not cur.endswith(":"):
                if not cur.startswith("v_mfma") and _agprs(cur) & dst:
                    found.append((i, ins, j, cur))
                    continue
                m = re.match(r"s_nop\s+(\d+)", cur)
                cost = int(m.group(1)) + 1 if m else 1
            for k in succ(j):
                stack.append((k, left - cost))
    return found


def _vgprs(ins):
    regs = set()
    for lo, hi in re.findall(r"\bv\[(\d+):(\d+)\]", ins):
        regs.update(range(int(lo), int(hi) + 1))
    for r in re.findall(r"\bv(\d+)\b", ins):
        regs.add(int(r))
    return regs


_SMEM = ("s_load", "s_buffer_load", "s_memtime", "s_memrealtime", "s_scratch_load", "s_dcache")


def _lds_races(body, limit=4000):
    """Accesses to the destination VGPRs of an LDS read before the read is
    known to have landed.  Along every path from a ds_read the read is known
    to have landed at an `s_waitcnt lgkmcnt(N)` once N or more LDS operations
    were issued after it (LDS operations return in order), or at
    lgkmcnt(0) once a scalar memory operation (which may return out of order)
    was issued; before that, any instruction that reads or writes one of its
    destination registers is a race (the compiler cannot see the inline-asm
    reads' latency, so nothing else orders them)."""
    succ = _cfg(body)
    found = []
    for p, ins in enumerate(body):
        if not ins.startswith("ds_read"):
            continue
        dst = _vgprs(ins.split(",")[0])
        stack = [(j, 0, False, 0) for j in succ(p)]
        seen = set()
        while stack:
            j, after, smem, depth = stack.pop()
            key = (j, min(after, 64), smem)
            if key in seen or depth > limit:
                continue
            seen.add(key)
            cur = body[j]
            if not cur.endswith(":"):
                m = re.search(r"lgkmcnt\((\d+)\)", cur)
                if cur.startswith("s_waitcnt") and m:
                    n = int(m.group(1))
                    if n == 0 or (not smem and after >= n):
                        continue
                if _vgprs(cur) & dst:
                    found.append((p, ins, j, cur))
                    continue
                if cur.startswith("ds_"):
                    after += 1
                elif cur.startswith(_SMEM):
                    smem = True
            for k in succ(j):
                stack.append((k, after, smem, depth + 1))
    return found


def _loops_with_mfma(body):
    """(start, end) index ranges of the innermost loops (a backward branch)
    that issue MFMAs: the slice loops, not the tile loops around them, whose
    per-tile code may spill"""
    labels = {l[:-1]: i for i, l in enumerate(body) if l.endswith(":")}
    loops = []
    for i, ins in enumerate(body):
        if ins.startswith("s_cbranch") or ins.startswith("s_branch"):
            t = labels.get(ins.split()[-1])
            if t is not None and t < i and any(b.startswith("v_mfma") for b in body[t:i]):
                loops.append((t, i))
    return [(s, e) for s, e in loops
            if not any((s2, e2) != (s, e) and s <= s2 and e2 <= e for s2, e2 in loops)]


@pytest.mark.parametrize("kernel", list(KERNELS))
def test_no_spill_in_mfma_loops(asm, kernel):
    body = _function(asm, KERNELS[kernel])
    loops = _loops_with_mfma(body)
    assert loops, "no MFMA loop found"
    for s, e in loops:
        spills = [b for b in body[s:e] if b.startswith("scratch_") or "Spill" in b]
        assert not spills, (kernel, spills[:4])


@pytest.mark.parametrize("kernel", list(KERNELS))
def test_no_early_accumulator_access(asm, kernel):
    body = _function(asm, KERNELS[kernel])
    assert any(b.startswith("v_mfma") for b in body)
    bad = _hazards(body)
    assert not bad, [(kernel, m, a) for _, m, _, a in bad[:4]]


@pytest.mark.parametrize("kernel", list(KERNELS))
def test_lds_reads_land_before_their_registers_are_used(asm, kernel):
    body = _function(asm, KERNELS[kernel])
    bad = _lds_races(body)
    assert not bad, [(kernel, r, a) for _, r, _, a in bad[:4]]


def _first_core(asm):
    # every instance of the first core's kernels (inline-asm fragment reads
    # with explicit waits, MFMAs by builtin)
    names = re.findall(r"^(_ZN7trimmoe\w*k_(?:ffn|exit)_mma\w*):", asm, re.M)
    assert names
    return names


def test_first_core_lds_reads_land_before_use(asm):
    for name in _first_core(asm):
        bad = _lds_races(_function(asm, name))
        assert not bad, [(name, r, a) for _, r, _, a in bad[:4]]


def test_first_core_hot_loops_do_not_spill(asm):
    # the offline argmax variant of the exit tile (Lb1E) is not on the hot path
    for name in _first_core(asm):
        if "k_exit_mma" in name and name.endswith("Lb1EEEvNS_8ExitArgsE"):
            continue
        body = _function(asm, name)
        for s, e in _loops_with_mfma(body):
            spills = [b for b in body[s:e] if b.startswith("scratch_")]
            assert not spills, (name, spills[:4])


def test_race_checker_finds_planted_races():
    ok = ["ds_read_b128 v[0:3], v9", "ds_read_b128 v[4:7], v9 offset:16",
          "s_waitcnt lgkmcnt(1)", "v_mov_b32 v10, v1", "s_endpgm"]
    assert not _lds_races(ok)
    # the wait is one read too weak for the first read
    weak = ["ds_read_b128 v[0:3], v9", "ds_read_b128 v[4:7], v9 offset:16",
            "s_waitcnt lgkmcnt(2)", "v_mov_b32 v10, v1", "s_endpgm"]
    assert _lds_races(weak)
    # a register of a read still in flight written on the way out of a loop
    loop = ["ds_read_b128 v[0:3], v9", ".LBB0_1:", "s_waitcnt lgkmcnt(0)",
            "ds_read_b128 v[0:3], v9", "s_cbranch_scc1 .LBB0_1", "v_sub_u32 v2, s4, 1",
            "s_waitcnt lgkmcnt(0)", "s_endpgm"]
    assert _lds_races(loop)
    # a scalar load in between: only lgkmcnt(0) orders the read
    smem = ["ds_read_b128 v[0:3], v9", "ds_read_b128 v[4:7], v9 offset:16",
            "s_load_dword s0, s[2:3], 0x0", "s_waitcnt lgkmcnt(1)", "v_mov_b32 v10, v1",
            "s_endpgm"]
    assert _lds_races(smem)


def test_checker_finds_a_planted_hazard():
    # a read of an MFMA result right after it, and the same read after wait states
    body = ["v_mfma_f32_16x16x32_bf16 a[0:3], v[0:3], v[4:7], a[0:3]",
            "v_accvgpr_read_b32 v8, a2", "s_endpgm"]
    assert _hazards(body)
    body = ["v_mfma_f32_16x16x32_bf16 a[0:3], v[0:3], v[4:7], a[0:3]",
            "s_nop 7", "s_nop 7", "s_nop 7", "v_accvgpr_read_b32 v8, a2", "s_endpgm"]
    assert not _hazards(body)
    # through a branch to a block that copies the accumulator
    body = ["v_mfma_f32_16x16x32_bf16 a[4:7], v[0:3], v[4:7], a[4:7]",
            "s_branch .LBB0_2", ".LBB0_1:", "s_endpgm", ".LBB0_2:",
            "v_accvgpr_mov_b32 a9, a5", "s_branch .LBB0_1"]
    assert _hazards(body)
