"""Checks on the generated gfx950 code of the prepared-path attention kernel
(CPU only: hipcc cross-compiles the kernels to assembly).

The kernel issues its score MFMAs and its LDS tile copies as inline assembly,
which the compiler's hazard recognizer and register allocator do not see.
These tests check the properties that make that safe on the code the
compiler actually produced:
  * no instruction reads or overwrites an MFMA's result registers, or
    overwrites its accumulator input, within the 12 wait states an 8-pass
    MFMA needs -- for the inline MFMAs and the compiler's own alike;
  * no instance spills (no scratch memory instruction anywhere), so the
    copy-count waits see only the copies;
  * no VALU instruction writes an SGPR that a tile copy reads within the 5
    wait states such a read needs;
  * M0, which the copies set without saving it, is used by nothing else.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_35110_amd import build as pkg_build

SRC = os.path.join(pkg_build.CSRC, "sol_kernels.hip")
WAIT_STATES = 12  # an 8-pass XDL MFMA result, VALU read or write


@pytest.fixture(scope="module")
def asm_text(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    flags = [f for f in pkg_build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    out = str(tmp_path_factory.mktemp("asm") / "sol_kernels.s")
    cmd = [hipcc] + flags + ["--cuda-device-only", "-S", "-I", pkg_build.INCLUDE, "-I", pkg_build.CSRC,
                             "-x", "hip", SRC, "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    return open(out).read()


def functions(text, name):
    """(mangled name, body lines) of every function whose name contains `name`."""
    out = []
    for m in re.finditer(r"^(\S*%s\S*):\s*(;.*)?$" % re.escape(name), text, re.M):
        end = text.index(".Lfunc_end", m.end())
        out.append((m.group(1), text[m.end():end].split("\n")))
    return out


def instructions(lines):
    """[(text, in_inline_asm)] without comments, directives and labels."""
    res, in_asm = [], False
    for ln in lines:
        if ";;#ASMSTART" in ln:
            in_asm = True
            continue
        if ";;#ASMEND" in ln:
            in_asm = False
            continue
        t = ln.split(";")[0].strip()
        if not t or t.startswith(".") or t.endswith(":"):
            continue
        res.append((t, in_asm))
    return res


def regs(tok):
    m = re.match(r"([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def operands(t):
    return [x.strip() for x in t.split(None, 1)[1].split(",")] if " " in t else []


STORE_PREFIXES = ("ds_write", "global_store", "buffer_store", "scratch_store", "flat_store")


N_INSTANCES = 20  # (rope, pass, sparse, records, output records) combinations launched


def template_args(name):
    """(kRope, kRobust, kSparse, kRec, kOutRec) of an attn_prepared_kernel instance
    from its mangled name."""
    m = re.search(r"attn_prepared_kernelILb(\d)ELb(\d)ELb(\d)ELb(\d)ELb(\d)EE", name)
    assert m, name
    return tuple(bool(int(x)) for x in m.groups())


def test_mfma_latency_respected(asm_text):
    """Every MFMA of the twenty kernels (rotary or not, first or second pass,
    dense or block-sparse, queries from bf16 or from records, output records
    or not), inline or not:
    the compiler's own hazard handling is checked too (it once let a spill
    reload overwrite an accumulator still being read)."""
    kernels = functions(asm_text, "attn_prepared_kernel")
    assert len(kernels) == N_INSTANCES
    for name, body in kernels:
        ins = instructions(body)
        n_asm = 0
        for i, (t, in_asm) in enumerate(ins):
            if not t.startswith("v_mfma"):
                continue
            n_asm += in_asm
            ops = operands(t)
            dst, srcc = regs(ops[0]), regs(ops[3])
            ws = 0
            for t2, _ in ins[i + 1:]:
                if ws >= WAIT_STATES:
                    break
                m = re.match(r"s_nop (\d+)", t2)
                if m:
                    ws += int(m.group(1)) + 1
                    continue
                ws += 1
                if t2.startswith("s_"):
                    continue  # scalar code touches no VGPRs
                if t2.startswith("v_mfma"):
                    # a chained MFMA (same accumulator) is interlocked; any
                    # other use of the result as an operand is not
                    o2 = operands(t2)
                    assert not ((regs(o2[1]) | regs(o2[2])) & dst), "%s: %r reads %r" % (name, t2, t)
                    assert regs(o2[3]) == dst or not (regs(o2[3]) & dst), "%s: %r" % (name, t2)
                    continue
                ops2 = operands(t2)
                if not ops2:
                    continue
                if t2.startswith(STORE_PREFIXES):
                    written, read = set(), set().union(*(regs(x) for x in ops2))
                elif t2.endswith(" lds"):  # a copy into LDS: its operand is an address
                    written, read = set(), set().union(*(regs(x) for x in ops2))
                else:
                    written, read = regs(ops2[0]), set().union(set(), *(regs(x) for x in ops2[1:]))
                assert not (written & (dst | srcc)), "%s: %r overwrites registers of %r" % (name, t2, t)
                assert not (read & dst), "%s: %r reads the result of %r too early" % (name, t2, t)
        assert n_asm >= 32, "%s: expected the score MFMAs as inline assembly" % name


def test_no_instance_spills(asm_text):
    """No scratch memory anywhere in the attention kernels.  A kernel that
    spills issues memory instructions the inline copies' waits do not count,
    and spill code beside the inline MFMAs is where generated-code hazards
    have appeared (a build whose instance spilled 41 reloads returned wrong
    row blocks); the register budget is checked here instead of trusted."""
    kernels = functions(asm_text, "attn_prepared_kernel")
    assert len(kernels) == N_INSTANCES
    for name, body in kernels:
        ins = instructions(body)
        assert not any(t.startswith("scratch_") for t, _ in ins), "%s spills" % name
        assert not any(re.match(r"(buffer|global)_(load|store)\S* .*\boff, s\[0:3\]", t) for t, _ in ins), name


def sregs(tok):
    m = re.match(r"s\[(\d+):(\d+)\]$", tok.strip())
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"s(\d+)$", tok.strip())
    return {int(m.group(1))} if m else set()


def test_copy_sgprs_not_written_by_valu_just_before(asm_text):
    """A vector-memory instruction reading an SGPR that a VALU instruction
    (v_readfirstlane, a compare) wrote needs 5 wait states between them; the
    compiler inserts them for its own instructions, not for the tile copies
    written as inline assembly, whose offset and resource operands it
    computes."""
    for name, body in functions(asm_text, "attn_prepared_kernel"):
        ins = instructions(body)
        for i, (t, in_asm) in enumerate(ins):
            if not (t.startswith("buffer_load") and t.endswith(" lds")):
                continue
            used = set().union(*(sregs(o) for o in operands(t)))
            ws = 0
            for t2, _ in reversed(ins[max(0, i - 40):i]):
                m = re.match(r"s_nop (\d+)", t2)
                ws += int(m.group(1)) + 1 if m else 1
                if ws > 5:
                    break
                if t2.startswith("v_") and operands(t2):
                    assert not (sregs(operands(t2)[0]) & used), "%s: %r then %r" % (name, t2, t)


def test_m0_used_only_by_tile_copies(asm_text):
    kernels = functions(asm_text, "attn_prepared_kernel")
    assert len(kernels) == N_INSTANCES
    implicit_m0 = ("s_movrel", "v_movrel", "s_sendmsg", "ds_gws", "v_interp", "ds_append", "ds_consume",
                   "ds_ordered", "s_setreg")
    for name, body in kernels:
        ins = instructions(body)
        copies = 0
        for i, (t, in_asm) in enumerate(ins):
            assert not t.startswith(implicit_m0), "%s: %r uses M0" % (name, t)
            if re.search(r"\bm0\b", t):
                assert in_asm and re.match(r"s_mov_b32 m0, s\d+$", t), "%s: %r" % (name, t)
                assert ins[i + 1][0] == "s_nop 0" and ins[i + 2][0].startswith("buffer_load_dwordx4"), name
            if t.startswith(("buffer_load", "global_load")) and t.endswith(" lds"):
                assert in_asm and re.match(r"s_mov_b32 m0, s\d+$", ins[i - 2][0]), "%s: %r" % (name, t)
                copies += 1
        assert copies >= 12, name


def test_first_pass_copy_count_waits_see_only_copies(asm_text):
    """The closing barrier's vmcnt(4) (a vmcnt(4) wait right before
    s_barrier; vmcnt(12) in the block-sparse walk) assumes the last four (twelve)
    vector-memory instructions of the wave are its tile copies: between the previous vmcnt wait and such a barrier wait
    the compiler must issue no load, store or spill of its own.  (Its own
    vmcnt waits for its own loads, e.g. in the prologue, wait for at least as
    much as they need: the counter retires in order.)"""
    kernels = functions(asm_text, "attn_prepared_kernel")
    assert len(kernels) == N_INSTANCES
    for name, body in kernels:
        ins = instructions(body)
        since, n_waits = [], 0
        for i, (t, in_asm) in enumerate(ins):
            if t.startswith(("buffer_", "global_", "flat_")):
                since.append((t, in_asm))
            if t.startswith("s_waitcnt") and "vmcnt" in t:
                # the dense walk leaves its four copies in flight, the sparse walk twelve
                want = "vmcnt(12)" if template_args(name)[2] else "vmcnt(4)"
                if want in t and i + 1 < len(ins) and ins[i + 1][0] == "s_barrier":
                    n_waits += 1
                    others = [x for x, a in since if not (a and x.endswith(" lds"))]
                    assert not others, "%s: %r before a copy-count wait" % (name, others[:3])
                since = []
        assert n_waits >= 2, name


def _vregs(text):
    """VGPR and AGPR names (v12, a3, ...) in an operand list."""
    out = set()
    for m in re.finditer(r"\b([va])(\d+)\b", text):
        out.add(m.group(1) + m.group(2))
    for m in re.finditer(r"\b([va])\[(\d+):(\d+)\]", text):
        out.update(m.group(1) + str(r) for r in range(int(m.group(2)), int(m.group(3)) + 1))
    return out


def test_loaded_registers_read_after_their_vmcnt_wait(asm_text):
    """A register that a vector-memory load writes is read only after a vmcnt
    wait that retires the load, counting every vector-memory instruction
    issued after it -- the inline-asm tile copies included, which the
    compiler's own wait insertion does not see.  (The counter retires in
    order, so a wait the compiler places for its own loads is at least as
    strict as it needs; this checks that on the generated code, in program
    order within each instance.)"""
    for name, body in functions(asm_text, "attn_prepared_kernel"):
        pending = []  # vector-memory instructions in issue order: (index, registers it loads)
        for i, (t, _) in enumerate(instructions(body)):
            op = t.split()[0]
            ops = operands(t)
            if op == "s_waitcnt":
                m = re.search(r"vmcnt\((\d+)\)", t)
                if m and len(pending) > int(m.group(1)):
                    pending = pending[len(pending) - int(m.group(1)):]
                continue
            if ops:
                reads = _vregs(",".join(ops if op.startswith(STORE_PREFIXES) else ops[1:]))
                for j, dst in pending:
                    assert not (dst & reads), "%s: %r reads a register loaded by instruction %d before its wait" % (
                        name, t, j)
            if op.startswith(("buffer_", "global_", "scratch_", "flat_")):
                loads = "load" in op and not t.endswith(" lds")
                pending.append((i, _vregs(ops[0]) if loads else set()))
