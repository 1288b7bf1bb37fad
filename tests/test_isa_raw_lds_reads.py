"""The weight-gradient kernels read their LDS-DMA stages with transposing LDS
reads (ds_read_b64_tr_b16) issued as inline assembly.  The compiler does not
know that such a read fills its destination registers later, so correctness
rests on every destination register being left alone (neither read nor
written) until an s_waitcnt lgkmcnt that covers the read.  This test compiles
the GEMM source for gfx950 to assembly on the CPU and proves that property for
every kernel holding such reads, by a forward dataflow pass over each kernel's
control-flow graph.  (The register-staged variants issue the same instruction
through the compiler's builtin, which places its own waits; the pass covers
those kernels too.)

Abstract state: the LDS operations that may still be outstanding, newest
first, each with the registers it will fill.  LDS operations complete in
issue order, so after s_waitcnt lgkmcnt(N) at most the N newest ones can be
outstanding (scalar-memory and message operations also count towards lgkmcnt
but only lower the number of LDS operations that can still be pending, so
ignoring them keeps the model sound).  At a join the states are merged
position by position by union."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_1910_13444_amd import build

RAW_READ = "ds_read_b64_tr_b16"
_REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")
_LABEL = re.compile(r"^(\.L\w+):")
_LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def _regs(text):
    out = set()
    for m in _REG.finditer(text):
        if m.group(3) is not None:
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return frozenset(out)


def _blocks(lines):
    """Split a kernel body into basic blocks: (label or None, instructions,
    successor labels, falls through)."""
    blocks, cur, label = [], [], None

    def close(succ, falls):
        nonlocal cur, label
        blocks.append((label, cur, succ, falls))
        cur, label = [], None

    for raw in lines:
        line = raw.split(";")[0].strip()
        if not line or line.startswith("."):
            m = _LABEL.match(line)
            if m:
                if cur or label is not None:
                    close([], True)
                label = m.group(1)
            continue
        op = line.split()[0]
        cur.append(line)
        if op == "s_branch":
            close([line.split()[1]], False)
        elif op.startswith("s_cbranch_"):
            close([line.split()[1]], True)
        elif op in ("s_endpgm", "s_setpc_b64"):
            assert op == "s_endpgm", f"indirect branch not modelled: {line!r}"
            close([], False)
    if cur or label is not None:
        close([], False)
    return blocks


def _join(a, b):
    n = max(len(a), len(b))
    return tuple((a[i] if i < len(a) else frozenset()) | (b[i] if i < len(b) else frozenset()) for i in range(n))


_CAP = 32   # deeper entries are merged; lgkmcnt never names more than 15


def _step(state, line, where):
    """Transfer one instruction; raise if it touches a pending register."""
    op = line.split()[0]
    if op.startswith("s_waitcnt"):
        m = _LGKM.search(line)
        return state[:int(m.group(1))] if m else state
    if op.startswith("s_"):
        return state
    pending = frozenset().union(*state) if state else frozenset()
    touched = _regs(line[len(op):])
    if touched & pending:
        raise AssertionError(f"{where}: register(s) v{sorted(touched & pending)} of an LDS read still "
                             f"in flight are touched by {line!r}")
    if op.startswith("ds_"):
        fills = _regs(line[len(op):].split(",")[0]) if op == RAW_READ else frozenset()
        state = (fills,) + state
        if len(state) > _CAP:
            state = state[:_CAP - 1] + (frozenset().union(*state[_CAP - 1:]),)
    return state


def check_kernel(name, lines):
    """Number of raw reads proven safe in one kernel body (raises on a hazard).

    Only the raw reads' registers are tracked: the compiler accounts for the
    LDS operations it emits itself."""
    blocks = _blocks(lines)
    index = {b[0]: i for i, b in enumerate(blocks) if b[0] is not None}
    preds = [[] for _ in blocks]
    for i, (_, _, succ, falls) in enumerate(blocks):
        for s in succ:
            assert s in index, f"{name}: branch to unknown label {s}"
            preds[index[s]].append(i)
        if falls and i + 1 < len(blocks):
            preds[i + 1].append(i)
    out = [None] * len(blocks)
    work = list(range(len(blocks)))
    while work:
        i = work.pop(0)
        st = ()
        for p in preds[i]:
            if out[p] is not None:
                st = _join(st, out[p])
        for line in blocks[i][1]:
            st = _step(st, line, f"{name} block {blocks[i][0] or i}")
        if st != out[i]:
            out[i] = st
            _, _, succ, falls = blocks[i]
            nxt = [index[s] for s in succ] + ([i + 1] if falls and i + 1 < len(blocks) else [])
            work.extend(j for j in nxt if j not in work)
    return sum(line.startswith(RAW_READ) for b in blocks for line in b[1])


def _kernels(asm):
    for m in re.finditer(r"^(_Z\w+):", asm, re.M):
        end = asm.find(".Lfunc_end", m.end())
        body = asm[m.end():end]
        if RAW_READ in body:
            yield m.group(1), body.split("\n")


def test_checker_finds_planted_hazards():
    """The checker itself, on small hand-written fragments."""
    ok = ["ds_read_b64_tr_b16 v[0:1], v10", "ds_read_b64_tr_b16 v[2:3], v11",
          "ds_write_b32 v12, v13", "s_waitcnt lgkmcnt(1)",
          "v_mfma_f32_32x32x16_bf16 v[20:35], v[0:3], v[4:7], v[20:35]", "s_endpgm"]
    assert check_kernel("ok", ok) == 2
    # the partial wait releases only the reads issued before the newest one
    partial = ["ds_read_b64_tr_b16 v[0:1], v10", "ds_read_b64_tr_b16 v[2:3], v11",
               "s_waitcnt lgkmcnt(1)", "v_add_f32 v4, v2, v5", "s_endpgm"]
    with pytest.raises(AssertionError, match="in flight"):
        check_kernel("partial", partial)
    # an overwrite before the wait is a hazard too
    with pytest.raises(AssertionError, match="in flight"):
        check_kernel("waw", ["ds_read_b64_tr_b16 v[0:1], v10", "v_mov_b32 v1, 0", "s_waitcnt lgkmcnt(0)", "s_endpgm"])
    # a wait on one path only does not cover the join
    branchy = ["ds_read_b64_tr_b16 v[0:1], v10", "s_cbranch_vccz .LBB0_2",
               "s_waitcnt lgkmcnt(0)", ".LBB0_2:", "v_add_f32 v4, v0, v5", "s_endpgm"]
    with pytest.raises(AssertionError, match="in flight"):
        check_kernel("branchy", branchy)
    # a loop whose back edge carries an unwaited read into the use at its head
    loop = ["s_branch .LBB0_2", ".LBB0_1:", "v_add_f32 v4, v0, v5", "s_waitcnt lgkmcnt(0)",
            ".LBB0_2:", "ds_read_b64_tr_b16 v[0:1], v10", "s_cbranch_scc1 .LBB0_1", "s_waitcnt lgkmcnt(0)", "s_endpgm"]
    with pytest.raises(AssertionError, match="in flight"):
        check_kernel("loop", loop)


def test_raw_transposing_reads_are_waited_for():
    hipcc = build.hipcc()
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    d = tempfile.mkdtemp()
    try:
        out = os.path.join(d, "gemm.s")
        r = subprocess.run([hipcc, *build.common_flags(), "--cuda-device-only", "-S",
                            os.path.join(build.CSRC, "gemm.hip"), "-o", out], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        with open(out) as f:
            asm = f.read()
    finally:
        shutil.rmtree(d, ignore_errors=True)
    kernels = dict(_kernels(asm))
    assert any("k_gemm_dw_tr" in k for k in kernels), "no kernel with raw transposing reads found"
    for name, lines in kernels.items():
        assert check_kernel(name, lines) > 0
