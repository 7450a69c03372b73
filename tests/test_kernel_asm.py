"""Checks on the gfx950 assembly of the library's kernels, compiled here with the library's own
flags (no GPU needed).

The K-major B fragments of the transposed dW GEMM are read with ds_read_b64_tr_b16 issued as
inline assembly (in the dW kernel and in the launch that runs dhidden and dW together), which
the compiler does not track: the kernel waits for those reads itself
(s_waitcnt lgkmcnt(0)).  On every control-flow path from such a read to the next full LDS
wait, no instruction may read or write the read's destination registers (a copy or a use
before the wait would see stale data).  Packed fp32 VALU instructions are kept out of every
kernel by a compile flag; the assembly is checked for them too.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36932_amd", "csrc")
DWT_KERNEL = "_ZN6fastrl14lm_gemm_kernelItLi3EEEvNS_10GemmParamsE"  # bf16, transposed dW
BWD_KERNEL = "_ZN6fastrl13lm_bwd_kernelENS_10GemmParamsES0_"       # dhidden + transposed dW
KERNELS_WITH_TR_READS = [DWT_KERNEL, BWD_KERNEL]
REG = re.compile(r"\b([va])(\d+)\b|\b([va])\[(\d+):(\d+)\]")
LABEL = re.compile(r"^(\.?[A-Za-z_][\w.$]*):")


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return shutil.which("hipcc")


def _compile(src, tmp_path):
    from paper_2609_36932_amd.build import FLAGS
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc not available")
    out = os.path.join(str(tmp_path), os.path.basename(src) + ".s")
    flags = [f for f in FLAGS if f != "-fPIC"]
    r = subprocess.run([hipcc, *flags, "--cuda-device-only", "-S", src, "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


def _regs(text):
    out = set()
    for m in REG.finditer(text):
        if m.group(1):
            out.add((m.group(1), int(m.group(2))))
        else:
            out.update((m.group(3), i) for i in range(int(m.group(4)), int(m.group(5)) + 1))
    return out


def _body(asm, name):
    i = asm.index(name + ":")
    j = asm.index(".Lfunc_end", i)
    lines = []
    for raw in asm[i:j].split("\n")[1:]:
        line = raw.split(";")[0].rstrip()
        if not line.strip() or line.lstrip().startswith("."):
            m = LABEL.match(line.strip())
            if m:
                lines.append(("label", m.group(1), ""))
            continue
        m = LABEL.match(line.strip())
        if m:
            lines.append(("label", m.group(1), ""))
            continue
        parts = line.split(None, 1)
        lines.append(("inst", parts[0], parts[1] if len(parts) > 1 else ""))
    return lines


def _uses_before_wait(lines, start, dest):
    """Instructions that touch `dest` on some path from lines[start] to a full LDS wait."""
    where = {name: k for k, (kind, name, _) in enumerate(lines) if kind == "label"}
    bad, seen, stack = [], set(), [start + 1]
    while stack:
        k = stack.pop()
        while k < len(lines) and k not in seen:
            seen.add(k)
            kind, op, args = lines[k]
            if kind == "label":
                k += 1
                continue
            if op == "s_waitcnt" and "lgkmcnt(0)" in args:
                break
            if op == "s_endpgm":
                break
            if _regs(args) & dest:
                bad.append(f"{op} {args}")
            if op == "s_branch":
                k = where[args.strip()]
                continue
            if op.startswith("s_cbranch"):
                stack.append(where[args.strip()])
            k += 1
    return bad


def test_checker_finds_early_uses():
    """The path check itself, on hand-written assembly: a copy before the wait is found on the
    fall-through path and behind a branch; uses after the wait are not reported."""
    asm = "\n".join([
        "k:",
        "\tds_read_b64_tr_b16 v[6:7], v2",
        "\ts_cbranch_scc0 .LBB0_2",
        "\tv_add_u32_e32 v3, 1, v3",
        "\ts_waitcnt lgkmcnt(0)",
        "\tv_mov_b32_e32 v9, v6",
        "\ts_endpgm",
        ".LBB0_2:",
        "\tv_mfma_f32_16x16x32_bf16 v[10:13], v[20:23], v[4:7], v[10:13]",
        "\ts_waitcnt lgkmcnt(0)",
        "\ts_endpgm",
        ".Lfunc_end0:"])
    lines = _body(asm, "k")
    bad = _uses_before_wait(lines, 0, _regs("v[6:7]"))
    assert len(bad) == 1 and bad[0].startswith("v_mfma"), bad
    assert _uses_before_wait(lines, 0, _regs("v[30:31]")) == []


@pytest.fixture(scope="module")
def lmhead_asm(tmp_path_factory):
    return _compile(os.path.join(CSRC, "lmhead.hip"), tmp_path_factory.mktemp("asm"))


@pytest.mark.parametrize("kernel", KERNELS_WITH_TR_READS)
def test_transposing_reads_are_waited_for_before_use(lmhead_asm, kernel):
    lines = _body(lmhead_asm, kernel)
    reads = [k for k, (kind, op, _) in enumerate(lines) if op == "ds_read_b64_tr_b16"]
    # two per B fragment, four fragments, three places (prologue, loop, last tile) at least
    assert len(reads) >= 24, len(reads)
    for k in reads:
        dest = _regs(lines[k][2].split(",")[0])
        assert len(dest) == 2, lines[k]
        bad = _uses_before_wait(lines, k, dest)
        assert not bad, (lines[k], bad[:5])


@pytest.mark.parametrize("kernel", KERNELS_WITH_TR_READS)
def test_transposing_read_pairs_fill_one_operand(lmhead_asm, kernel):
    """The two halves of a fragment land in adjacent registers, so the MFMA reads them in
    place (no copy that could run before the data arrives)."""
    lines = _body(lmhead_asm, kernel)
    dests = [sorted(_regs(args.split(",")[0])) for kind, op, args in lines
             if op == "ds_read_b64_tr_b16"]
    mfma_b = set()
    for kind, op, args in lines:
        if op.startswith("v_mfma"):
            mfma_b.add(tuple(sorted(_regs(args.split(",")[2]))))
    for d in dests:
        assert any(set(d) <= set(b) for b in mfma_b), d


@pytest.mark.parametrize("src", ["lmhead.hip", "optim.hip", "prune.hip", "advantage.hip"])
def test_no_packed_fp32_valu(src, tmp_path):
    asm = _compile(os.path.join(CSRC, src), tmp_path)
    found = re.findall(r"\bv_pk_(?:add|mul|fma|mov)_f32\b", asm)
    assert not found, found[:5]
