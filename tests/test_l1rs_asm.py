"""The bf16 row-split first layer issues its stage memory operations (W1 and
feature-row DMAs into LDS, the next tile's ID loads) from inline assembly and
waits for them with explicit s_waitcnt counts, so the compiler does not know
that the ID registers are still being written.  This test compiles embed.hip
for gfx950 and checks, on the generated assembly, what that design relies on:

  * no instruction reads or writes a register that an inline-assembly load
    has not finished writing (simulating the in-order vector-memory queue in
    program order, and the loop bodies a second time for their back edges);
  * no spill (scratch) access and no other vector-memory wait inside the
    stage code, where it would not be counted;
  * one explicit wait per stage, with the counts the issue order needs.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_1711_06505_amd", "csrc", "embed.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
KERNEL = "_ZN12_GLOBAL__N_19l1rs_bf16"
REG = re.compile(r"\b([va])\[(\d+):(\d+)\]|\b([va])(\d+)\b")


def rs_constant(name):
    """A compile-time constant of the kernel (namespace rs in embed.hip)."""
    text = open(SRC).read()
    ns = text[text.index("namespace rs {"):]
    m = re.search(rf"constexpr int {name} = (\d+);", ns[:ns.index("}  // namespace rs")])
    return int(m.group(1))


def regs_of(text):
    out = set()
    for m in REG.finditer(text):
        if m.group(1):
            out.update((m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1))
        else:
            out.add((m.group(4), int(m.group(5))))
    return out


@pytest.fixture(scope="module")
def kernel_asm(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "embed.s"
    cmd = [HIPCC, "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "--cuda-device-only", "-S", SRC, "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    lines = out.read_text().splitlines()
    start = next(i for i, l in enumerate(lines) if re.match(rf"^{KERNEL}\S*:", l))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
    return lines[start:end]


def parse(lines):
    body, in_asm, flag = [], [], False
    for l in lines:
        if ";;#ASMSTART" in l:
            flag = True
        elif ";;#ASMEND" in l:
            flag = False
        body.append(l.split(";")[0].strip())
        in_asm.append(flag)
    return body, in_asm


def simulate(body, in_asm, seq, queue, errors):
    """In-order vector-memory queue: (destination registers, text) per op."""
    for idx in seq:
        ins = body[idx]
        if not ins or ins.endswith(":") or ins.startswith("."):
            continue
        op = ins.split()[0]
        m = re.match(r"s_waitcnt\s+.*vmcnt\((\d+)\)", ins)
        if m:
            del queue[:max(0, len(queue) - int(m.group(1)))]
            continue
        if op.startswith("s_waitcnt"):
            continue
        touched = regs_of(ins[len(op):])
        for dst, text in queue:
            if dst & touched:
                errors.append(f"{idx}: '{ins}' touches the registers of in-flight '{text}'")
        if op.startswith(("global_", "buffer_", "scratch_", "flat_")):
            tracked = in_asm[idx] and "load" in op and "lds" not in op
            queue.append((regs_of(ins[len(op):].split(",")[0]) if tracked else set(), ins))
    return queue


def test_no_register_is_touched_before_its_load_lands(kernel_asm):
    body, in_asm = parse(kernel_asm)
    errors = []
    simulate(body, in_asm, range(len(body)), [], errors)
    labels = {l[:-1]: i for i, l in enumerate(body) if l.endswith(":")}
    for i, ins in enumerate(body):
        m = re.match(r"s_cbranch_\w+\s+(\S+)", ins)
        if m and m.group(1) in labels and labels[m.group(1)] < i:
            a = labels[m.group(1)]
            q = simulate(body, in_asm, range(0, a), [], [])
            q = simulate(body, in_asm, range(a, i + 1), q, [])
            simulate(body, in_asm, range(a, i + 1), q, errors)      # the back edge
    assert not errors, "\n".join(sorted(set(errors))[:20])


def test_stage_code_has_no_spills_and_only_the_explicit_waits(kernel_asm):
    body, in_asm = parse(kernel_asm)
    dmas = [i for i, l in enumerate(body) if l.startswith("global_load_lds_dwordx4") and in_asm[i]]
    first, last = dmas[0], dmas[-1]
    region = body[first:last + 1]
    assert not [l for l in region if l.startswith("scratch_")]
    waits = [l for l in region if re.match(r"s_waitcnt\s+.*vmcnt", l)]
    stages = rs_constant("kF") // rs_constant("KS")
    dma, wait, wait_ids = rs_constant("DMA"), rs_constant("WAIT"), rs_constant("WAIT_AFTER_IDS")
    plain = [w for w in waits if f"vmcnt({wait})" in w]
    after_ids = [w for w in waits if f"vmcnt({wait_ids})" in w]
    # every stage waits once: the stage after the ID loads with the larger count
    assert len(plain) == stages - 1 and len(after_ids) == 1 and len(waits) == stages, set(waits)
    assert all("lgkmcnt(0)" in w for w in waits)
    # the prologue's three slots (rows, W1, rows) and two slots per stage
    assert len(dmas) == 3 * dma + 2 * dma * stages
    # the next tile's four ID loads, once per tile, from inline assembly
    ids = [i for i in range(first, last + 1) if body[i].startswith("global_load_dword ") and in_asm[i]]
    assert len(ids) == 4
