"""Inline asm in the HIP sources stays within what the compiler's hazard
handling does not need to see.

The hardware does not interlock a VALU read of an MFMA result, nor an LDS DMA
that follows an SALU write of M0: the compiler inserts the wait states these
need (12 after v_mfma_f32_32x32x16_{f16,bf16} on gfx950, 1 after the M0
write) for instructions it generates, never inside inline asm.  So asm may
hold only waits, barriers, no-ops, and the direct-to-LDS load with its M0
write and the wait state after it; a vector ALU instruction in asm (such as a
v_max3_f32 of accumulators) would read registers an MFMA may not have written
yet.
"""
import os
import re

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2110_14007_amd", "csrc")
ALLOWED = ("s_waitcnt", "s_barrier", "s_nop", "s_mov_b32", "global_load_lds_dwordx4")


def asm_bodies():
    """(file, asm template string) of every asm statement in the sources."""
    out = []
    for name in sorted(os.listdir(CSRC)):
        if not name.endswith((".h", ".hip")):
            continue
        text = open(os.path.join(CSRC, name)).read()
        text = re.sub(r"//[^\n]*", "", text)  # comments may mention instructions
        for m in re.finditer(r"\basm\s*(?:volatile\s*)?\(\s*((?:\"(?:[^\"\\]|\\.)*\"\s*)+)", text):
            body = "".join(re.findall(r"\"((?:[^\"\\]|\\.)*)\"", m.group(1)))
            out.append((name, body.replace("\\n", "\n").replace("\\t", " ")))
    return out


def test_asm_holds_no_vector_alu():
    bodies = asm_bodies()
    assert bodies, "no asm statements found: the scan is broken"
    for name, body in bodies:
        for line in body.split("\n"):
            op = line.strip().split(" ")[0] if line.strip() else ""
            if not op:
                continue
            assert op in ALLOWED, "%s: asm instruction %r outside the allowed set" % (name, op)
            assert not op.startswith("v_"), (name, op)


def test_m0_write_waits_before_lds_dma():
    seen = 0
    for name, body in asm_bodies():
        ops = [l.strip().split(" ")[0] for l in body.split("\n") if l.strip()]
        for i, op in enumerate(ops):
            if op == "s_mov_b32":
                assert "m0" in body.split("\n")[i], "%s: s_mov_b32 in asm writes only M0" % name
            if op == "global_load_lds_dwordx4":
                seen += 1
                j = ops.index("s_mov_b32") if "s_mov_b32" in ops else -1
                assert 0 <= j < i, "%s: the LDS DMA sets M0 in the same statement" % name
                assert "s_nop" in ops[j + 1:i], "%s: no wait state between M0 write and LDS DMA" % name
    assert seen >= 1
