"""The library's inline assembly must not write SCC (CPU only).

The compiler does not know that an asm statement changes the scalar condition code, so it
may place one between its own SCC producer and consumer: the low and high halves of a
64-bit address add (a lost carry puts the address 4 GiB too low) or a compare and the
branch that ends a loop (a kernel that never leaves its loop). This scans every asm
statement in the HIP sources and allows only instructions that leave SCC unchanged."""
import glob
import os
import re

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                    "paper_2608_06690_amd", "csrc")
# mnemonics (or prefixes) that never write SCC
ALLOWED = ("s_mov_b32", "s_nop", "s_waitcnt", "s_barrier", "global_load_lds_", "v_mfma", "v_accvgpr")


def asm_statements(src):
    for m in re.finditer(r"\basm\s+(?:volatile\s*)?\(", src):
        i, depth = m.end(), 1
        while depth:
            depth += {"(": 1, ")": -1}.get(src[i], 0)
            i += 1
        body = src[m.end():i - 1]
        template = body.split(":")[0]
        yield "".join(re.findall(r'"((?:[^"\\]|\\.)*)"', template))


def test_inline_asm_leaves_scc_alone():
    seen = 0
    for path in sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.h"))):
        for tmpl in asm_statements(open(path).read()):
            for ins in re.split(r"\\n|\n|;", tmpl):
                ins = ins.replace("\\t", " ").strip()
                if not ins:
                    continue
                seen += 1
                assert ins.startswith(ALLOWED), f"{os.path.basename(path)}: '{ins}' may write SCC"
    assert seen >= 5  # the copies, waits and barriers were found


def test_scanner_flags_an_scc_writer():
    src = 'asm volatile("s_add_u32 m0, %2, %3\\n\\ts_nop 0" :: "s"(a), "n"(1) : "m0");'
    ins = [i.replace("\\t", " ").strip() for t in asm_statements(src) for i in re.split(r"\\n", t)]
    assert ins[0].startswith("s_add_u32") and not ins[0].startswith(ALLOWED)
