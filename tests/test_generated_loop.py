"""The hand-scheduled key loops (head dims 128 and 64): the committed
assembly is what the generator writes, and the generator's own checks hold
and catch planted mistakes (CPU only)."""
import importlib.util
import os

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2607_15650_amd", "csrc")


def load_gen():
    spec = importlib.util.spec_from_file_location("gen_attn_loop", os.path.join(CSRC, "gen_attn_loop.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def committed_body(d):
    text = open(os.path.join(CSRC, f"attn_d{d}_loop.inc")).read()
    head = f'#define DITANGO_D{d}_LOOP_ASM \\\n  "'
    start = text.index(head) + len(head)
    end = text.index('\\n"\n', start)
    return text[start:end].split("\\n\\t")


@pytest.mark.parametrize("d", [128, 64])
def test_committed_loop_matches_generator(d):
    g = load_gen()
    g.configure(d)
    assert committed_body(d) == g.generate()


@pytest.mark.parametrize("d", [128, 64])
def test_generated_loop_passes_its_checks(d):
    g = load_gen()
    g.configure(d)
    lines = g.generate()
    assert g.check_hazards(lines) == []
    assert g.check_fragments(lines) == []
    mfma = [x for x in lines if x.startswith("v_mfma")]
    # scores of tile 0, four unrolled iterations, four last iterations:
    # 2 MFMAs per fragment step; D/8 score steps and D/8 P V steps per tile
    steps = d // 8
    assert len(mfma) == 2 * (steps + 4 * 2 * steps + 4 * steps)
    # every scalar register the block writes is declared scratch or is a pinned in/out operand
    written = set()
    for x in lines:
        op = x.split()[0]
        if op.startswith("s_") and op not in ("s_waitcnt", "s_barrier", "s_branch", "s_nop", "s_setpc_b64") \
                and not op.startswith(("s_cbranch", "s_cmp")):
            dst = x.split()[1].rstrip(",")
            if dst.startswith("s["):
                lo, hi = dst[2:-1].split(":")
                written |= set(range(int(lo), int(hi) + 1))
            elif dst.startswith("s") and dst[1:].isdigit():
                written.add(int(dst[1:]))
    allowed = set(g.SCRATCH_SGPRS) | set(range(g.S_KD, g.S_KD + 4)) | set(range(g.S_VD, g.S_VD + 4))
    assert written <= allowed, sorted(written - allowed)


def test_checks_catch_a_buffer_refilled_too_early():
    g = load_gen()
    old = g.LA
    try:
        g.LA = g.NFRAG          # the read of step f+8 lands in step f's buffer
        probs = g.check_fragments(g.generate())
    finally:
        g.LA = old
    assert any("reread" in p for p in probs)


def test_checks_catch_a_wait_that_leaves_a_read_outstanding():
    g = load_gen()
    lines = g.generate()
    # weaken the first wait of the steady loop by one
    k = next(i for i, x in enumerate(lines) if x.startswith(".Lloop"))
    w = next(i for i in range(k, len(lines)) if lines[i].startswith("s_waitcnt lgkmcnt("))
    n = int(lines[w].split("(")[1].rstrip(")"))
    lines[w] = f"s_waitcnt lgkmcnt({n + 1})"
    assert any("outstanding" in p for p in g.check_fragments(lines))


def test_checks_catch_an_early_use_of_an_mfma_result():
    g = load_gen()
    lines = g.generate()
    # read the scores of the first score MFMA right after it
    k = next(i for i, x in enumerate(lines) if x.startswith("v_mfma"))
    dst = lines[k].split()[1].rstrip(",")
    first = int(dst[2:-1].split(":")[0])
    lines.insert(k + 1, f"v_mov_b32 v{g.TMP}, v{first}")
    assert any(p.startswith("MFMA->v_mov") for p in g.check_hazards(lines))
