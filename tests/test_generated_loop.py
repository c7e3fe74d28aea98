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


def committed_body(d, form="LOOP"):
    text = open(os.path.join(CSRC, f"attn_d{d}_loop.inc")).read()
    head = f'#define DITANGO_D{d}_{form}_ASM \\\n  "'
    start = text.index(head) + len(head)
    end = text.index('\\n"\n', start)
    return text[start:end].split("\\n\\t")


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("fast", [False, True])
def test_committed_loop_matches_generator(d, fast):
    g = load_gen()
    g.configure(d)
    assert committed_body(d, "FAST" if fast else "LOOP") == g.generate(fast=fast)


@pytest.mark.parametrize("d", [128, 64])
def test_fast_form_differs_from_the_checked_one_only_in_the_maximum(d):
    """The fast form has no per-tile test of the running maximum and no slow
    path; its prologue sets m from tile 0's scores; every MFMA, LDS read,
    tile load, wait and barrier is the checked form's, in the same order."""
    g = load_gen()
    g.configure(d)
    checked, fast = g.generate(), g.generate(fast=True)
    assert not any(x.startswith("v_cmp_nle") for x in fast)
    assert not any("Lslow" in x for x in fast)
    assert sum(1 for x in checked if x.startswith("v_cmp_nle")) == 2 * 12   # 4 block + 4 tail + 4 last iterations
    keep = ("v_mfma", "ds_read", "buffer_load", "global_load", "s_waitcnt", "s_barrier")
    pick = lambda lines: [x for x in lines if x.startswith(keep)]
    assert pick(fast) == pick(checked)
    # outside the prologue's maximum and the removed tests, the VALU work is
    # the checked form's minus its slow blocks
    exps = lambda lines: sum(1 for x in lines if x.startswith("v_exp"))
    slow = checked[checked.index(".Lslow0_%=:"):]
    assert exps(fast) == exps(checked) - exps(slow)
    # tile 0's maximum: per query block, 31 maxima over its 32 scores, the
    # lane pair's exchange, the scale, before the first exponential
    first_exp = next(i for i, x in enumerate(fast) if x.startswith("v_exp"))
    pro = fast[:first_exp]
    assert sum(1 for x in pro if x.startswith("v_permlane32_swap")) == 2
    assert sum(1 for x in pro if x.startswith("v_max_f32")) == 2 * (31 + 2)


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("fast", [False, True])
def test_generated_loop_passes_its_checks(d, fast):
    g = load_gen()
    g.configure(d)
    lines = g.generate(fast=fast)
    assert g.check_hazards(lines) == []
    assert g.check_fragments(lines) == []
    mfma = [x for x in lines if x.startswith("v_mfma")]
    # scores of tile 0, the block of four iterations, the four iterations of
    # the tail loop, four last iterations: 2 MFMAs per fragment step; D/8
    # score steps and D/8 P V steps per tile
    steps = d // 8
    assert len(mfma) == 2 * (steps + 2 * 4 * 2 * steps + 4 * steps)
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
