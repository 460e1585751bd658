"""The generated K loop of the four-wave GEMM tile (gemm_loop_4w.inc).

The loop is inline assembly with hand-placed waits, so the compiler checks
nothing in it. These tests run the generator's own replay checker on the
committed file and confirm that the checker rejects planted schedule
mistakes (each one a way the loop could read stale or unfinished data).
"""
import importlib.util
import os

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
GEN = os.path.join(HERE, "..", "paper_2601_01513_amd", "csrc", "gen_gemm_loop.py")


def _gen():
    spec = importlib.util.spec_from_file_location("gen_gemm_loop", GEN)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_committed_loop_matches_generator_and_checks():
    g = _gen()
    lines = g.generate()
    assert g.check(lines, nmax=14)
    with open(g.OUT) as f:
        body = f.read()
    assert body.endswith(g.render(lines)), "gemm_loop_4w.inc is stale: rerun the generator"
    assert sum("v_mfma" in l for l in lines) == 18 * 64  # 6 full, 6 second-to-last, 6 last panels


def _mutations(lines):
    bars = [k for k, l in enumerate(lines) if l == "s_barrier"]
    reads = [k for k, l in enumerate(lines) if l.startswith("ds_read")]
    i, j = bars[1], reads[20]
    assert lines[i - 2] == "s_waitcnt lgkmcnt(0)"
    late = lambda k: k > bars[0]
    return {
        "drain before the barrier dropped": lines[:i - 2] + lines[i - 1:],
        "fragment read dropped": lines[:j] + lines[j + 1:],
        "barrier dropped": [l for k, l in enumerate(lines) if not (l == "s_barrier" and late(k))],
        "load wait dropped": [l for k, l in enumerate(lines)
                              if not (l == "s_waitcnt vmcnt(0)" and late(k))],
        "lgkmcnt one too loose": [l.replace("lgkmcnt(6)", "lgkmcnt(7)") for l in lines],
        "M0 of a load slot swapped": [l.replace("%[mw], 4096", "%[mw], 8192") if late(k) else l
                                      for k, l in enumerate(lines)],
        "one load slot not advanced": [l for l in lines if not l.startswith("v_add_u32 %[dB5]")],
        "hand-off waits for one load too few": [l.replace("vmcnt(8)", "vmcnt(9)") for l in lines],
        "k-steps swapped": [l.replace("%[rdA1]", "%[rdAx]").replace("%[rdA2]", "%[rdA1]")
                            .replace("%[rdAx]", "%[rdA2]") for l in lines],
    }


@pytest.mark.parametrize("name", sorted(_mutations(_gen().generate())))
def test_checker_rejects_planted_mistake(name):
    g = _gen()
    bad = _mutations(g.generate())[name]
    with pytest.raises((AssertionError, KeyError)):
        g.check(bad)
