"""The oracle's pins catch plausible mistakes.

Each mutation below edits one line of a scratch copy of oracle/efq_oracle.c
(built with gcc into a temporary directory, on the CPU; the real build is
untouched).  The pins listed for it are then run against the mutated oracle
and at least one of them must fail.  A mutation that every pin accepts would
mean the oracle could carry that mistake unnoticed.
"""
import os

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))

# name -> (original line fragment, replacement, pins that must catch it)
MUTATIONS = {
    # Eq. (alpha): rescaling of the history dropped
    "alpha_one": ("double alpha = (m == -INFINITY) ? 0.0 : exp((double)m - (double)mnew);",
                  "double alpha = 1.0;", ["twin"]),
    # grouped-query attention: every query head reads V~ of kv head 0
    "kv_head_zero": ("const double *vr = vhat + (((long)b * Hkv + g) * nblk * 32 + j0 + t) * D;",
                     "const double *vr = vhat + (((long)b * Hkv + 0) * nblk * 32 + j0 + t) * D;",
                     ["twin"]),
    # grouped-query head map: modulo instead of division
    "gqa_map": ("const int g = hq / group;", "const int g = hq % Hkv;", ["twin"]),
    # Eq. (d8-index): the "+1" after the floor dropped
    "code_plus_one": ("float bias32 = fmaf(bias, 32.0f, 31.5f);",
                      "float bias32 = fmaf(bias, 32.0f, -0.5f);", ["contract", "threshold"]),
    # Eq. (k-rule): ceiling instead of floor
    "k_ceil": ("float fq = floorf(q);", "float fq = ceilf(q);", ["contract", "k_interval"]),
    # Eq. (z-def): log 6 term with the wrong sign
    "z_sign": ("float c0 = F_LN6 + tau;", "float c0 = -F_LN6 + tau;", ["contract", "threshold"]),
    # running maximum not updated from the tile (Eq. rowmax-update)
    "stale_max": ("            m = mnew;\n        }", "            m = m;\n        }", ["twin"]),
    # exp-then-quantize: scale exponent off by one
    "expq_scale": ("k = clampi(scale6 ? ceil_log2_over6((double)amax) : floor_log2((double)amax) - 2,",
                   "k = clampi(scale6 ? ceil_log2_over6((double)amax) : floor_log2((double)amax) - 1,",
                   ["twin_expq", "expq_def"]),
}


def _pins():
    import test_oracle_pins as P
    twin_case = (1, 300, 300, 8, 2, 128, True, "qwen")
    return {
        "twin": lambda: P.test_recurrence_matches_numpy_twin(oracle, twin_case, "efq"),
        "twin_expq": lambda: P.test_recurrence_matches_numpy_twin(oracle, twin_case, "expq"),
        "contract": lambda: P.test_contract_vs_real_valued(oracle, "mean"),
        "threshold": lambda: P.test_code_matches_threshold_form(oracle, "mean"),
        "k_interval": lambda: P.test_k_rule_interval(oracle),
        "expq_def": lambda: P.test_expq_definition(oracle),
    }


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path, monkeypatch):
    old, new, pins = MUTATIONS[name]
    src = open(oracle._SRC).read()
    assert src.count(old) == 1, f"mutation site of {name} not found exactly once"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = oracle.load(oracle.compile_c(str(path), str(tmp_path / "libmutant.so")))
    monkeypatch.setattr(oracle, "_lib", lib)
    caught = []
    for pin in pins:
        try:
            _pins()[pin]()
        except AssertionError:
            caught.append(pin)
    assert caught, f"no pin caught mutation {name}"


def test_unmutated_oracle_passes_the_same_pins():
    """Control: the real oracle passes every pin the mutations are run against."""
    for pin in _pins().values():
        pin()
