"""The oracle against its pins, and the pins against planted mistakes.

Each mutant is a copy of oracle/fc_oracle.c with one plausible mistake (a
dropped term, a wrong sign, a wrong index, the other summation order, ...),
compiled on the CPU; at least one pin must reject it."""
import os
import subprocess

import pytest

import oracle
from oracle import build as obuild

from oracle_pins import PINS


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


MUTANTS = {
    "pair_wrong_index": [("L[m] = L[2 * m] + L[2 * m + 1];", "L[m] = L[2 * m] + L[2 * m];")],
    "odd_node_dropped": [("L[pairs] = L[n - 1];", "L[pairs] = 0.0f;")],
    "odd_node_first": [("L[pairs] = L[n - 1];\n            n = pairs + 1;",
                        "for (int q = pairs; q > 0; --q) L[q] = L[q - 1];\n"
                        "            L[0] = L[n - 1];\n            n = pairs + 1;")],
    "tree_is_linear": [("(order == ORC_TREE) ? tree_sum(L, K) : linear_sum(L, K)", "linear_sum(L, K)")],
    "linear_is_tree": [("(order == ORC_TREE) ? tree_sum(L, K) : linear_sum(L, K)", "tree_sum(L, K)")],
    "linear_double_first": [("for (int k = 1; k < n; ++k)\n        s = s + L[k];",
                             "for (int k = 0; k < n; ++k)\n        s = s + L[k];")],
    "last_worker_dropped": [("for (int k = 0; k < K; ++k)\n                L[k] = leaf(",
                             "for (int k = 0; k < K; ++k)\n                L[k] = (k == K - 1 && K > 1) ? 0.0f : leaf(")],
    "f16_bias_off_by_one": [("e - 25);", "e - 24);")],
    "f16_subnormal_scale": [("ldexpf((float)m, -24)", "ldexpf((float)m, -25)")],
    "f16_sign_lost": [("return s ? -mag : mag;", "return mag;")],
    "no_average": [("const float ga = g[i] * c;", "const float ga = g[i];")],
    "average_over_twice_batch": [("const float c = 1.0f / (float)batch;",
                                  "const float c = 1.0f / (float)(2 * batch);")],
    "decay_dropped": [("const float d = ga + decay;", "const float d = ga;")],
    "decay_sign": [("const float d = ga + decay;", "const float d = ga - decay;")],
    "momentum_on_w": [("const float mom = mu * v[i];", "const float mom = mu * w[i];")],
    "momentum_dropped": [("const float vn = mom + step;", "const float vn = step;")],
    "update_sign": [("const float wn = w[i] - vn;", "const float wn = w[i] + vn;")],
    "lr_after_momentum": [("const float step = lr_j * d;", "const float step = d;"),
                          ("const float wn = w[i] - vn;", "const float wn = w[i] - lr_j * vn;")],
    "mults_swapped": [("lr * segs[j].lr_mult", "lr * segs[j].decay_mult"),
                      ("wd * segs[j].decay_mult", "wd * segs[j].lr_mult")],
    "segment_end_inclusive": [("for (uint64_t i = segs[j].offset; i < segs[j].offset + segs[j].length; ++i) {\n"
                               "            for (int k",
                               "for (uint64_t i = segs[j].offset; i <= segs[j].offset + segs[j].length; ++i) {\n"
                               "            for (int k")],
    "broadcast_skips_worker0": [("for (int k = 0; k < K; ++k)\n        for (int j",
                                 "for (int k = 1; k < K; ++k)\n        for (int j")],
    "step_broadcasts_old_w": [("rc = orc_sgd_step(segs, nseg, w, v, scratch, lr, mu, wd, batch);\n    if (rc) return rc;",
                               "if (bcast_dst) orc_broadcast(segs, nseg, K, w, bcast_dst);\n"
                               "    rc = orc_sgd_step(segs, nseg, w, v, scratch, lr, mu, wd, batch);\n"
                               "    if (rc) return rc;\n    bcast_dst = 0;")],
    "lr_poly_power_dropped": [("factor = pow(remaining, power);", "factor = remaining;")],
    "lr_step_off_by_one": [("int64_t drops = iter / stepsize;", "int64_t drops = (iter + 1) / stepsize;")],
    "lr_scale_inverted": [("(double)batch / (double)base_batch", "(double)base_batch / (double)batch")],
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    src = open(obuild.SRC).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) == 1, f"mutation anchor missing or ambiguous: {old!r}"
        src = src.replace(old, new, 1)
    path = tmp_path / "mutant.c"
    path.write_text(src)
    lib = obuild.build(src=str(path), lib=str(tmp_path / "libmutant.so"))
    failed = []
    with oracle.use(lib):
        for pin in PINS:
            try:
                pin()
            except AssertionError:
                failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
