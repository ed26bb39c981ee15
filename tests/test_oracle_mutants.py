"""Planted mistakes in the oracle must each trip at least one pin.

Every mutant is a textual edit of a copy of ``oracle/bmoe_oracle.c``, built
with gcc into a temporary library; the original file is never touched. All
edits keep every memory access in bounds.
"""
import os
import tempfile

import pytest

import oracle
from oracle_pins import ALL_PINS

MUTANTS = {
    "silu_sign": ("g / (1.0 + exp(-g))", "g / (1.0 + exp(g))"),
    "gate_up_swapped": ("hbuf[j] = silu * u;", "hbuf[j] = (u / (1.0 + exp(-u))) * g;"),
    "merge_drops_later_members": ("if (e2g[pick[j]] == r) g += w[j];", "if (j == i) g += w[j];"),
    "ties_to_higher_index": ("z[e] > z[best]) best = e;", "z[e] >= z[best]) best = e;"),
    "unstable_group_order": ("for (int t = 0; t < T; ++t) {\n            for (int i = 0; i < k; ++i) {",
                             "for (int t = T - 1; t >= 0; --t) {\n            for (int i = 0; i < k; ++i) {"),
    "router_bias_dropped": ("if (bias) acc += (double)bias[e];", ""),
    "norm_topk_ignored": ("if (norm_topk) {", "if (0) {"),
    "softmax_unnormalised": ("w[i] = exp(z[best] - m) / s;", "w[i] = exp(z[best] - m);"),
    "shared_experts_dropped": ("if (y_shared) acc +=", "if (0) acc +="),
    "remap_uses_first_pick": ("int r = e2g[pick[i]];", "int r = e2g[pick[0]];"),
    "down_proj_skips_last_hidden": ("for (int j = 0; j < d_ff; ++j) acc +=", "for (int j = 0; j + 1 < d_ff; ++j) acc +="),
    "f32_logits_read_transposed": ("z[e] = (double)zf[(size_t)t * E + e];",
                                   "z[e] = (double)zf[(size_t)e * T + t];"),
    "hidden_output_drops_up": ("h_out[(size_t)r * d_ff + j] = (float)hbuf[j];",
                               "h_out[(size_t)r * d_ff + j] = (float)silu;"),
    "combine_ignores_gate": ("acc += (double)slot_gate[(size_t)t * k + i] * (double)y", "acc += (double)y"),
}


@pytest.fixture(scope="module")
def src_text():
    return open(oracle._SRC).read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, src_text):
    old, new = MUTANTS[name]
    assert src_text.count(old) == 1, f"mutation anchor for {name} not unique in the oracle source"
    with tempfile.TemporaryDirectory() as td:
        src = os.path.join(td, "mutant.c")
        open(src, "w").write(src_text.replace(old, new))
        lib = oracle.build(force=True, src=src, out=os.path.join(td, "libmutant.so"))
        orc = oracle.Oracle(lib)
        failed = []
        for pin in ALL_PINS:
            try:
                pin(orc)
            except AssertionError:
                failed.append(pin.__name__)
        assert failed, f"planted mistake {name!r} passed every pin"
