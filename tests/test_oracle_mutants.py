"""Planted mistakes in the oracle (CPU only): each mutant is a copy of the
oracle source with one plausible slip (a dropped term, a wrong sign or index,
a transposed operand, a swapped operand), compiled on the side.  The pins in
test_oracle.py must reject every one of them, which shows they constrain
each part of the oracle.
"""
import os

import pytest

import oracle as oracle_pkg
from tests import test_oracle as pins

SRC = os.path.join(os.path.dirname(oracle_pkg.__file__), "moe_oracle.c")

MUTANTS = {
    "gate_up_swapped": [("const uint16_t *gr = w13 + (int64_t)i * H;", "const uint16_t *gr = w13 + (int64_t)(Is + i) * H;"),
                        ("const uint16_t *ur = w13 + (int64_t)(Is + i) * H;", "const uint16_t *ur = w13 + (int64_t)i * H;")],
    "silu_dropped": [("a[i] = g / (1.0 + exp(-g)) * u;", "a[i] = g * u;")],
    "silu_sign": [("exp(-g)", "exp(g)")],
    "up_reads_gate_row": [("u += xv * bf16v(ur[h]);", "u += xv * bf16v(gr[h]);")],
    "w2_transposed": [("s += a[i] * bf16v(dr[i]);", "s += a[i] * bf16v(w2[(int64_t)i * H + h]);")],
    "tie_to_higher_id": [("l[e] > l[best]", "l[e] >= l[best]")],
    "no_renormalise": [("w[t * k + j] = p[ids[t * k + j]] / s;", "w[t * k + j] = p[ids[t * k + j]];")],
    "permute_slot_major": [("        for (int64_t t = 0; t < T; ++t)\n            for (int j = 0; j < k; ++j)\n                if (ids[t * k + j] == e0 + le) {",
                            "        for (int j = 0; j < k; ++j)\n            for (int64_t t = 0; t < T; ++t)\n                if (ids[t * k + j] == e0 + le) {")],
    "combine_drops_last_slot": [("            for (int j = 0; j < k; ++j) {\n                int32_t r = pair_to_row",
                                 "            for (int j = 0; j + 1 < k; ++j) {\n                int32_t r = pair_to_row")],
    "shared_range_off_by_one": [("if (sc > 0 && t >= sb && t < sb + sc)", "if (sc > 0 && t >= sb && t <= sb + sc)")],
    "layer_skips_weight": [("o[h] += w[t * k + j] * y[h];", "o[h] += y[h];")],
    "permute_total_off_by_one": [("offsets[El] = (int32_t)n;", "offsets[El] = (int32_t)n - 1;")],
    # the grouped FFN's row -> expert lookup takes the first row of the next
    # expert as its own last row
    "ffn_lookup_boundary": [("while (!(offsets[le] <= r && r < offsets[le + 1])) ++le;",
                             "while (!(offsets[le] <= r && r <= offsets[le + 1])) ++le;")],
    # the combine reads the row of the token's first slot for every slot
    "combine_reads_slot0_row": [("int32_t r = pair_to_row[t * k + j];", "int32_t r = pair_to_row[t * k];")],
}

# mutants that only the composition of the stages against the dense layer
# can see (the stage functions have no other value pin)
COMPOSITION_ONLY = ("ffn_lookup_boundary", "combine_reads_slot0_row")

PIN_SUITE = [
    lambda o: [pins.test_route_ids_match_lexsort(o, E, k, kind)
               for E, k in [(8, 2), (64, 8)] for kind in ("normal", "ties")],
    lambda o: pins.test_route_closed_forms(o),
    lambda o: pins.test_permute_matches_stable_argsort(o, 37, 8, 2, 8),
    lambda o: pins.test_layer_matches_dense_masked_evaluation(o, pins.tiny(E=8, k=3, P=4, layout="ep", rank=2)),
    lambda o: pins.test_layer_matches_dense_masked_evaluation(o, pins.tiny(E=8, k=2, P=2, layout="tp", rank=1, I=32)),
    lambda o: pins.test_shared_expert_partials(o),
    lambda o: [pins.test_stages_compose_to_dense_layer(o, c) for c in pins.COMPOSE_CFGS],
    lambda o: pins.test_combine_relabelled_rows(o),
    lambda o: pins.test_combine_accumulate_and_shared_are_additive(o),
    lambda o: pins.test_grouped_ffn_experts_are_independent(o),
]


def test_unmutated_source_passes_suite(oracle):
    for pin in PIN_SUITE:
        pin(oracle)


def build_mutant(tmp_path, name):
    src = open(SRC).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) >= 1, f"mutation anchor missing: {old!r}"
        src = src.replace(old, new)
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src)
    lib = str(tmp_path / "libmutant.so")
    oracle_pkg.build(str(msrc), lib)
    return oracle_pkg.Oracle(lib)


def rejects(pin, mut) -> bool:
    try:
        pin(mut)
    except (AssertionError, ValueError, IndexError):
        return True
    return False


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(tmp_path, name):
    mut = build_mutant(tmp_path, name)
    caught = sum(rejects(pin, mut) for pin in PIN_SUITE)
    assert caught > 0, f"no pin rejects mutant {name}"


@pytest.mark.parametrize("name", COMPOSITION_ONLY)
def test_composition_pin_alone_rejects(tmp_path, name):
    """The stage functions' slips are caught by the composition pin itself
    (not only by some other pin of the suite)."""
    mut = build_mutant(tmp_path, name)
    assert rejects(lambda o: [pins.test_stages_compose_to_dense_layer(o, c) for c in pins.COMPOSE_CFGS], mut)
