"""The pins must reject a broken oracle.

Each case plants one plausible mistake in a copy of ``oracle/mustafar_oracle.c``
(compiled into a temporary library on the CPU) and runs the pins of
``test_oracle_pins`` against that build; at least one pin must fail. The
unmodified source must pass the same battery.
"""
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "mustafar_oracle.c")

# (name, original text, planted text)
MUTATIONS = [
    ("tie-break towards the higher channel",
     "return (a->idx > b->idx) - (a->idx < b->idx);",
     "return (a->idx < b->idx) - (a->idx > b->idx);"),
    ("smallest magnitudes kept",
     "    if (a->mag > b->mag)\n        return -1;\n    if (a->mag < b->mag)\n        return 1;",
     "    if (a->mag > b->mag)\n        return 1;\n    if (a->mag < b->mag)\n        return -1;"),
    ("ranked by signed value instead of magnitude",
     "r[c].mag = fabs(oracle_half_to_double(x[c]));",
     "r[c].mag = oracle_half_to_double(x[c]);"),
    ("padding to a multiple of 4", "#define ORACLE_PAD 8 ", "#define ORACLE_PAD 4 "),
    ("no padding",
     "int padded = (count + ORACLE_PAD - 1) / ORACLE_PAD * ORACLE_PAD;",
     "int padded = count;"),
    ("bitmap bit order reversed", "bm |= (uint64_t)1 << i;", "bm |= (uint64_t)1 << (63 - i);"),
    ("non-zero pad value", "values[pos + w] = 0x0000;", "values[pos + w] = 0x3c00;"),
    ("kept count truncates instead of rounding",
     "floor((double)sparsity * (double)d + 0.5)", "floor((double)sparsity * (double)d)"),
    ("subnormal exponent off by one", "v = ldexp((double)f, -24);", "v = ldexp((double)f, -25);"),
    ("score scale dropped", "s[j] = scale * acc;", "s[j] = acc;"),
    ("keys used as values",
     "const uint16_t* vj = (j < n_s) ? vc + (int64_t)j * d : vl + (int64_t)(j - n_s) * d;",
     "const uint16_t* vj = (j < n_s) ? kc + (int64_t)j * d : kl + (int64_t)(j - n_s) * d;"),
    ("softmax not normalised", "o += (s[j] / l) *", "o += s[j] *"),
    ("dense window left out of the softmax", "int n = n_s + n_d;", "int n = n_s;"),
]


def _battery():
    """Run the pins (fixed parameters) and return the name of the first failure."""
    checks = [
        ("half decoding", pins.test_half_decoding_matches_numpy_for_every_pattern),
        ("keep count", lambda: pins.test_keep_count_values(128, 0.7, 38)),
        ("keep count half up", lambda: pins.test_keep_count_values(128, 0.50390625, 63)),
        ("stable argsort", lambda: pins.test_prune_equals_stable_argsort(64)),
        ("brute force", lambda: pins.test_prune_equals_brute_force_enumeration(6)),
        ("hand example", pins.test_hand_worked_example),
        ("round trip", lambda: pins.test_round_trip_and_layout_invariants(0.5)),
        ("sdpa", lambda: pins.test_attention_equals_torch_sdpa_on_zero_filled_caches(4, 32, 0.7)),
        ("zero query", pins.test_zero_query_gives_the_mean_value_row),
    ]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure of a pin counts
            return name
    return None


def _build(tmp_path, text, tag):
    c = tmp_path / f"oracle_{tag}.c"
    so = tmp_path / f"liboracle_{tag}.so"
    c.write_text(text)
    subprocess.run(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", "-o", str(so), str(c), "-lm"],
                   check=True)
    return str(so)


def test_unmodified_oracle_passes_the_battery(tmp_path):
    so = _build(tmp_path, open(SRC).read(), "clean")
    with oracle.using_library(so):
        assert _battery() is None


@pytest.mark.parametrize("name,orig,planted", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(tmp_path, name, orig, planted):
    text = open(SRC).read()
    assert text.count(orig) == 1, f"mutation anchor not unique: {orig!r}"
    so = _build(tmp_path, text.replace(orig, planted), "mut")
    with oracle.using_library(so):
        assert _battery() is not None, f"no pin caught: {name}"


# Mistakes in the pruner variants, caught by the variant pins.
VARIANT_MUTATIONS = [
    ("2:4 keeps the two smallest", "keep[r[i].idx] = i < 2;", "keep[r[i].idx] = i >= 2;"),
    ("2:4 groups of three", "for (int g = 0; g + 4 <= d; g += 4) {",
     "for (int g = 0; g + 4 <= d; g += 3) {"),
    ("output-aware score ignores the weights", "const float score = mag * w[c];",
     "const float score = mag;"),
    ("output-aware score ignores the magnitude", "const float score = mag * w[c];",
     "const float score = w[c];"),
]


def _variant_battery():
    from tests import test_oracle_variants as v
    checks = [
        ("24 enumeration", v.test_24_equals_enumeration_of_each_group),
        ("24 numpy", v.test_24_numpy_stable_sort_and_invariants),
        ("oa unit", v.test_output_aware_with_unit_weights_is_magnitude_pruning),
        ("oa numpy", lambda: v.test_output_aware_equals_numpy_float32_scores(64)),
    ]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure of a pin counts
            return name
    return None


def test_unmodified_oracle_passes_the_variant_battery(tmp_path):
    so = _build(tmp_path, open(SRC).read(), "vclean")
    with oracle.using_library(so):
        assert _variant_battery() is None


@pytest.mark.parametrize("name,orig,planted", VARIANT_MUTATIONS, ids=[m[0] for m in VARIANT_MUTATIONS])
def test_planted_variant_mistake_is_caught(tmp_path, name, orig, planted):
    text = open(SRC).read()
    assert text.count(orig) == 1, f"mutation anchor not unique: {orig!r}"
    so = _build(tmp_path, text.replace(orig, planted), "vmut")
    with oracle.using_library(so):
        assert _variant_battery() is not None, f"no pin caught: {name}"


CHANNEL_MUTATIONS = [
    ("channel group keeps one more", "for (int i = 0; i < k && i < n; ++i)\n            keep[(int64_t)r[i].idx * d + c] = 1;",
     "for (int i = 0; i <= k && i < n; ++i)\n            keep[(int64_t)r[i].idx * d + c] = 1;"),
    ("channel key ignores the token weights", "const float score = (float)mag * w[j];",
     "const float score = (float)mag;"),
    ("channel key ignores the magnitude", "const float score = (float)mag * w[j];",
     "const float score = w[j];"),
    ("channel key kept in double", "const float score = (float)mag * w[j];\n                r[j].mag = (double)score;",
     "r[j].mag = mag * (double)w[j];"),
    ("channel and token indexes swapped",
     "const double mag = fabs(oracle_half_to_double(x[(int64_t)j * d + c]));",
     "const double mag = fabs(oracle_half_to_double(x[(int64_t)c * n + j]));"),
    ("channel ranked by signed value",
     "const double mag = fabs(oracle_half_to_double(x[(int64_t)j * d + c]));",
     "const double mag = oracle_half_to_double(x[(int64_t)j * d + c]);"),
    ("probabilities without the scale", "p[j] = scale * acc;", "p[j] = acc;"),
    ("probabilities not normalised", "p[j] /= l;", "p[j] /= 1.0;"),
    ("probabilities without the dense tokens", "const int n_all = n_s + n_d;",
     "const int n_all = n_s;"),
]


def _channel_battery():
    from tests import test_oracle_channel as ch
    checks = [
        ("argsort", lambda: ch.test_channel_prune_equals_stable_argsort(10)),
        ("brute force", ch.test_channel_prune_equals_brute_force),
        ("oa numpy", lambda: ch.test_output_aware_channel_prune_equals_numpy_float32(10)),
        ("oa invariances", ch.test_output_aware_invariances),
        ("oa fp32", ch.test_output_aware_key_is_rounded_to_fp32),
        ("probs", lambda: ch.test_attention_probs_equal_numpy_softmax(4)),
        ("probs x values", ch.test_attention_output_equals_probabilities_times_values),
    ]
    for name, fn in checks:
        try:
            fn()
        except Exception:  # noqa: BLE001 - any failure of a pin counts
            return name
    return None


def test_unmodified_oracle_passes_the_channel_battery(tmp_path):
    so = _build(tmp_path, open(SRC).read(), "cclean")
    with oracle.using_library(so):
        assert _channel_battery() is None


@pytest.mark.parametrize("name,orig,planted", CHANNEL_MUTATIONS, ids=[m[0] for m in CHANNEL_MUTATIONS])
def test_planted_channel_mistake_is_caught(tmp_path, name, orig, planted):
    text = open(SRC).read()
    assert text.count(orig) == 1, f"mutation anchor not unique: {orig!r}"
    so = _build(tmp_path, text.replace(orig, planted), "cmut")
    with oracle.using_library(so):
        assert _channel_battery() is not None, f"no pin caught: {name}"
