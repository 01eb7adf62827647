"""Mutation check of the oracle pins: each plausible mistake is planted in a *copy* of
oracle.c (never in the GPU library), the copy is built, and the pin suite must fail on it.
This shows that a dropped term, a flipped comparison, a swapped child, a wrong index or a
lower-precision sum in the oracle would not go unnoticed."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, text in oracle.c, replacement, which occurrence: 0 = first only, None = all)
MUTANTS = [
    ("tie_rule_flipped", "return x >= theta;", "return x > theta;", None),
    ("strict_rule_flipped", "return x > theta;", "return x >= theta;", None),
    ("branch_right_goes_left", "next = right[n];", "next = left[n];", None),
    ("pred_right_child_is_left", "kids[1] = right[n];", "kids[1] = left[n];", None),
    ("first_tree_dropped", "for (int32_t t = 0; t < n_trees; t++) {\n            int64_t a = tree_offsets[t];",
     "for (int32_t t = 1; t < n_trees; t++) {\n            int64_t a = tree_offsets[t];", 0),
    ("float_accumulator", "double s = 0.0;", "float s = 0.0f;", None),
    ("feature_index_off_by_one", "goes_right(x[f], threshold[n], rule)", "goes_right(x[f > 0 ? f - 1 : f], threshold[n], rule)", None),
    ("leaf_value_index_shifted", "s += (double)value[a + leaf];", "s += (double)value[a + leaf - (leaf > 1)];", None),
    ("padded_walk_mirrored", "i = (i << 1) + 1 + goes_right(", "i = (i << 1) + 2 - goes_right(", None),
    ("padded_dummy_loses_leaf", "pad_fill(2 * slot + 2, node, level + 1,", "pad_fill(2 * slot + 2, 0, level + 1,", None),
    ("visit_count_doubled", "        k++;\n", "        k += 2;\n", None),
    ("threshold_of_wrong_node", "goes_right(x[f], threshold[n], rule)", "goes_right(x[f], threshold[n > 0 ? n - 1 : n], rule)", None),
]

# mistakes in the feature-access trace, caught by tests/test_oracle_usage.py
USAGE_MUTANTS = [
    ("usage_wrong_bit", "seen[f / 32] |= (uint32_t)1 << (f % 32);",
     "seen[f / 32] |= (uint32_t)1 << ((f + 1) % 32);", None),
    ("usage_one_word", "seen[f / 32] |= (uint32_t)1 << (f % 32);",
     "seen[0] |= (uint32_t)1 << (f % 32);", None),
    ("usage_not_reset_per_doc", "memset(seen, 0, (size_t)words * sizeof(uint32_t));", "", None),
    ("usage_right_goes_left", "? right[a + n] : left[a + n];", "? left[a + n] : left[a + n];", None),
    ("usage_rule_ignored", "goes_right(x[f], threshold[a + n], rule)", "goes_right(x[f], threshold[a + n], 0)", None),
    ("usage_last_tree_dropped", "for (int32_t t = 0; t < n_trees; t++) {\n                const int64_t a",
     "for (int32_t t = 0; t + 1 < n_trees; t++) {\n                const int64_t a", None),
    ("usage_count_first_word", "for (int64_t w = 0; w < words; w++) {\n                for (int b = 0;",
     "for (int64_t w = 0; w < words; w++) {\n                if (w) break;\n                for (int b = 0;", None),
]

# mistakes in the vector-valued / bagged sum, caught by tests/test_oracle_multi.py
MULTI_MUTANTS = [
    ("multi_row_stride_dropped", "const float *v = value + (a + leaf) * (int64_t)n_outputs;",
     "const float *v = value + (a + leaf);", None),
    ("multi_component_shifted", "out[c] += (double)v[c];", "out[c] += (double)v[(c + 1) % n_outputs];", None),
    ("multi_bags_not_averaged", "out[c] /= (double)n_bags;", "out[c] /= 1.0;", None),
    ("multi_bags_summed_wrongly", "out[c] /= (double)n_bags;", "out[c] /= (double)(n_bags + 1);", None),
    ("multi_float_accumulator", "out[c] += (double)v[c];", "out[c] = (double)((float)out[c] + v[c]);", None),
]


def _run_pins(lib, pin_file):
    env = dict(os.environ, ORACLE_LIB=lib)
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", pin_file)],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def _build_mutant(tmp_path, name, old, new, occ):
    src = open(oracle.SRC).read()
    assert old in src, f"mutation site for {name} vanished from oracle.c; update the mutant list"
    mutated = src.replace(old, new, 1) if occ == 0 else src.replace(old, new)
    assert mutated != src
    csrc = tmp_path / "oracle_mutant.c"
    csrc.write_text(mutated)
    lib = str(tmp_path / "liboracle_mutant.so")
    oracle.build(out=lib, src=str(csrc), extra=("-Wno-error",))
    return lib


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new, occ):
    r = _run_pins(_build_mutant(tmp_path, name, old, new, occ), "test_oracle_pins.py")
    assert r.returncode != 0, f"pins did not catch mutant {name}:\n{r.stdout[-2000:]}"


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new,occ", USAGE_MUTANTS, ids=[m[0] for m in USAGE_MUTANTS])
def test_usage_pins_catch_mutant(tmp_path, name, old, new, occ):
    r = _run_pins(_build_mutant(tmp_path, name, old, new, occ), "test_oracle_usage.py")
    assert r.returncode != 0, f"usage pins did not catch mutant {name}:\n{r.stdout[-2000:]}"


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new,occ", MULTI_MUTANTS, ids=[m[0] for m in MULTI_MUTANTS])
def test_multi_pins_catch_mutant(tmp_path, name, old, new, occ):
    r = _run_pins(_build_mutant(tmp_path, name, old, new, occ), "test_oracle_multi.py")
    assert r.returncode != 0, f"multi-output pins did not catch mutant {name}:\n{r.stdout[-2000:]}"


@pytest.mark.slow
@pytest.mark.parametrize("pin_file", ["test_oracle_pins.py", "test_oracle_usage.py", "test_oracle_multi.py"])
def test_unmutated_copy_passes(tmp_path, pin_file):
    # control: the same build-and-run route with the source unchanged must pass, so a failure
    # above is the mutation's doing and not the harness's
    lib = str(tmp_path / "liboracle_copy.so")
    oracle.build(out=lib)
    r = _run_pins(lib, pin_file)
    assert r.returncode == 0, r.stdout[-3000:]
