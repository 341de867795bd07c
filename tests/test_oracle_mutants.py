"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of the oracle source (never in the
oracle itself), builds it on the CPU, and runs the CPU pin tests against the
planted build in a subprocess: they must fail.  Covered mistakes: wrong
rounding, a dropped term, a wrong constant, a swapped nibble order, a wrong
group size, a transposed metadata index, a wrong sign, a wrong head mapping,
a missing causal mask, a dropped decode tail or a wrong tail stride, a
swapped merge.
"""
import os
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
SRC = (ROOT / "oracle" / "lynx_oracle.c").read_text()

MUTANTS = {
    "floor_not_rint": ("float c = rintf(y);", "float c = floorf(y);"),
    "round_half_away": ("float c = rintf(y);", "float c = roundf(y);"),
    "dropped_zero_term": ("float y = (x - zero) * inv;", "float y = x * inv;"),
    "scale_over_256": ("*scale = range / 255.0f;", "*scale = range / 256.0f;"),
    "anchor_offset_8": ("kq = 16.0 * get_nibble(k_plane + off, d) + 7.5;\n        vq = 16.0 * get_nibble(v_plane + off, d) + 7.5;",
                        "kq = 16.0 * get_nibble(k_plane + off, d) + 8.0;\n        vq = 16.0 * get_nibble(v_plane + off, d) + 8.0;"),
    "nibble_order_swapped": ("    int shift = (e % 2) * 4;\n    row[j]", "    int shift = (1 - e % 2) * 4;\n    row[j]"),
    "k_group_64": ("#define K_GROUP 128", "#define K_GROUP 64"),
    "k_meta_transposed": ("size_t m = (((size_t)b * Hkv + h) * n_groups_max + g) * HEAD_DIM + d;",
                          "size_t m = (((size_t)b * n_groups_max + g) * Hkv + h) * HEAD_DIM + d;"),
    "softmax_sign": ("s[t] = exp(s[t] - m);", "s[t] = exp(m - s[t]);"),
    "no_sm_scale": ("s[t] = acc * sm_scale;", "s[t] = acc;"),
    "gqa_strided": ("int hq = kvh * G + g;", "int hq = g * Hkv + kvh;"),
    "no_causal_mask": ("const int n_new = J->mode == 1 ? i + 1 : J->n_tail;",
                       "const int n_new = J->mode == 1 ? J->nq : J->n_tail;"),
    "decode_tail_dropped": ("const int n_new = J->mode == 1 ? i + 1 : J->n_tail;",
                            "const int n_new = J->mode == 1 ? i + 1 : 0;"),
    "decode_tail_stride": ("const int stride = J->mode == 1 ? J->nq : J->n_tail;",
                           "const int stride = J->nq;"),
    "merge_swapped": ("codes[e] = (uint8_t)(a * 16 + r);", "codes[e] = (uint8_t)(r * 16 + a);"),
    "v_meta_wrong_stride": ("size_t vm = ((size_t)b * Hkv + h) * (size_t)max_tokens + t;\n    double kq",
                            "size_t vm = ((size_t)h * 1 + b) * (size_t)max_tokens + t;\n    double kq"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    edits = MUTANTS[name]
    edits = [edits] if isinstance(edits, tuple) else edits
    text = SRC
    for find, repl in edits:
        assert text.count(find) == 1, f"mutation anchor for {name} not unique/present"
        text = text.replace(find, repl)
    src = tmp_path / "mutant.c"
    src.write_text(text)
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-shared", "-fPIC",
                    "-pthread", str(src), "-o", str(lib), "-lm"], check=True)
    env = dict(os.environ, LYNX_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_codec.py", "tests/test_oracle_attention.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"


# Mistakes planted in the hierarchical codec (Alg. 1), caught by its own pins.
HIER_MUTANTS = {
    "sign_of_normalized_value": ("const int S = xc > 0.0f ? 1 : (xc < 0.0f ? -1 : 0);",
                                 "const int S = 1;"),
    "mean_not_restored": ("const float X = xc + mu_a[cm];", "const float X = xc;"),
    "chunk_64": ("#define H_CHUNK 32", "#define H_CHUNK 64"),
    "no_rounding_bias": ("V = (I + 7) >> 4;", "V = I >> 4;"),
    "centred_correction_not_centred": ("r = I - 16 * V - 8;", "r = I - 16 * V;"),
    "centred_anchor_at_bucket_floor": ("alevel[v] = (float)(expm1(((16 * v + 7.5) / 127.0)",
                                       "alevel[v] = (float)(expm1(((16 * v + 0.0) / 127.0)"),
    "int4_with_seven_bit_transform": ("return variant == H_INT4 ? 7 : 127;", "return 127;"),
    "centred_merged_offset_dropped": ("Ip = 16 * V + 8 + sext4(row[d] & 0xF);",
                                      "Ip = 16 * V + sext4(row[d] & 0xF);"),
}


@pytest.mark.parametrize("name", sorted(HIER_MUTANTS))
def test_hier_pins_catch_mutant(name, tmp_path):
    find, repl = HIER_MUTANTS[name]
    assert SRC.count(find) == 1, f"mutation anchor for {name} not unique/present"
    src = tmp_path / "mutant.c"
    src.write_text(SRC.replace(find, repl))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-shared", "-fPIC",
                    "-pthread", str(src), "-o", str(lib), "-lm"], check=True)
    env = dict(os.environ, LYNX_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_hier.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"


# Planted mistakes in the acceptance of sampled drafts, each of which the pins
# in test_oracle_spec_sample.py must catch.
SAMPLE_MUTANTS = {
    "residual_without_draft": ("return q ? p[v] - q[v] : p[v];", "return p[v];"),
    "keep_test_inverted": ("if (!(prod <= pb[(size_t)n * V + x])) break;",
                           "if (!(prod >= pb[(size_t)n * V + x])) break;"),
    "draw_reuses_rejected_uniform": ("qb + (size_t)n * V, ub[k]);", "qb + (size_t)n * V, ub[n]);"),
    "draw_by_first_prefix_reaching_t": ("if (acc > t) return v;", "if (acc >= t) return v;"),
}


@pytest.mark.parametrize("name", sorted(SAMPLE_MUTANTS))
def test_sample_pins_catch_mutant(name, tmp_path):
    find, repl = SAMPLE_MUTANTS[name]
    assert SRC.count(find) == 1, f"mutation anchor for {name} not unique/present"
    src = tmp_path / "mutant.c"
    src.write_text(SRC.replace(find, repl))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-shared", "-fPIC",
                    "-pthread", str(src), "-o", str(lib), "-lm"], check=True)
    env = dict(os.environ, LYNX_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_spec_sample.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"


# Planted mistakes in the split widths, each of which the pins in
# test_oracle_split.py must catch.
SPLIT_MUTANTS = {
    "field_bits_reversed": ("v |= ((row[bit / 8] >> (bit % 8)) & 1) << i;",
                            "v |= ((row[bit / 8] >> (bit % 8)) & 1) << (w - 1 - i);"),
    "merge_shifts_by_anchor_width": ("codes[r * HEAD_DIM + e] = (uint8_t)((get_field(anc + r * 16 * A, e, A) << R) |",
                                     "codes[r * HEAD_DIM + e] = (uint8_t)((get_field(anc + r * 16 * A, e, A) << A) |"),
    "anchor_value_at_bucket_floor": ("const float half = (float)((1 << R) - 1) / 2.0f;", "const float half = 0.0f;"),
}


@pytest.mark.parametrize("name", sorted(SPLIT_MUTANTS))
def test_split_pins_catch_mutant(name, tmp_path):
    find, repl = SPLIT_MUTANTS[name]
    assert SRC.count(find) == 1, f"mutation anchor for {name} not unique/present"
    src = tmp_path / "mutant.c"
    src.write_text(SRC.replace(find, repl))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-shared", "-fPIC",
                    "-pthread", str(src), "-o", str(lib), "-lm"], check=True)
    env = dict(os.environ, LYNX_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_split.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"


# Planted mistakes in the anchor decode over split-width anchors, each of which
# the pins in test_oracle_split_decode.py must catch.
SPLIT_DECODE_MUTANTS = {
    "decode_anchor_centre_2R_half": ("const double w = (double)(1 << R), half = ((double)(1 << R) - 1.0) / 2.0;",
                                     "const double w = (double)(1 << R), half = (double)(1 << R) / 2.0;"),
    "decode_anchor_weight_2A": ("const double w = (double)(1 << R), half",
                                "const double w = (double)(1 << A), half"),
    "decode_rows_of_nibble_width": ("const int row_bytes = mode == 0 ? NIBBLE_ROW : mode == 1 ? CODE_ROW : 16 * A;",
                                    "const int row_bytes = mode == 0 ? NIBBLE_ROW : mode == 1 ? CODE_ROW : NIBBLE_ROW;"),
    "decode_fields_of_residual_width": ("kq = w * get_field(k_plane + off, d, A) + half;\n        vq = w * get_field(v_plane + off, d, A) + half;",
                                        "kq = w * get_field(k_plane + off, d, R) + half;\n        vq = w * get_field(v_plane + off, d, R) + half;"),
}


@pytest.mark.parametrize("name", sorted(SPLIT_DECODE_MUTANTS))
def test_split_decode_pins_catch_mutant(name, tmp_path):
    find, repl = SPLIT_DECODE_MUTANTS[name]
    assert SRC.count(find) == 1, f"mutation anchor for {name} not unique/present"
    src = tmp_path / "mutant.c"
    src.write_text(SRC.replace(find, repl))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-shared", "-fPIC",
                    "-pthread", str(src), "-o", str(lib), "-lm"], check=True)
    env = dict(os.environ, LYNX_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_split_decode.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"

