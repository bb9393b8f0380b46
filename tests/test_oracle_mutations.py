"""The pins are strong enough: each plausible mistake planted in a copy of the
oracle makes the pin suite fail.

Every mutant is built from oracle/oracle.c with one textual change (applied
at every place the mutated text occurs), loaded by
a separate pytest process (APS_ORACLE_LIB) that runs tests/test_oracle_pins.py
and must fail.  CPU only; the real oracle is untouched."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTANTS = {
    "no_subnormals": ("const int Eq = E > emin ? E : emin;", "const int Eq = E;"),
    "ties_away": ("const double k = nearbyint(", "const double k = round("),
    "no_overflow": ("if (v > oracle_maxfinite(f)) v = INFINITY;", ""),
    "emax_off_by_one": ("int oracle_emax(oracle_format f) { return (1 << f.e) - 2 - f.bias; }",
                        "int oracle_emax(oracle_format f) { return (1 << f.e) - 1 - f.bias; }"),
    "sign_dropped": ("return copysign(v, y);", "return v;"),
    "unrounded_accumulator": ("s = (w == 0) ? q : oracle_round(s + q, f);", "s = (w == 0) ? q : s + q;"),
    "scale_off_by_one": ("return oracle_emax(f) - oracle_ceil_log2((double)t);",
                         "return oracle_emax(f) - oracle_ceil_log2((double)t) + 1;"),
    "floor_not_ceil_on_powers_of_two": ("return (r == 0.5) ? E - 1 : E;", "return E;"),
    "reversed_worker_order": ("const float x = G[(int64_t)w * ld + j];",
                              "const float x = G[(int64_t)(W - 1 - w) * ld + j];"),
    "unscale_wrong_direction": ("out[j] = (flags & ORACLE_OUTPUT_SCALED) ? g : (float)ldexp((double)g, -ft);",
                                "out[j] = (flags & ORACLE_OUTPUT_SCALED) ? g : (float)ldexp((double)g, ft);"),
    "nan_ignored_in_maxabs": ("if (isnan(x))\n                    saw_nan = 1;", "if (0)\n                    saw_nan = 1;"),
    "scale_before_rounding_skipped": (
        "(not when the input is already scaled) */\n"
        "                const float y = (flags & ORACLE_INPUT_QUANTIZED) ? x : scale_fp32(x, ft);",
        "(not when the input is already scaled) */\n"
        "                const float y = x;"),
    "format_ok_admits_emax_128": ("if (oracle_emax(f) > 127) return 0;", "if (oracle_emax(f) > 128) return 0;"),
    "format_ok_admits_minsub_below_fp32": ("if (oracle_emin(f) - f.m < -149) return 0;",
                                           "if (oracle_emin(f) - f.m < -150) return 0;"),
    "literal_exponent_counts_zeros": ("return v == 0.0f ? INT32_MIN : oracle_ceil_log2(fabs((double)v));",
                                      "return v == 0.0f ? -200 : oracle_ceil_log2(fabs((double)v));"),
    "kahan_compensation_sign": ("const double y = oracle_round(x - *c, f);",
                                "const double y = oracle_round(x + *c, f);"),
    "ring_starts_one_master_late": ("const int32_t g = (int32_t)((seg + gi) % ng);",
                                    "const int32_t g = (int32_t)((seg + gi + 1) % ng);"),
    "mantissa_bits_off_by_one": ("const double k = nearbyint(ldexp(a, f.m - Eq));",
                                 "const double k = nearbyint(ldexp(a, f.m + 1 - Eq));"),
    "gemm_product_not_cast": ("const double p = oracle_round(a * b, acc);", "const double p = a * b;"),
    "gemm_inputs_not_cast": ("const double a = oracle_round((double)A[(int64_t)i * lda + k], in);",
                             "const double a = (double)A[(int64_t)i * lda + k];"),
    "gemm_accumulates_in_input_format": ("chain_add(&s, &c, p, acc, accumulator);",
                                         "chain_add(&s, &c, p, in, accumulator);"),
    "decode_subnormal_exponent": ("a = ldexp((double)mant, oracle_emin(f) - f.m);",
                                  "a = ldexp((double)mant, oracle_emin(f) - f.m - 1);"),
    "encode_bias_off_by_one": ("ef = (uint32_t)(E + f.bias);", "ef = (uint32_t)(E + f.bias + 1);"),
    "encode_nan_low_mantissa_bit": ("mant = f.m > 0 ? (1u << (f.m - 1)) : 0u;", "mant = f.m > 0 ? 1u : 0u;"),
    "nibble_order_swapped": ("(int)(j & 1) * 4", "(int)(~j & 1) * 4"),
    "uint16_codes_big_endian": ("b[2 * j] = (uint8_t)(c & 0xFF);\n        b[2 * j + 1] = (uint8_t)(c >> 8);",
                                "b[2 * j] = (uint8_t)(c >> 8);\n        b[2 * j + 1] = (uint8_t)(c & 0xFF);"),
    "group_members_reversed": ("const float x = G[(int64_t)(g * k + m) * ld + j];",
                               "const float x = G[(int64_t)(g * k + (k - 1 - m)) * ld + j];"),
    "ring_not_rotated": ("const int64_t seg = j * ng / n;", "const int64_t seg = 0;"),
    "round_off_counts_zero_grad_h": ("if (grad_h[j] == 0.0f) continue;", "if (0) continue;"),
    "round_off_signed": ("sum += fabs(((double)grad_h[j] - (double)grad_l[j]) / (double)grad_h[j]);",
                         "sum += ((double)grad_h[j] - (double)grad_l[j]) / (double)grad_h[j];"),
    "dequantize_scale_not_undone": ("out[j] = (float)ldexp(v, -ft);", "out[j] = (float)v;"),
    "codes_reduce_unrounded": ("s = (w == 0) ? q : oracle_round(s + q, f); /* low-precision accumulator */",
                               "s = (w == 0) ? q : s + q; /* low-precision accumulator */"),
    "nibble_row_stride": ("return bits <= 4 ? ld / 2 : (bits <= 8 ? ld : 2 * ld);",
                          "return bits <= 4 ? ld : (bits <= 8 ? ld : 2 * ld);"),
}


def _run_mutant(src: str, tmp, name: str):
    """Build the oracle with one mutation and run the pins against it in a
    process of its own; returns (name, pytest's exit status or None when the
    mutation site is missing, the tail of its output)."""
    old, new = MUTANTS[name]
    if src.count(old) < 1:
        return name, None, "mutation site not found"
    d = tmp / name
    d.mkdir()
    mutated = d / "oracle_mut.c"
    mutated.write_text(src.replace(old, new))
    lib = O.build(force=True, src=str(mutated), out=str(d / "liboracle_mut.so"))
    env = dict(os.environ, APS_ORACLE_LIB=lib, OMP_NUM_THREADS="1")
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    return name, res.returncode, res.stdout[-2000:]


def test_pins_catch_every_mutant(tmp_path):
    """Every mutant, each in a pin run of its own, several at a time."""
    src = open(SRC).read()
    workers = max(1, min(8, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(lambda nm: _run_mutant(src, tmp_path, nm), sorted(MUTANTS)))
    missing = [nm for nm, rc, _ in results if rc is None]
    survivors = [(nm, out) for nm, rc, out in results if rc == 0]
    assert not missing, f"mutation sites not found: {missing}"
    assert not survivors, "mutants that survived the pins:\n" + "\n".join(f"{nm}:\n{out}" for nm, out in survivors)
