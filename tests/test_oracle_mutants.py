"""Planted mistakes in the oracle must fail its pins.

Each case copies the oracle (C source and Python module) with the CPU pin tests into a
scratch directory, plants one plausible mistake in the copy (a wrong constant, a dropped
term, a flipped sign, a swapped index or nibble, a truncating rounding), builds it, and runs
the pin suites there: at least one pin must fail.  The repository's own oracle is never
touched.  Nothing here runs on a GPU.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, file under oracle/, original text, planted text)
MUTANTS = [
    ("q4k_min_truncated", "qf_oracle.c",
     "                lm[j] = (dmin != 0.0f) ? clampi(rne_int(mu[j] / dmin), 0, 63) : 0;",
     "                lm[j] = (dmin != 0.0f) ? clampi(floor(mu[j] / dmin), 0, 63) : 0;"),
    ("q4k_scale_truncated", "qf_oracle.c",
     "                ls[j] = (d != 0.0f) ? clampi(rne_int(a[j] / d), 0, 63) : 0;",
     "                ls[j] = (d != 0.0f) ? clampi(floor(a[j] / d), 0, 63) : 0;"),
    ("q4k_code_nibbles_swapped", "qf_oracle.c",
     "(uint8_t)((q[64 * c + l] & 15) | ((q[64 * c + 32 + l] & 15) << 4))",
     "(uint8_t)((q[64 * c + 32 + l] & 15) | ((q[64 * c + l] & 15) << 4))"),
    ("q4k_scale_high_bits_shift", "qf_oracle.c",
     "sc[j]     = (uint8_t)((ls[j] & 63) | ((ls[j + 4] >> 4) << 6));",
     "sc[j]     = (uint8_t)((ls[j] & 63) | ((ls[j + 4] >> 3) << 6));"),
    ("q4k_offset_sign", "qf_oracle.c",
     "or_bf16_from_f32(prod - t2);\n                    }",
     "or_bf16_from_f32(prod + t2);\n                    }"),
    ("nvfp4_tensor_scale_constant", "qf_oracle.c",
     "float S = g / 2688.0f;", "float S = g / 2048.0f;"),
    ("nvfp4_block_scale_dropped_factor", "qf_oracle.c",
     "float six_s = 6.0f * S;", "float six_s = S;"),
    ("nvfp4_even_element_high_nibble", "qf_oracle.c",
     "if ((k & 1) == 0) *p = (uint8_t)((*p & 0xF0) | code);",
     "if ((k & 1) != 0) *p = (uint8_t)((*p & 0xF0) | code);"),
    ("e2m1_ties_to_odd", "qf_oracle.c",
     "if (d < bd || (d == bd && (m % 2) == 0)) { best = m; bd = d; }",
     "if (d < bd || (d == bd && (m % 2) == 1)) { best = m; bd = d; }"),
    ("e4m3_saturates_to_nan", "qf_oracle.c",
     "if (t >= 448.0) return 0x7E;", "if (t >= 448.0) return 0x7F;"),
    ("mxfp4_scale_exponent_off_by_one", "qf_oracle.c",
     "p = (e2 - 1) - 2;", "p = (e2 - 1) - 1;"),
    ("bf16_ties_to_odd", "qf_oracle.c",
     "if (rem > 0.5 || (rem == 0.5 && fmod(lo, 2.0) != 0.0)) lo += 1.0;\n    return lo * q;",
     "if (rem > 0.5 || (rem == 0.5 && fmod(lo, 2.0) == 0.0)) lo += 1.0;\n    return lo * q;"),
    ("amax_drops_abs", "qf_oracle.c",
     "float a = fabsf(or_bf16_to_f32(x[r * ldx + k]));", "float a = or_bf16_to_f32(x[r * ldx + k]);"),
    ("dx_uses_transposed_weight", "__init__.py",
     "return bf16_array_to_f64(dy) @ bf16_array_to_f64(what)\n",
     "return bf16_array_to_f64(dy) @ bf16_array_to_f64(what).T\n"),
]

PIN_SUITES = ["tests/test_oracle_codecs.py", "tests/test_oracle_quant.py",
              "tests/test_oracle_gemm.py"]


def _run_mutant(tmp_root, name, fname, old, new):
    d = os.path.join(tmp_root, name)
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"),
                    ignore=shutil.ignore_patterns("_build", "__pycache__"))
    shutil.copytree(os.path.join(ROOT, "tests"), os.path.join(d, "tests"),
                    ignore=shutil.ignore_patterns("__pycache__", "test_gpu_*", "test_abi_*",
                                                  "test_oracle_mutants.py"))
    shutil.copytree(os.path.join(ROOT, "workloads"), os.path.join(d, "workloads"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    path = os.path.join(d, "oracle", fname)
    src = open(path).read()
    assert src.count(old) == 1, f"{name}: the text to mutate must occur exactly once"
    open(path, "w").write(src.replace(old, new))
    b = subprocess.run([sys.executable, "-c", "import oracle.build as b; b.build()"], cwd=d,
                       capture_output=True, text=True, timeout=120)
    if b.returncode != 0:
        return name, "build failed: " + b.stderr[-400:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", *PIN_SUITES], cwd=d, capture_output=True, text=True,
                       timeout=600)
    return name, r.returncode


def test_every_planted_mistake_fails_a_pin(tmp_path):
    # the unmutated copy must pass, or the mutants prove nothing
    name, rc = _run_mutant(str(tmp_path), "unmutated", "qf_oracle.c", "float S = g / 2688.0f;",
                           "float S = g / 2688.0f;")
    assert rc == 0, f"the unmutated oracle copy fails its pins ({rc})"
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda m: _run_mutant(str(tmp_path), *m), MUTANTS))
    survivors = [n for n, rc in results if rc == 0]
    broken = [(n, rc) for n, rc in results if isinstance(rc, str)]
    assert not broken, broken
    assert not survivors, f"planted mistakes that pass every pin: {survivors}"


@pytest.mark.parametrize("m", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutation_text_is_present(m):
    _, fname, old, _ = m
    assert open(os.path.join(ROOT, "oracle", fname)).read().count(old) == 1
