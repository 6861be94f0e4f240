"""Every plausible mistake planted in the oracle must fail at least one pin.

Each mutant is a copy of the oracle source with one edit (a swapped index, a
dropped stride, a transposed operand, a wrong sign, an off-by-one, a ceiling
for a floor), compiled on the CPU into a temporary directory and run through
the same pin checks as the real oracle."""
import json
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, text in oracle.c, replacement, occurrence to replace: 0-based, or None for all)
MUTANTS = [
    ("extent_ceil", "return (in - k) / s + 1;", "return (in - k + s - 1) / s + 1;", None),
    ("input_swap_uv", "in[((i * Hi + (m * s + u)) * Wi + (n * s + v)) * Ci + r]",
     "in[((i * Hi + (m * s + v)) * Wi + (n * s + u)) * Ci + r]", 0),
    ("input_drop_col_stride", "in[((i * Hi + (m * s + u)) * Wi + (n * s + v)) * Ci + r]",
     "in[((i * Hi + (m * s + u)) * Wi + (n + v)) * Ci + r]", 0),
    ("filter_transposed", "filt[((u * Kw + v) * Ci + r) * Co + j]",
     "filt[((v * Kh + u) * Ci + r) * Co + j]", 0),
    ("filter_channel_swap", "filt[((u * Kw + v) * Ci + r) * Co + j]",
     "filt[((u * Kw + v) * Co + j) * Ci + r]", 0),
    ("sign", "acc += x * w;", "acc -= x * w;", 0),
    ("dropped_last_row", "for (int64_t u = 0; u < Kh; ++u) {", "for (int64_t u = 0; u + 1 < Kh; ++u) {", 0),
    ("dropped_channel", "for (int64_t r = 0; r < Ci; ++r) {", "for (int64_t r = 1; r < Ci; ++r) {", 0),
    ("abs_dropped", "aacc += fabs(x) * fabs(w);", "aacc += fabs(x * w) * 0.5;", 0),
    ("points_wrong_row", "in[((i * Hi + (m * s + u)) * Wi + (n * s + v)) * Ci + r]",
     "in[((i * Hi + (m + u)) * Wi + (n * s + v)) * Ci + r]", 1),
    ("im2win_col_major", "int64_t d = ((i * Ho + m) * (Wi * Kh) + (k * Kh + u)) * Ci + r;",
     "int64_t d = ((i * Ho + m) * (Wi * Kh) + (u * Wi + k)) * Ci + r;", 0),
    ("im2win_no_stride", "int64_t x = ((i * Hi + (m * s + u)) * Wi + k) * Ci + r;",
     "int64_t x = ((i * Hi + (m + u)) * Wi + k) * Ci + r;", 0),
    ("windowed_uses_Kw", "double x = w[((n * s + v) * Kh + u) * Ci + r];",
     "double x = w[((n * s + v) * Kw + u) * Ci + r];", 0),
    ("window_elems_no_Kh", "return N * Ho * Wi * Kh * Ci;", "return N * Ho * Wi * Ci;", 0),
    ("im2col_elems_Kh_twice", "return N * Ho * Wo * Kh * Kw * Ci;", "return N * Ho * Wo * Kh * Kh * Ci;", 0),
    ("pad_shift_sign", "int64_t h = m * s + u - ph, w = n * s + v - pw;",
     "int64_t h = m * s + u + ph, w = n * s + v - pw;", 0),
    ("pad_swapped_axes", "int64_t h = m * s + u - ph, w = n * s + v - pw;",
     "int64_t h = m * s + u - pw, w = n * s + v - ph;", 0),
    ("pad_bound_off_by_one", "return h >= 0 && h < Hi && w >= 0 && w < Wi;",
     "return h >= 0 && h < Hi && w >= 0 && w + 1 < Wi;", 0),
    ("pad_extent_one_side", "int64_t Ho = oracle_out_extent(Hi + 2 * ph, Kh, s);",
     "int64_t Ho = oracle_out_extent(Hi + ph, Kh, s);", 0),
    ("im2win_pad_no_shift", "int64_t h = m * s + u - ph, w = k - pw;", "int64_t h = m * s + u, w = k;", 0),
    ("im2win_pad_strip_width", "int64_t d = ((i * Ho + m) * (Wp * Kh) + (k * Kh + u)) * Ci + r;",
     "int64_t d = ((i * Ho + m) * (Wi * Kh) + (k * Kh + u)) * Ci + r;", 0),
    ("dil_row_undilated", "int64_t h = m * s + u * d - ph, w = n * s + v * d - pw;",
     "int64_t h = m * s + u - ph, w = n * s + v * d - pw;", 0),
    ("dil_extent_k_times_d", "return oracle_out_extent(in, (k - 1) * d + 1, s);",
     "return oracle_out_extent(in, k * d, s);", 0),
    ("dil_group_order_swapped", "int64_t k = (P % Wq) * d + P / Wq;", "int64_t k = (P / d) * d + P % d;", 0),
    ("dil_window_col_swapped", "return (c % d) * Wq + c / d;", "return (c / d) * Wq + c % d;", 0),
    ("im2win_dil_row_undilated", "int64_t h = m * s + u * d - ph, w = k - pw;",
     "int64_t h = m * s + u - ph, w = k - pw;", 0),
    ("windowed_dil_uses_Kw", "span[(v * Kh + u) * Ci + r]", "span[(v * Kw + u) * Ci + r]", 0),
]


def _replace(src, old, new, occ):
    assert old in src, old
    if occ is None:
        return src.replace(old, new)
    parts = src.split(old)
    assert len(parts) > occ + 1, (old, occ)
    return old.join(parts[:occ + 1]) + new + old.join(parts[occ + 1:])


# Runs every pin against the mutant in a child process: a planted index
# mistake can read outside the C arrays, and a crash there must not take the
# test runner down (a crash also counts as caught).
_RUNNER = r"""
import importlib.util, json, sys
sys.path.insert(0, sys.argv[2])
from oracle_checks import ALL_CHECKS
spec = importlib.util.spec_from_file_location("oracle_mutant", sys.argv[1] + "/__init__.py")
mod = importlib.util.module_from_spec(spec)
spec.loader.exec_module(mod)
mod.build(force=True)
failed = []
for check in ALL_CHECKS:
    try:
        check(mod)
    except Exception:
        failed.append(check.__name__)
print(json.dumps(failed))
"""


@pytest.mark.parametrize("name,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new, occ):
    d = tmp_path / name
    d.mkdir()
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    mutated = _replace(src, old, new, occ)
    assert mutated != src
    (d / "oracle.c").write_text(mutated)
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), d / "__init__.py")
    env = dict(os.environ, OMP_NUM_THREADS="2")
    p = subprocess.run([sys.executable, "-c", _RUNNER, str(d), os.path.join(ROOT, "tests")],
                       capture_output=True, text=True, timeout=300, env=env)
    if p.returncode != 0:
        return          # the mutant crashed the pins' process: caught
    failed = json.loads(p.stdout.strip().splitlines()[-1])
    assert failed, "no pin catches mutant %s" % name
