"""Planted mistakes in copies of the oracle must each fail at least one pin.

Every mutant is a plausible slip (a dropped term, a wrong sign, index or
coefficient, an update reading the wrong time level); the pins in
tests/pins.py must catch all of them.  Mutants are compiled into a temporary
directory and run in a child process, so a mutant that crashes counts as
caught without taking the test runner down.  The real oracle is never
modified.
"""

import json
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (id, text in tc_oracle.c, replacement)
MUTANTS = [
    ("offset_off_by_one", "offsets[t + 1] = offsets[t] + sizes[t];",
     "offsets[t + 1] = offsets[t] + sizes[t] + (t == 3);"),
    ("offset_start_one", "offsets[0] = 0;", "offsets[0] = 1;"),
    ("pack_skips_first", "for (int64_t e = 0; e < sizes[t]; ++e)\n            memcpy(dst + (start + e) * elem_bytes",
     "for (int64_t e = (t == 0 && sizes[t] > 1); e < sizes[t]; ++e)\n            memcpy(dst + (start + e) * elem_bytes"),
    ("unpack_wrong_source", "memcpy(dst + e * elem_bytes, src + (start + e) * elem_bytes",
     "memcpy(dst + e * elem_bytes, src + (start + e + (e + 1 < sizes[t])) * elem_bytes"),
    ("bf16_bias", "expo - 127", "expo - 126"),
    ("bf16_subnormal_scale", "ldexp((double)frac / 128.0, -126)", "ldexp((double)frac / 128.0, -127)"),
    ("bf16_hidden_bit", "ldexp(1.0 + (double)frac / 128.0", "ldexp((double)frac / 128.0"),
    ("reduce_avg_divisor", "sum / (double)K", "sum / (double)(K + (K > 2))"),
    ("reduce_skips_worker", "for (int32_t i = 0; i < K; ++i)\n            sum +=",
     "for (int32_t i = (K > 2); i < K; ++i)\n            sum +="),
    ("reduce_ops_swapped", "(op == ORACLE_AVG) ? sum / (double)K : sum", "(op == ORACLE_SUM) ? sum / (double)K : sum"),
    ("spread_sign", "spread += x[i][j] - c;", "spread += c - x[i][j];"),
    ("center_mean_not_sum", "xc[j] = c + alpha * spread;", "xc[j] = c + alpha * spread / K;"),
    ("center_drops_rho", "double alpha = eta * rho;", "double alpha = eta;"),
    ("center_frozen", "xc[j] = c + alpha * spread;", "xc[j] = c;"),
    ("worker_elastic_sign", "x[i][j] = xi - eta * (gi + rho * (xi - c));",
     "x[i][j] = xi - eta * (gi - rho * (xi - c));"),
    ("worker_drops_eta", "x[i][j] = xi - eta * (gi + rho * (xi - c));",
     "x[i][j] = xi - (gi + rho * (xi - c));"),
    ("worker_drops_grad", "x[i][j] = xi - eta * (gi + rho * (xi - c));",
     "x[i][j] = xi - eta * (rho * (xi - c));"),
    ("worker_grad_sign", "x[i][j] = xi - eta * (gi + rho * (xi - c));",
     "x[i][j] = xi + eta * gi - eta * rho * (xi - c);"),
    ("worker_reads_new_center", "x[i][j] = xi - eta * (gi + rho * (xi - c));",
     "x[i][j] = xi - eta * (gi + rho * (xi - (c + alpha * spread)));"),
    ("worker_uses_other_gradient", "double gi = stored_value(g[i], g_dtype, j);",
     "double gi = stored_value(g[K - 1 - i], g_dtype, j);"),
    ("tensor_slot_width", "return ((e / 4) * K + i) * 4 + (e % 4);", "return ((e / 2) * K + i) * 2 + (e % 2);"),
    ("tensor_worker_major", "return ((e / 4) * K + i) * 4 + (e % 4);", "return (i * ((e / 4) + 1) + (e / 4)) * 4 + (e % 4);"),
    ("sgd_sign", "x[i][j] = x[i][j] - eta * stored_value(g[i], g_dtype, j);",
     "x[i][j] = x[i][j] + eta * stored_value(g[i], g_dtype, j);"),
    ("async_center_sign", "xc[j] = xc[j] + alpha * d;", "xc[j] = xc[j] - alpha * d;"),
    ("async_worker_reads_new_center", "x[w][j] = x[w][j] - alpha * d;",
     "x[w][j] = x[w][j] - alpha * (x[w][j] - xc[j]);"),
    ("async_ignores_order", "int32_t w = order[r];", "int32_t w = r % K;"),
    ("sync_sgd_drops_rescale", "x[i][j] = x[i][j] - eta * rescale * S;", "x[i][j] = x[i][j] - eta * S;"),
    ("sync_sgd_own_gradient", "x[i][j] = x[i][j] - eta * rescale * S;",
     "x[i][j] = x[i][j] - eta * rescale * K * stored_value(g[i], g_dtype, j);"),
    ("broadcast_short", "memcpy(dst[i], src, (size_t)(N * elem_bytes));",
     "memcpy(dst[i], src, (size_t)((N - (N > 1)) * elem_bytes));"),
    ("center_reads_new_workers",
     "        for (int32_t i = 0; i < K; ++i)\n            spread += x[i][j] - c;\n",
     ""),
]


def _mutant_source(find, repl):
    src = open(oracle.SOURCE).read()
    assert src.count(find) >= 1, f"mutation anchor not found in the oracle: {find!r}"
    if find.startswith("        for (int32_t i = 0; i < K; ++i)\n            spread"):
        # Gauss-Seidel slip: accumulate the spread from the already-updated
        # workers instead of the time-t ones.
        src = src.replace(find, repl, 1)
        return src.replace("x[i][j] = xi - eta * (gi + rho * (xi - c));",
                           "x[i][j] = xi - eta * (gi + rho * (xi - c));\n"
                           "            spread += x[i][j] - c;", 1)
    return src.replace(find, repl, 1)


@pytest.mark.parametrize("mid,find,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, mid, find, repl):
    src = tmp_path / "mutant.c"
    src.write_text(_mutant_source(find, repl))
    lib = tmp_path / "libmutant.so"
    oracle.build(str(src), str(lib))
    proc = subprocess.run([sys.executable, "-m", "tests.pins", str(lib)], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)
    if proc.returncode != 0:
        return  # the mutant crashed the pins: caught
    failed = json.loads(proc.stdout.strip().splitlines()[-1])
    assert failed, f"mutant {mid} passed every pin"


def test_unmodified_copy_passes(tmp_path):
    """Control: the same harness on an unmodified copy reports no failure."""
    src = tmp_path / "copy.c"
    src.write_text(open(oracle.SOURCE).read())
    lib = tmp_path / "libcopy.so"
    oracle.build(str(src), str(lib))
    proc = subprocess.run([sys.executable, "-m", "tests.pins", str(lib)], cwd=ROOT,
                          capture_output=True, text=True, timeout=300, check=True)
    assert json.loads(proc.stdout.strip().splitlines()[-1]) == []
