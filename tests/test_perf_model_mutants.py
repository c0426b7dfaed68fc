"""The performance-model pins are sensitive: each plausible mistake planted in
a copy of oracle/perf_model.py (a wrong sum bound, a dropped factor, a swapped
ratio) makes tests/test_perf_model_pins.py fail; the unmodified copy passes."""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "perf_model.py")
PINS = os.path.join(ROOT, "tests", "test_perf_model_pins.py")

MUTANTS = [
    ("eq1_drops_kv_projections", "att = 4.0 * h * h + 4.0 * h * h / s", "att = 4.0 * h * h"),
    ("eq2_inverted_sparsity", "return C_gpu / B_io * N_e / N_k", "return C_gpu / B_io * N_k / N_e"),
    ("eq3_uses_g_plus_one", "return 2.0 * (p + g) / ((2.0 * p + g) * g)",
     "return 2.0 * (p + g) / ((2.0 * p + g) * (g + 1))"),
    ("eq4_max_instead_of_min", "return min(pme(p, g) * M_tokens / dlt, T_gpu)",
     "return max(pme(p, g) * M_tokens / dlt, T_gpu)"),
    ("eq5_weight_over_total", "return M_total_bytes / M_weight_bytes * B_io",
     "return M_weight_bytes / M_total_bytes * B_io"),
    ("eq7_full_generation", "return (p + g) / (p + g / 2.0) * C_kv", "return (p + g) / (p + g) * C_kv"),
    ("eq8_sum_misses_last_step", "for i in range(g + 1))", "for i in range(g))"),
    ("eq8_floor_not_ceiling", "sum(-(-(p + i) // b)", "sum(((p + i) // b)"),
    ("eq10_drops_epilogue", "return K * g / ((K / q + g) * dlt)", "return K * g / ((K / q) * dlt)"),
    ("eq11_decode_share", "return T_gpu_iter * p / (p + g)", "return T_gpu_iter * g / (p + g)"),
    ("eq12_prologue_not_halved", "(K * p - (tp + T_gpu_iter) / 2.0 * g) / tp",
     "(K * p - (tp + T_gpu_iter) * g) / tp"),
    ("eq12_one_ramp", "return 2.0 * g + (K * p", "return 1.0 * g + (K * p"),
    ("eq6_drops_factor_two", "return 2.0 * s * I_attn * B_kv", "return s * I_attn * B_kv"),
    ("eq6_drops_group_size", "return 2.0 * s * I_attn * B_kv", "return 2.0 * I_attn * B_kv"),
    ("t_gpu_times_delta", "T_gpu = n_sat / dlt", "T_gpu = n_sat * dlt"),
    ("b_kv_times_delta", 'B_kv = inp["kv_capacity_bytes"] / dlt', 'B_kv = inp["kv_capacity_bytes"] * dlt'),
    ("delta_eff_uses_min", 'd_eff = max(dlt, inp["kv_capacity_bytes"] / inp["attn_bw"])',
     'd_eff = min(dlt, inp["kv_capacity_bytes"] / inp["attn_bw"])'),
]


def _run(tmp, name, text):
    path = os.path.join(tmp, f"{name}.py")
    with open(path, "w") as f:
        f.write(text)
    env = dict(os.environ, PERF_MODEL_ORACLE=path)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", PINS],
                       cwd=ROOT, env=env, capture_output=True, text=True)
    return r.returncode


def test_pins_fail_on_every_planted_mistake():
    src = open(SRC).read()
    for name, old, new in MUTANTS:
        assert src.count(old) == 1, f"mutant {name}: fragment not unique"
    with tempfile.TemporaryDirectory() as tmp:
        jobs = [("control", src)] + [(n, src.replace(o, w)) for n, o, w in MUTANTS]
        with ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
            rcs = dict(zip([j[0] for j in jobs], ex.map(lambda j: _run(tmp, *j), jobs)))
    assert rcs.pop("control") == 0, "unmodified oracle must pass its pins"
    survivors = [n for n, rc in rcs.items() if rc == 0]
    assert not survivors, f"planted mistakes not caught by any pin: {survivors}"
