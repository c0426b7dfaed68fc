"""The oracle pins are sensitive: each plausible mistake planted in a copy of
oracle.c (a dropped term, a wrong index or sign, a swapped operand, a wrong
causal limit) makes the pin suite fail.  The mistakes are planted on the CPU
only, in a temporary build; the real oracle is untouched (the control run
must pass)."""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")

# (name, exact source fragment, replacement)
MUTANTS = [
    ("gqa_head_map", "const int32_t g = h / s;\n  const int32_t C = p->context_lens[b];",
     "const int32_t g = h % p->H_kv;\n  const int32_t C = p->context_lens[b];"),
    ("slot_index", "int32_t slot = t % p->P;", "int32_t slot = (t + 1) % p->P;"),
    ("page_index", "p->max_pages_per_seq + t / p->P];\n  int32_t slot",
     "p->max_pages_per_seq + (t + 1) / p->P];\n  int32_t slot"),
    ("kv_layout_transposed", "return (((int64_t)page * p->H_kv + g) * p->P + slot) * p->D;",
     "return (((int64_t)page * p->P + slot) * p->H_kv + g) * p->D;"),
    ("causal_limit_drops_diagonal", "const int32_t n_vis = C - L + r + 1; /* keys",
     "const int32_t n_vis = C - L + r; /* keys"),
    ("causal_top_left_aligned", "const int32_t n_vis = C - L + r + 1; /* keys",
     "const int32_t n_vis = (r + 1 < C ? r + 1 : C); /* keys"),
    ("scale_dropped", "x[t] = acc * p->scale;", "x[t] = acc;"),
    ("max_sign", "x[t] = expf(x[t] - m);\n    l += x[t];", "x[t] = expf(m - x[t]);\n    l += x[t];"),
    ("sum_drops_last_term", "x[t] = expf(x[t] - m);\n    l += x[t];",
     "x[t] = expf(x[t] - m);\n    if (t + 1 < n_vis) l += x[t];"),
    ("k_used_for_v", "out_row[d] += x[t] * load_elem(p->v,", "out_row[d] += x[t] * load_elem(p->k,"),
    ("q_row_uses_kv_head", "const int64_t q0 = (qrow * p->H_q + h) * p->D;\n  int32_t t, d;",
     "const int64_t q0 = (qrow * p->H_q + g) * p->D;\n  int32_t t, d;"),
    ("bf16_widen_shift", "uint32_t u = (uint32_t)b << 16;", "uint32_t u = (uint32_t)b << 15;"),
    ("gather_slot", "rows_out[n++] = (int64_t)page * P + t % P;",
     "rows_out[n++] = (int64_t)page * P + t / P;"),
    ("weights_not_normalised", "for (int32_t t = 0; t < n_vis; ++t) w_out[t] = w_out[t] / l;",
     "for (int32_t t = 0; t < n_vis; ++t) w_out[t] = w_out[t];"),
    ("append_position_one_late", "const int32_t pos = C - L + j;\n      const int32_t page",
     "const int32_t pos = C - L + j + 1;\n      const int32_t page"),
    ("append_head_layout", "const size_t dst = (((size_t)page * H_kv + g) * P + slot) * row_bytes;",
     "const size_t dst = (((size_t)page * P + slot) * H_kv + g) * row_bytes;"),
    ("append_rows_reversed", "const size_t src = ((size_t)(row0 + j) * H_kv + g) * row_bytes;",
     "const size_t src = ((size_t)(row0 + L - 1 - j) * H_kv + g) * row_bytes;"),
    ("append_v_from_k", "(const char *)v_new + src", "(const char *)k_new + src"),
    ("append_decode_skips_nothing", "L = C > 0 ? 1 : 0;\n    }", "L = 1;\n    }"),
    ("sched_preempts_oldest", "slot_order[s] > slot_order[newest])) newest = s;",
     "slot_order[s] < slot_order[newest])) newest = s;"),
    ("sched_need_off_by_one", "if (slot_seq[s] >= 0 && context_lens[s] % 16 == 0) ++need;",
     "if (slot_seq[s] >= 0 && context_lens[s] % 16 == 1) ++need;"),
    ("sched_admits_while_preempting", "if (!info[0]) {\n    const int32_t token_budget",
     "if (1) {\n    const int32_t token_budget"),
    ("sched_finished_pages_leak", "/ 16; ++p)\n      free_pages[free_n++] = block_table",
     "/ 16 - 1; ++p)\n      free_pages[free_n++] = block_table"),
    ("sched_budget_ignores_decode_rows", "const int32_t token_budget = n_real - info[4];",
     "const int32_t token_budget = n_real;"),
    ("sched_budget_checked_before_adding", "tokens + len > token_budget", "tokens > token_budget"),
    ("sched_preempted_queue_reversed", "const int32_t at = (head + k++) % Q;",
     "const int32_t at = (head + n_pre - 1 - k++) % Q;"),
    ("sched_arrivals_fill_reserve", "qlen >= Q - S) continue;", "qlen >= Q) continue;"),
    ("sched_admit_pops_from_bottom", "block_table[(int64_t)slot * MP + j] = free_pages[--free_n];",
     "block_table[(int64_t)slot * MP + j] = free_pages[P - free_n--];"),
    ("sched_decode_token_not_counted", "context_lens[s] += 1;\n    rows[s] = 1;",
     "rows[s] = 1;"),
]


def _build_and_run(tmp, name, src_text):
    c = os.path.join(tmp, f"{name}.c")
    so = os.path.join(tmp, f"{name}.so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    "-o", so, c, "-lm"], check=True, capture_output=True)
    env = dict(os.environ, ORACLE_LIB=so, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        PINS], cwd=ROOT, env=env, capture_output=True, text=True)
    return r.returncode


def test_pins_fail_on_every_planted_mistake():
    src = open(SRC).read()
    for name, old, new in MUTANTS:
        assert src.count(old) == 1, f"mutant {name}: fragment not unique in oracle.c"
    with tempfile.TemporaryDirectory() as tmp:
        jobs = [("control", src)] + [(n, src.replace(o, w)) for n, o, w in MUTANTS]
        with ThreadPoolExecutor(min(8, os.cpu_count() or 1)) as ex:
            rcs = dict(zip([j[0] for j in jobs],
                           ex.map(lambda j: _build_and_run(tmp, *j), jobs)))
    assert rcs.pop("control") == 0, "unmodified oracle must pass its pins"
    survivors = [n for n, rc in rcs.items() if rc == 0]
    assert not survivors, f"planted mistakes not caught by any pin: {survivors}"
