"""Mutation test of the oracle's pins.

Each mutant is a copy of oracle.c with one plausible mistake planted (a
dropped term, a wrong sign, index or operand, a wrong log base, a missed
skip).  Every mutant must fail at least one pin in tests/oracle_pins.py;
a mutant that survives means the pins leave part of the oracle unchecked.
Mutants run in child processes so that a crashing one is also counted as
caught.  CPU only; nothing here touches the GPU library.
"""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle.build as obuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, text in oracle.c, replacement)
MUTANTS = [
    ("drop_rope_term",
     "dot += oracle_bf16_to_f64(qp[d]) * kpe_at(&kv, b, t, d);", "(void)qp;"),
    ("no_scale", "score[n] = scale * dot;", "score[n] = dot;"),
    ("log2_lse", "double L = M + log(l);", "double L = M + log2(l);"),
    ("unnormalised_weights", "double w = exp(score[k] - L);", "double w = exp(score[k] - M);"),
    ("skip_block_table",
     "int64_t b = table[(int64_t)r * NB + (sel_tokens ? s / ORACLE_BLOCK : s)];",
     "int64_t b = (sel_tokens ? s / ORACLE_BLOCK : s);"),
    ("token_offset_dropped", "int t0 = sel_tokens ? s % ORACLE_BLOCK : 0;", "int t0 = 0;"),
    ("token_block_is_id",
     "int64_t b = table[(int64_t)r * NB + (sel_tokens ? s / ORACLE_BLOCK : s)];",
     "int64_t b = table[(int64_t)r * NB + (sel_tokens ? s % NB : s)];"),
    ("token_whole_block", "const int per_slot = sel_tokens ? 1 : ORACLE_BLOCK;",
     "const int per_slot = sel_tokens ? 2 : ORACLE_BLOCK;"),
    ("per_row_reads_row0",
     "const int32_t* row_sel = sel + (int64_t)r * sel_s0 + (int64_t)i * sel_s1;",
     "const int32_t* row_sel = sel + (int64_t)r * sel_s0;"),
    ("ckv_transposed", "int64_t i = (b * ORACLE_BLOCK + t) * ORACLE_DLAT + d;",
     "int64_t i = (b * ORACLE_DLAT + d) * ORACLE_BLOCK + t;"),
    ("value_wrong_token", "o[d] += w * ckv_at(&kv, blk[k], tok[k], d);",
     "o[d] += w * ckv_at(&kv, blk[k], 0, d);"),
    ("e4m3_bias", "mag = ldexp(1.0 + (double)m / 8.0, e - 7);",
     "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    ("e4m3_subnormal", "mag = ldexp((double)m, -9);", "mag = ldexp(1.0 + (double)m / 8.0, -7);"),
    ("fp8_scale_dropped",
     "return oracle_e4m3fn_to_f64(((const uint8_t*)kv->ckv)[i]) * (double)kv->ckv_scale[b];",
     "return oracle_e4m3fn_to_f64(((const uint8_t*)kv->ckv)[i]);"),
    ("fp8_kpe_uses_ckv_scale", "* (double)kv->kpe_scale[b];", "* (double)kv->ckv_scale[b];"),
    ("merge_weight_uses_max", "double w = exp(v - L);", "double w = exp(v - Lam);"),
    ("merge_log2", "double L = Lam + log(l);", "double L = Lam + log2(l);"),
    ("merge_no_skip_in_sum",
     "      if (v == -INFINITY) continue;\n      double w = exp(v - L);",
     "      double w = exp(v - L);"),
    ("bf16_shift", "uint32_t u = ((uint32_t)bits) << 16;", "uint32_t u = ((uint32_t)bits) << 15;"),
    ("query_row_of_job", "const uint16_t* ql = q_lat + row * ORACLE_DLAT;",
     "const uint16_t* ql = q_lat + (int64_t)r * ORACLE_DLAT;"),
    ("job_index_ignores_mq", "int r = (int)(row / ((int64_t)Mq * H));", "int r = (int)(row / H);"),
    ("empty_lse_zero", "      lse[row] = -INFINITY;\n      if (max_out)",
     "      lse[row] = 0.0;\n      if (max_out)"),
    ("rope_query_uses_latent",
     "dot += oracle_bf16_to_f64(qp[d]) * kpe_at(&kv, b, t, d);",
     "dot += oracle_bf16_to_f64(ql[d]) * kpe_at(&kv, b, t, d);"),
    ("max_is_min", "if (score[k] > M) M = score[k];", "if (score[k] < M) M = score[k];"),
    ("wire_max_is_lse", "if (max_out) max_out[row] = M;", "if (max_out) max_out[row] = L;"),
    ("wire_denom_unshifted", "if (denom_out) denom_out[row] = l;",
     "if (denom_out) denom_out[row] = l * exp(M);"),
]

_RUNNER = r"""
import sys
sys.path.insert(0, {root!r})
import oracle
from tests import oracle_pins
lib = oracle._load({lib!r})
for pin in oracle_pins.ALL_PINS:
    try:
        pin(lib)
    except Exception as e:
        print("CAUGHT", pin.__name__, type(e).__name__)
        sys.exit(3)
print("SURVIVED")
"""


def _run_mutant(m, tmp):
    name, old, new = m
    with open(obuild.SRC) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutant {name}: pattern must occur exactly once"
    path = os.path.join(tmp, f"{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = os.path.join(tmp, f"lib{name}.so")
    obuild.build(path, lib, extra=["-w"])
    p = subprocess.run([sys.executable, "-c", _RUNNER.format(root=ROOT, lib=lib)],
                       capture_output=True, text=True, timeout=300)
    return name, p.returncode, p.stdout.strip().splitlines()[-1:] if p.stdout else p.stderr[-200:]


def test_every_mutant_is_caught():
    with tempfile.TemporaryDirectory() as tmp:
        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 2)) as ex:
            results = list(ex.map(lambda m: _run_mutant(m, tmp), MUTANTS))
    survivors = [(n, out) for (n, rc, out) in results if rc == 0]
    assert not survivors, f"mutants not caught by any pin: {survivors}"


def test_unmutated_oracle_passes_runner():
    """The runner itself reports SURVIVED for the real oracle."""
    p = subprocess.run([sys.executable, "-c", _RUNNER.format(root=ROOT, lib=obuild.LIB)],
                       capture_output=True, text=True, timeout=300)
    assert p.returncode == 0 and "SURVIVED" in p.stdout, p.stdout + p.stderr
