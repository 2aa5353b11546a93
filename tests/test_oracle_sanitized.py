"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer
(host code only): a small driver calls every mode of oracle_partial (bf16 and
e4m3 caches, shared, per-row and token selections, empty and duplicated
slots, the invalid-id path) and oracle_merge (with dead parts) on tiny
inputs; any sanitizer report fails the run.  CPU only."""
import os
import shutil
import subprocess
import tempfile

import pytest

import oracle.build as obuild

DRIVER = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_partial(int R, int Mq, int H, int64_t P, int NB, int K, const uint16_t* q_lat,
                   const uint16_t* q_pe, int kv_kind, const void* ckv, const void* kpe,
                   const float* ckv_scale, const float* kpe_scale, const int32_t* table,
                   const int32_t* sel, int sel_per_row, int sel_tokens, double scale,
                   double* out, double* lse, double* max_out, double* denom_out,
                   int n_threads);
int oracle_merge(int n_parts, int64_t n_rows, int dv, const double* o, const double* lam,
                 double* out, double* lse_out, int n_threads);

static uint32_t st = 12345u;
static uint32_t next(void) { st = st * 1664525u + 1013904223u; return st; }
static uint16_t bf16(void) { return (uint16_t)(0x3c00u + (next() >> 22)) ^ ((next() & 1u) << 15); }

int main(void) {
  enum { R = 2, MQ = 3, H = 5, P = 6, NB = 4, K = 7 };
  uint16_t* ql = malloc(sizeof(uint16_t) * R * MQ * H * 512);
  uint16_t* qp = malloc(sizeof(uint16_t) * R * MQ * H * 64);
  uint16_t* ckv = malloc(sizeof(uint16_t) * P * 64 * 512);
  uint16_t* kpe = malloc(sizeof(uint16_t) * P * 64 * 64);
  uint8_t* ckv8 = malloc((size_t)P * 64 * 512);
  uint8_t* kpe8 = malloc((size_t)P * 64 * 64);
  float cs[P], ks[P];
  for (int i = 0; i < R * MQ * H * 512; ++i) ql[i] = bf16();
  for (int i = 0; i < R * MQ * H * 64; ++i) qp[i] = bf16();
  for (int i = 0; i < P * 64 * 512; ++i) { ckv[i] = bf16(); ckv8[i] = (uint8_t)(next() >> 24) & 0x7e; }
  for (int i = 0; i < P * 64 * 64; ++i) { kpe[i] = bf16(); kpe8[i] = (uint8_t)(next() >> 24) & 0x7e; }
  for (int i = 0; i < P; ++i) { cs[i] = 0.01f * (i + 1); ks[i] = 0.02f * (i + 1); }
  int32_t table[R * NB] = {5, 0, 3, 1, 2, 4, 0, 5};
  int32_t sel[R * K] = {0, 3, -1, 3, 1, -1, 2, -1, -1, -1, -1, -1, -1, -1};
  int32_t sel_rows[R * MQ * K];
  for (int i = 0; i < R * MQ * K; ++i) sel_rows[i] = (int32_t)(next() % (NB + 1)) - 1;
  int32_t sel_tok[R * K];
  for (int i = 0; i < R * K; ++i) sel_tok[i] = (int32_t)(next() % (NB * 64 + 1)) - 1;
  double* out = malloc(sizeof(double) * R * MQ * H * 512);
  double* lse = malloc(sizeof(double) * R * MQ * H);
  double* mx = malloc(sizeof(double) * R * MQ * H);
  double* den = malloc(sizeof(double) * R * MQ * H);
  int rc = 0;
  rc |= oracle_partial(R, MQ, H, P, NB, K, ql, qp, 0, ckv, kpe, NULL, NULL, table, sel, 0, 0, 0.07, out, lse, NULL, NULL, 2);
  rc |= oracle_partial(R, MQ, H, P, NB, K, ql, qp, 1, ckv8, kpe8, cs, ks, table, sel, 0, 0, 0.07, out, lse, mx, den, 2);
  rc |= oracle_partial(R, MQ, H, P, NB, K, ql, qp, 0, ckv, kpe, NULL, NULL, table, sel_rows, 1, 0, 0.07, out, lse, mx, den, 2);
  rc |= oracle_partial(R, MQ, H, P, NB, K, ql, qp, 0, ckv, kpe, NULL, NULL, table, sel_tok, 0, 1, 0.07, out, lse, NULL, NULL, 2);
  rc |= oracle_partial(R, MQ, H, P, NB, K, ql, qp, 1, ckv8, kpe8, cs, ks, table, sel_tok, 0, 1, 0.07, out, lse, NULL, NULL, 2);
  if (rc != 0) { fprintf(stderr, "valid calls failed\n"); return 2; }
  int32_t bad[R * K];
  memcpy(bad, sel, sizeof bad);
  bad[3] = NB;  /* out of range: the call reports it */
  if (oracle_partial(R, MQ, H, P, NB, K, ql, qp, 0, ckv, kpe, NULL, NULL, table, bad, 0, 0, 0.07, out, lse, NULL, NULL, 2) != -1) {
    fprintf(stderr, "invalid id not reported\n");
    return 3;
  }
  enum { N = 4, ROWS = 9, DV = 16 };
  double o[N * ROWS * DV], lam[N * ROWS], mo[ROWS * DV], ml[ROWS];
  for (int i = 0; i < N * ROWS * DV; ++i) o[i] = (double)(next() % 1000) / 500.0 - 1.0;
  for (int i = 0; i < N * ROWS; ++i) lam[i] = (i % 5 == 0) ? -INFINITY : (double)(next() % 100) / 10.0;
  if (oracle_merge(N, ROWS, DV, o, lam, mo, ml, 2) != 0) return 4;
  free(ql); free(qp); free(ckv); free(kpe); free(ckv8); free(kpe8); free(out); free(lse); free(mx); free(den);
  puts("ok");
  return 0;
}
"""


def test_oracle_under_address_and_ub_sanitizers():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    with tempfile.TemporaryDirectory() as tmp:
        drv = os.path.join(tmp, "driver.c")
        exe = os.path.join(tmp, "driver")
        with open(drv, "w") as f:
            f.write(DRIVER)
        cmd = ["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", exe, drv,
               obuild.SRC, "-lm"]
        subprocess.run(cmd, check=True, capture_output=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
        p = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
        assert p.returncode == 0 and "ok" in p.stdout, p.stdout + p.stderr[-2000:]
