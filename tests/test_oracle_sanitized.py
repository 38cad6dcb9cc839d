"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

A small C driver steps the oracle over edge sizes (n = 0, 1, 7, 8, 1000),
K = 1..5 and 64, both replica types, all eight switch combinations, a
rollback round and NaN/Inf inputs, and takes the decision from exactly sized
Gram arrays (same K and switches, NaN/Inf entries), with the sanitizers
aborting on the first report.  Only host code is compiled here (gcc), nothing for a GPU.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include "edit_oracle.h"

static uint64_t s = 88172645463325252ull;
static double uni(void) { s ^= s << 13; s ^= s >> 7; s ^= s << 17; return (s >> 11) * 0x1.0p-53; }

static int run(int K, int64_t n, int bf16, uint32_t flags, int poison) {
  oracle_cfg_t cfg = {0.8, 0.85, 0.05, 1e-6, 0.02, 3.0, 2, flags};
  oracle_ema_t ema = {{0}, {0}, 0};
  oracle_record_t rec;
  float *theta = malloc(sizeof(float) * (n ? n : 1)), *mom = calloc(n ? n : 1, sizeof(float));
  void *reps[ORACLE_MAX_K];
  for (int64_t i = 0; i < n; ++i) theta[i] = (float)(0.02 * (uni() - 0.5));
  for (int j = 0; j < K; ++j) reps[j] = malloc((bf16 ? 2 : 4) * (n ? n : 1));
  for (int round = 0; round < 5; ++round) {
    double scale = round == 4 ? 100.0 : 1.0;  /* every worker x100: rollback after the warm-up */
    for (int j = 0; j < K; ++j)
      for (int64_t i = 0; i < n; ++i) {
        float r = (float)(theta[i] + scale * 1e-3 * (uni() - 0.5));
        if (bf16) ((uint16_t *)reps[j])[i] = oracle_f32_to_bf16(r);
        else ((float *)reps[j])[i] = r;
      }
    if (poison && n > 0 && K > 1) {
      if (bf16) ((uint16_t *)reps[1])[n - 1] = 0x7fc0; else ((float *)reps[1])[n - 1] = NAN;
      if (bf16) ((uint16_t *)reps[0])[0] = 0x7f80; else ((float *)reps[0])[0] = INFINITY;
    }
    if (oracle_step(&cfg, K, n, bf16, theta, mom, reps, &ema, &rec) != 0) return 1;
  }
  for (int j = 0; j < K; ++j) free(reps[j]);
  free(theta);
  free(mom);
  return 0;
}

/* The decision from a Gram matrix, over an exactly sized heap array. */
static int run_gram(int K, uint32_t flags, int poison) {
  oracle_cfg_t cfg = {0.8, 0.85, 0.05, 1e-6, 0.02, 3.0, 2, flags};
  oracle_ema_t ema = {{0}, {0}, 0};
  oracle_record_t rec;
  const int np = K * (K + 1) / 2;
  double *gram = malloc(sizeof(double) * np);
  for (int round = 0; round < 5; ++round) {
    for (int p = 0; p < np; ++p) gram[p] = 1e-3 * (uni() - 0.25);
    for (int j = 0, p = 0; j < K; p += K - j, ++j) gram[p] = (round == 4 ? 1e4 : 1.0) * 1e-2 * (1.0 + uni());
    if (poison && K > 1) { gram[1] = NAN; gram[np - 1] = INFINITY; }
    if (oracle_decide_gram(&cfg, K, gram, &ema, &rec) != 0) return 1;
  }
  free(gram);
  return 0;
}

int main(void) {
  const int Ks[] = {1, 2, 3, 4, 5, 64};
  const int64_t ns[] = {0, 1, 7, 8, 1000};
  int runs = 0;
  for (unsigned k = 0; k < sizeof Ks / sizeof Ks[0]; ++k)
    for (unsigned m = 0; m < sizeof ns / sizeof ns[0]; ++m)
      for (int bf16 = 0; bf16 < 2; ++bf16)
        for (uint32_t flags = 0; flags < 8; ++flags)
          for (int poison = 0; poison < 2; ++poison) {
            if (run(Ks[k], ns[m], bf16, flags, poison)) { printf("step failed\n"); return 1; }
            ++runs;
          }
  for (unsigned k = 0; k < sizeof Ks / sizeof Ks[0]; ++k)
    for (uint32_t flags = 0; flags < 8; ++flags)
      for (int poison = 0; poison < 2; ++poison) {
        if (run_gram(Ks[k], flags, poison)) { printf("decision failed\n"); return 1; }
        ++runs;
      }
  /* bad arguments are refused, not dereferenced */
  oracle_cfg_t cfg = {0.8, 0.85, 10, 1e-6, 0.02, 3, 10, 7};
  oracle_ema_t ema = {{0}, {0}, 0};
  if (oracle_step(&cfg, 0, 4, 0, NULL, NULL, NULL, &ema, NULL) != -1) return 2;
  if (oracle_step(&cfg, 65, 4, 0, NULL, NULL, NULL, &ema, NULL) != -1) return 2;
  if (oracle_step(&cfg, 2, 4, 0, NULL, NULL, NULL, &ema, NULL) != -1) return 2;
  double g[3] = {1, 0, 1};
  if (oracle_decide_gram(&cfg, 2, NULL, &ema, NULL) != -1) return 2;
  if (oracle_decide_gram(&cfg, 0, g, &ema, NULL) != -1) return 2;
  if (oracle_decide_gram(&cfg, 65, g, &ema, NULL) != -1) return 2;
  printf("ok %d runs\n", runs);
  return 0;
}
"""


def test_oracle_clean_under_asan_and_ubsan(tmp_path):
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no gcc")
    (tmp_path / "driver.c").write_text(DRIVER)
    exe = tmp_path / "driver"
    sanitize = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    subprocess.run([cc, "-std=c11", "-O1", "-g", *sanitize, "-ffp-contract=off",
                    "-I", os.path.join(ROOT, "oracle"), str(tmp_path / "driver.c"),
                    os.path.join(ROOT, "oracle", "edit_oracle.c"), "-lm", "-o", str(exe)], check=True)
    # the environment is passed on unchanged; ASan is told not to insist on
    # being first in the library load order
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok ")
