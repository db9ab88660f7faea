"""The boundary used from plain C on the GPU: a C99 program, with no Python
in the process, allocates device memory through the HIP C API, writes bf16
gradients of four units (ragged lengths over several work items, constant
magnitudes with a x20 spike in one unit), runs gnmr_init, gnmr_step and
gnmr_query over eight steps and prints every output.  The test compares
them with the oracle fed with the same values: masks, locks and counters
bit-exact, norms and ratios within 1e-5 (here the sums of squares are exact,
so they agree to the last bit in practice)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import BF16
from oracle import Controller as Oracle
from oracle import unit_norm

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
PKG = os.path.join(ROOT, "paper_2606_00539_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

U, T, N = 4, 8, [70001, 65536, 100003, 1]
MAG = [1.0, 0.5, 0.25, 2.0]             # magnitudes in units of 2^-10
SPIKE_UNIT, SPIKE_STEP, SPIKE = 2, 6, 20.0

PROGRAM = r"""
#include <stdio.h>
#include <stdlib.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>
#include "gnmr.h"

#define U 4
#define T 8
static const int64_t N[U] = {70001, 65536, 100003, 1};
static const double MAG[U] = {1.0, 0.5, 0.25, 2.0};

/* bf16 bits of v, which is exactly representable here */
static uint16_t bf16(float v) {
  union { float f; uint32_t u; } x;
  x.f = v;
  return (uint16_t)(x.u >> 16);
}

int main(void) {
  void* dev[U];
  uint16_t* host[U];
  int64_t off[U + 1], numel[U];
  int32_t dt[U];
  const void* ptrs[U];
  gnmr_config cfg = {U, 3, 1, 2, 0.0, NULL, GNMR_BUDGET_ACTIVE, 0};
  gnmr_segments segs;
  gnmr_ctx* ctx = NULL;
  int b, t;
  int64_t i;
  for (b = 0; b < U; ++b) {
    if (hipMalloc(&dev[b], (size_t)N[b] * 2) != hipSuccess) return 10;
    host[b] = (uint16_t*)malloc((size_t)N[b] * 2);
    off[b] = b;
    numel[b] = N[b];
    dt[b] = GNMR_BF16;
    ptrs[b] = dev[b];
  }
  off[U] = U;
  segs.num_segments = U;
  segs.unit_seg_off = off;
  segs.seg_numel = numel;
  segs.seg_dtype = dt;
  segs.seg_ptr = ptrs;
  if (gnmr_init(&ctx, &cfg, &segs, NULL) != GNMR_OK) {
    printf("init failed: %s\n", gnmr_last_error());
    return 11;
  }
  for (t = 1; t <= T; ++t) {
    uint8_t mask[U];
    int32_t lock[U];
    double norm[U], g[U], d[U], r[U];
    gnmr_stats st;
    for (b = 0; b < U; ++b) {
      float c = (float)(MAG[b] / 1024.0);
      if (b == 2 && t == 6) c *= 20.0f;
      for (i = 0; i < N[b]; ++i) host[b][i] = bf16(((i + t) % 3 == 0) ? -c : c);
      if (hipMemcpy(dev[b], host[b], (size_t)N[b] * 2, hipMemcpyHostToDevice) != hipSuccess)
        return 12;
    }
    if (gnmr_step(ctx, 1.5, 1.5, NULL, NULL) != GNMR_OK) {
      printf("step failed: %s\n", gnmr_last_error());
      return 13;
    }
    if (gnmr_query(ctx, mask, lock, norm, g, d, r, &st, NULL) != GNMR_OK) return 14;
    for (b = 0; b < U; ++b)
      printf("%d %d %d %d %.17g %.17g %.17g %.17g\n", t, b, mask[b], lock[b], norm[b], g[b],
             d[b], r[b]);
    printf("stats %d %lld %d %d %d %d %d %d %d\n", t, (long long)st.t, st.n_trig_gnmr,
           st.n_trig_dgnmr, st.n_trig, st.n_cand, st.n_active, st.hit_maxo, st.n_nonfinite);
  }
  gnmr_destroy(ctx);
  for (b = 0; b < U; ++b) {
    hipFree(dev[b]);
    free(host[b]);
  }
  return 0;
}
"""


def host_values(b, t):
    c = np.float32(MAG[b] / 1024.0)
    if b == SPIKE_UNIT and t == SPIKE_STEP:
        c = np.float32(c * np.float32(SPIKE))
    i = np.arange(N[b])
    v = np.where((i + t) % 3 == 0, -c, c).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def test_c_program_runs_the_controller_on_the_gpu(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc is not installed")
    src = tmp_path / "gnmr_c.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "gnmr_c"
    r = subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                        "-I", INCLUDE, "-I", os.path.join(ROCM, "include"), str(src), "-o",
                        str(exe), "-L", PKG, "-lgnmr", "-L", os.path.join(ROCM, "lib"),
                        "-lamdhip64", f"-Wl,-rpath,{PKG}", f"-Wl,-rpath,{ROCM}/lib"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    print("running the C program", flush=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout[-2000:], r.stderr[-2000:])
    rows, stats = {}, {}
    for line in r.stdout.splitlines():
        f = line.split()
        if f[0] == "stats":
            stats[int(f[1])] = [int(x) for x in f[2:]]
        elif len(f) == 8:
            rows[(int(f[0]), int(f[1]))] = f[2:]
    ora = Oracle(U, window=3, max_o=1, lock_len=2, eps=0.0)
    keys = ("t", "n_trig_gnmr", "n_trig_dgnmr", "n_trig", "n_cand", "n_active", "hit_maxo",
            "n_nonfinite")
    spiked = False
    for t in range(1, T + 1):
        ref = ora.step([unit_norm([(host_values(b, t), BF16)]) for b in range(U)], 1.5, 1.5)
        assert stats[t] == [ref.stats[k] for k in keys], (t, stats[t], ref.stats)
        for b in range(U):
            mask, lock, norm, g, d, rr = rows[(t, b)]
            assert int(mask) == ref.mask[b] and int(lock) == ref.lock[b], (t, b)
            for got, want in zip((norm, g, d, rr), (ref.norm[b], ref.gnmr[b], ref.dgnmr[b],
                                                     ref.risk[b])):
                assert abs(float(got) - want) <= 1e-5 * abs(want), (t, b, got, want)
        spiked |= bool(ref.mask[SPIKE_UNIT])
    assert spiked                                 # the spike reached the recovery path
