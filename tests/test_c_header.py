"""The boundary as C sees it: include/gnmr.h compiles on its own as C99 and
as C++ with every warning an error, and a plain C program links against
libgnmr.so and gets the documented status codes from calls that fail in
their argument checks (no device call is made).  CPU only."""
import ctypes
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
PKG = os.path.join(ROOT, "paper_2606_00539_amd")

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "gnmr.h"

static int fails = 0;
#define EXPECT(cond) do { if (!(cond)) { printf("FAIL line %d: %s\n", __LINE__, #cond); ++fails; } } while (0)

int main(void) {
  gnmr_ctx* ctx = (gnmr_ctx*)1;
  int64_t off[2] = {0, 0};
  gnmr_segments segs;
  gnmr_config cfg;
  gnmr_wgrad_problem prob;
  memset(&segs, 0, sizeof segs);
  memset(&cfg, 0, sizeof cfg);
  memset(&prob, 0, sizeof prob);
  segs.unit_seg_off = off;
  cfg.num_units = 1;
  cfg.window = 0;                                   /* delta must be >= 1 */
  EXPECT(gnmr_init(&ctx, &cfg, &segs, NULL) == GNMR_E_INVALID);
  EXPECT(ctx == NULL);
  EXPECT(strlen(gnmr_last_error()) > 0);
  EXPECT(gnmr_init(NULL, &cfg, &segs, NULL) == GNMR_E_INVALID);
  EXPECT(gnmr_step(NULL, 1.5, 1.5, NULL, NULL) == GNMR_E_INVALID);
  EXPECT(gnmr_destroy(NULL) == GNMR_OK);
  EXPECT(gnmr_actuator_destroy(NULL) == GNMR_OK);
  EXPECT(gnmr_wgrad_num_tiles(5120, 13824) == 20 * 54);
  EXPECT(gnmr_wgrad_num_tiles(0, 8) == 0);
  EXPECT(gnmr_wgrad_sumsq((const void*)4096, (const void*)8192, (void*)16384, 16, 12, 128,
                          (float*)32768, NULL) == GNMR_E_INVALID);  /* 12: not a multiple of 8 */
  prob.dy = (const void*)4096; prob.x = (const void*)8192; prob.dw = (void*)16384;
  prob.tokens = 16; prob.out_features = 64; prob.in_features = 128; prob.accumulate = 2;
  EXPECT(gnmr_wgrad_sumsq_batched(&prob, 1, (float*)32768, NULL) == GNMR_E_INVALID);
  EXPECT(gnmr_actuate_matrix((const void*)4096, (void*)8192, 4, 12, (const uint8_t*)65536, 0,
                             GNMR_FMT_E2M1, GNMR_FMT_BF16, NULL) == GNMR_E_INVALID);
  EXPECT(gnmr_actuate_matrix(NULL, NULL, 0, 64, NULL, 0, GNMR_FMT_INT8, GNMR_FMT_BF16,
                             NULL) == GNMR_OK);     /* no rows: nothing to do */
  EXPECT(gnmr_actuate(NULL, NULL, GNMR_FMT_E2M1, GNMR_FMT_BF16, NULL) == GNMR_E_INVALID);
  {  /* the allocation-free pass: refused in its host checks, before any device call */
    int64_t uoff[2] = {0, 1}, numel[1] = {(int64_t)1 << 36};  /* 2^21 bf16 items: 40 MiB */
    int32_t dt[1] = {GNMR_BF16};
    const void* ptrs[1] = {(const void*)4096};
    gnmr_segments big;
    big.num_segments = 1; big.unit_seg_off = uoff; big.seg_numel = numel;
    big.seg_dtype = dt; big.seg_ptr = ptrs;
    EXPECT(GNMR_NOALLOC_SCRATCH_BYTES == 32u << 20);
    EXPECT(gnmr_sumsq_noalloc(1, &big, (double*)8192, NULL) == GNMR_E_INVALID);
    EXPECT(strstr(gnmr_last_error(), "scratch") != NULL);
    big.seg_ptr = NULL;
    EXPECT(gnmr_sumsq_noalloc(1, &big, (double*)8192, NULL) == GNMR_E_INVALID);
    EXPECT(gnmr_sumsq_noalloc(0, &big, (double*)8192, NULL) == GNMR_E_INVALID);
  }
  printf("sizes %d %d %d %d %d\n", (int)sizeof(gnmr_config), (int)sizeof(gnmr_segments),
         (int)sizeof(gnmr_stats), (int)sizeof(gnmr_wgrad_problem), (int)sizeof(gnmr_act_segment));
  return fails;
}
"""


def compiler(name):
    path = shutil.which(name)
    if path is None:
        pytest.skip(f"{name} is not installed")
    return path


@pytest.mark.parametrize("lang", ["c99", "c11", "c++11", "c++17"])
def test_header_compiles_alone(tmp_path, lang):
    cc = compiler("g++" if lang.startswith("c++") else "gcc")
    src = tmp_path / ("h.cpp" if lang.startswith("c++") else "h.c")
    src.write_text('#include "gnmr.h"\n#include "gnmr.h"\nint gnmr_header_check;\n')
    r = subprocess.run([cc, f"-std={lang}", "-Wall", "-Wextra", "-Werror", "-pedantic",
                        "-I", INCLUDE, "-c", str(src), "-o", str(tmp_path / "h.o")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_program_links_and_gets_documented_statuses(tmp_path):
    cc = compiler("gcc")
    lib = os.path.join(PKG, "libgnmr.so")
    if not os.path.exists(lib):
        pytest.skip("libgnmr.so is not built")
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "abi"
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", INCLUDE,
                        str(src), "-o", str(exe), "-L", PKG, "-lgnmr", f"-Wl,-rpath,{PKG}"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    # the struct layouts C sees are the ones the Python binding declares
    from paper_2606_00539_amd import binding as B

    sizes = [int(v) for v in r.stdout.split("sizes")[1].split()]
    assert sizes == [ctypes.sizeof(B.gnmr_config), ctypes.sizeof(B.gnmr_segments),
                     ctypes.sizeof(B.gnmr_stats), ctypes.sizeof(B.gnmr_wgrad_problem),
                     ctypes.sizeof(B.gnmr_act_segment)]
