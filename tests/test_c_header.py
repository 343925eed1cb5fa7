"""The public headers are plain C: a C99 program includes them with every
warning an error, links against liblsgd.so and calls the entry points that
need no GPU (status strings, the host learning-rate schedule, the tuning
knobs, argument validation)."""
import os
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_1906_05936_amd")

PROGRAM = r"""
#include <math.h>
#include <stdio.h>
#include <string.h>
#include "lsgd.h"
#include "lsgd_bench.h"

int main(void) {
    lsgd_lr_schedule s = {0.1, 256.0, 16384.0, 390, 2340, 0.1};
    float lr0 = lsgd_lr_at(&s, 0), lr1 = lsgd_lr_at(&s, 390);
    int32_t c = 0, b = 0, u = 0;
    if (lsgd_get_launch_shape(&c, &b, &u) != LSGD_OK || c != LSGD_XCD_CHUNK_AUTO) return 1;
    if (lsgd_get_copy_out_mode() != LSGD_COPY_OUT_AUTO) return 2;
    if (lsgd_set_copy_out_mode(7) != LSGD_ERR_SIZE) return 3;
    if (strlen(lsgd_last_error()) == 0) return 4;
    if (lsgd_step_plan(NULL, 0.1f, 0.9f, 1e-4f, NULL) != LSGD_ERR_NULL) return 5;
    if (lsgd_stream_copy(NULL, NULL, 15, NULL) != LSGD_ERR_SIZE) return 6;
    if (!isnan(lsgd_lr_at(NULL, 0))) return 7;
    printf("%s|%.9g|%.9g\n", lsgd_status_string(LSGD_ERR_ALIAS), lr0, lr1);
    return 0;
}
"""


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="host-only program; runs where no GPU is visible")
def test_headers_compile_as_c99_and_link(tmp_path):
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "abi"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I" + os.path.join(ROOT, "include"),
           str(src), "-o", str(exe), "-L" + LIB_DIR, "-llsgd", "-Wl,-rpath," + LIB_DIR, "-lm"]
    subprocess.run(cmd, check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=60).stdout.strip()
    name, lr0, lr1 = out.split("|")
    assert name.startswith("LSGD_ERR_ALIAS")
    assert float(lr0) == pytest.approx(0.1) and float(lr1) == pytest.approx(6.4)
