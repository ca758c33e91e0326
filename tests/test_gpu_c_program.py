"""The library driven from a plain C program on the device: no Python and no
torch in that process.  Device buffers come from hipMalloc and the calls run
on the null stream; one training step (sections 3.2-3.4) and one forward pass
are checked against the CPU reference."""

import os
import subprocess

import numpy as np
import pytest

from oracle import mlp
from paper_1902_06714_amd import nf

from . import parity
from .gpu_run import note

pytestmark = pytest.mark.gpu

DIMS = (20, 16, 5)
BATCH = 37
ETA = 2.0

PROGRAM = r"""
#include <stdio.h>
#include <stdlib.h>
#include <hip/hip_runtime_api.h>
#include "nf.h"

static int io(const char* dir, const char* name, float* buf, size_t n, int write) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, write ? "wb" : "rb");
  if (!f) return 0;
  const size_t done = write ? fwrite(buf, sizeof(float), n, f) : fread(buf, sizeof(float), n, f);
  fclose(f);
  return done == n;
}

int main(int argc, char** argv) {
  if (argc != 2) return 2;
  const char* dir = argv[1];
  const int32_t dims[3] = {20, 16, 5};
  const int64_t B = 37;
  const size_t np = 20 * 16 + 16 + 16 * 5 + 5, nx = (size_t)B * 20, ny = (size_t)B * 5;
  float* theta = malloc(np * sizeof(float));
  float* x = malloc(nx * sizeof(float));
  float* y = malloc(ny * sizeof(float));
  float* out = malloc(ny * sizeof(float));
  if (!theta || !x || !y || !out) return 3;
  if (!io(dir, "theta0.bin", theta, np, 0) || !io(dir, "x.bin", x, nx, 0) ||
      !io(dir, "y.bin", y, ny, 0))
    return 4;
  nf_net* net = NULL;
  if (nf_net_create(dims, 3, NULL, 0, &net) != NF_OK) return 10;
  if (nf_param_count(net) != (int64_t)np) return 11;
  if (nf_set_params(net, theta, (int64_t)np) != NF_OK) return 12;
  float *dx = NULL, *dy = NULL, *dout = NULL;
  if (hipMalloc((void**)&dx, nx * sizeof(float)) != hipSuccess ||
      hipMalloc((void**)&dy, ny * sizeof(float)) != hipSuccess ||
      hipMalloc((void**)&dout, ny * sizeof(float)) != hipSuccess)
    return 13;
  if (hipMemcpy(dx, x, nx * sizeof(float), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(dy, y, ny * sizeof(float), hipMemcpyHostToDevice) != hipSuccess)
    return 14;
  if (nf_train_batch(net, dx, dy, B, 2.0f, 1, NULL) != NF_OK) return 15;
  if (nf_forward(net, dx, B, dout, NULL) != NF_OK) return 16;
  if (hipDeviceSynchronize() != hipSuccess) return 17;
  if (nf_get_params(net, theta, (int64_t)np) != NF_OK) return 18;
  if (hipMemcpy(out, dout, ny * sizeof(float), hipMemcpyDeviceToHost) != hipSuccess) return 19;
  if (!io(dir, "theta1.bin", theta, np, 1) || !io(dir, "out.bin", out, ny, 1)) return 20;
  nf_net_destroy(net);
  hipFree(dx);
  hipFree(dy);
  hipFree(dout);
  free(theta);
  free(x);
  free(y);
  free(out);
  puts("done");
  return 0;
}
"""


def test_c_program_trains_and_infers(tmp_path):
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    libdir = os.path.dirname(nf.LIB_PATH)
    src = tmp_path / "prog.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "prog"
    build = subprocess.run(
        ["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
         "-I", os.path.join(rocm, "include"), "-I", os.path.dirname(nf.HEADER), str(src),
         "-L", libdir, "-lnf", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
         f"-Wl,-rpath,{libdir}", f"-Wl,-rpath,{os.path.join(rocm, 'lib')}", "-o", str(exe)],
        capture_output=True, text=True)
    assert build.returncode == 0, build.stderr

    rng = np.random.default_rng(42)
    parts = []
    for l in range(1, len(DIMS)):
        parts.append(rng.normal(0, 1 / np.sqrt(DIMS[l - 1]), DIMS[l] * DIMS[l - 1]))
        parts.append(rng.normal(0, 1, DIMS[l]))
    theta0 = np.concatenate(parts).astype(np.float32)
    X = rng.uniform(0, 1, (BATCH, DIMS[0])).astype(np.float32)
    Y = np.zeros((BATCH, DIMS[-1]), np.float32)
    Y[np.arange(BATCH), rng.integers(0, DIMS[-1], BATCH)] = 1.0
    theta0.tofile(tmp_path / "theta0.bin")
    X.tofile(tmp_path / "x.bin")
    Y.tofile(tmp_path / "y.bin")

    note(f"C program dims={DIMS} batch={BATCH}")
    run = subprocess.run([str(exe), str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0 and run.stdout.strip() == "done", (run.returncode, run.stderr)

    acts = ["sigmoid"] * (len(DIMS) - 1)
    ref, _ = mlp.train_batch(theta0, DIMS, acts, X, Y, ETA)
    theta1 = np.fromfile(tmp_path / "theta1.bin", np.float32)
    out = np.fromfile(tmp_path / "out.bin", np.float32).reshape(BATCH, DIMS[-1])
    fails = parity.check_params(theta1, ref, DIMS)
    assert not fails, "\n".join(fails)
    e, i = parity.floored_rel(out, mlp.output(theta1.astype(np.float64), DIMS, acts, X))
    assert e <= parity.OUT_TOL, (e, i)
