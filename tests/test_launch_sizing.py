"""Host path of every compute entry point over degenerate and full-size
shapes, on the CPU, in the library's launch check mode: no host arithmetic
trap or crash (the driver runs in a child process, so a SIGFPE from an
integer division by zero shows up as its exit signal), every call returns
its expected status, and every kernel launch configuration is within the
gfx950 limits (grid, workgroup size, LDS)."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_launch_sizing_over_degenerate_shapes():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "launch_sizing_cases.py")], capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, f"driver ended with {r.returncode}\n{r.stderr[-3000:]}"
    out = json.loads(r.stdout.strip().splitlines()[-1])
    assert not out["bad_status"], out["bad_status"]
    assert not out["bad_launches"], out["bad_launches"]
    assert out["calls"] > 10000 and out["launches"] > out["calls"]
    for k in ("gemm_fast_kernel", "gemm_kernel", "wtile_kernel", "fold_kernel", "build3_kernel", "gemm_dma32_kernel", "gemm_dma_pers_kernel",
              "expand_kernel",
              "radix_hist_kernel",
              "embed_segsum_kernel", "quant_vec_kernel<8>", "reg_core_kernel"):
        assert k in out["kernels"], k
