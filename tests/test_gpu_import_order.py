"""The binding imported before torch, in a fresh process: the package brings torch in first,
so the library binds to torch's HIP runtime and the process holds a single one. A half-sweep
on the small workload then matches the fp64 oracle row by row (relative error <= 1e-4)."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import paper_1108_2580_amd as p  # before torch, on purpose
import sys
import numpy as np
import torch
import oracle
import workload

assert torch.cuda.is_available()
r = workload.make_config(1)
U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
print(f"config 1: {r.M} x {r.N}, nnz {r.row_ptr[-1]}, D {r.D}", flush=True)
with p.ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D) as als:
    out = torch.from_numpy(np.ascontiguousarray(U0, dtype=np.float32)).to("cuda:0")
    fixed = torch.from_numpy(np.ascontiguousarray(V0, dtype=np.float32)).to("cuda:0")
    als.half_sweep("users", fixed, r.lam, out, allow_flagged=True)
    xg = out.cpu().numpy()
xo, fl = oracle.half_sweep(r.row_ptr, r.col, r.val.astype(np.float64), V0, r.lam, U0)
num = np.linalg.norm(xg - xo, axis=1)
rel = num / np.maximum(np.linalg.norm(xo, axis=1), 1e-30)
print(f"rel max {rel.max():.2e}", flush=True)
sys.exit(0 if rel.max() <= 1e-4 and not (fl == 1).any() else 3)
"""


def test_package_imported_before_torch():
    print("child: import paper_1108_2580_amd before torch, one user half-sweep", flush=True)
    res = subprocess.run([sys.executable, "-c", CHILD], cwd=REPO, capture_output=True,
                         text=True, timeout=300)
    print(res.stdout, flush=True)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-2000:]
