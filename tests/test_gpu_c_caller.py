"""The C ABI from a plain C program (tests/c/abi_caller.c, built here with gcc against
include/ccdpp.h and libccdpp.so): no Python or PyTorch in that process.  Its factors
match the fp64 oracle, and bit for bit what the Python binding computes from the
same inputs."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP
from gpu_util import colscaled_max_rel_err

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_1511_02433_amd")
M, N, K, LAM, OUTER, INNER = 3000, 1200, 4, 0.05, 2, 3


def test_plain_c_caller(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    exe = str(tmp_path / "abi_caller")
    subprocess.run([gcc, "-O2", "-std=c11", "-Wall", f"-I{os.path.join(ROOT, 'include')}",
                    os.path.join(ROOT, "tests", "c", "abi_caller.c"), f"-L{PKG}", "-lccdpp",
                    f"-Wl,-rpath,{PKG}", "-o", exe], check=True, timeout=120)
    row, col, val, H0 = synth.small_random(M, N, 80_000, K, seed=123)
    (tmp_path / "problem.txt").write_text(f"{M} {N} {K} {LAM!r} {row.size} {OUTER} {INNER}\n")
    row.tofile(tmp_path / "row.bin")
    col.tofile(tmp_path / "col.bin")
    val.tofile(tmp_path / "val.bin")
    np.ascontiguousarray(H0, np.float32).tofile(tmp_path / "H0.bin")
    print(f"case: C caller m={M} n={N} k={K} nnz={row.size}", flush=True)
    r = subprocess.run([exe, str(tmp_path)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    Wc = np.fromfile(tmp_path / "W.bin", np.float32).reshape(M, K)
    Hc = np.fromfile(tmp_path / "H.bin", np.float32).reshape(N, K)
    rmse_c, mism = (tmp_path / "out.txt").read_text().split()
    assert int(mism) == 0

    o = Oracle(M, N, K, LAM, row, col, val, H0)
    o.run(OUTER, INNER)
    Wo, Ho = o.factors()
    assert colscaled_max_rel_err(Wc, Wo) <= 1e-3 and colscaled_max_rel_err(Hc, Ho) <= 1e-3
    assert abs(float(rmse_c) - o.train_rmse()) <= 1e-4

    g = CCDPP(M, N, K, LAM, row, col, val)
    g.set_factors(np.zeros((M, K), np.float32), H0)
    g.run(OUTER, INNER)
    Wp, Hp = g.factors()
    assert np.array_equal(Wc, Wp) and np.array_equal(Hc, Hp)
    assert float(rmse_c) == g.train_rmse()
    g.close()
