"""The allocation-free entry point ccdpp_rmse_noalloc against ccdpp_rmse.

ccdpp_rmse copies the held-out triplets from the host and sums in memory the
handle owns; ccdpp_rmse_noalloc takes them in device memory and sums in the
library's fixed per-device scratch array.  On the same triplets the two must
give bitwise the same RMSE (same kernel, same fixed order), call after call:
here two calls in a row, the second on a smaller set, so that the second reads
nothing the first left behind.  The held-out RMSE of Section 8 is also checked
against the oracle.  While the call runs, the library's next device allocation
is armed to fail: the call must still succeed, and the armed failure must still
be there for the allocating ccdpp_rmse afterwards.  Entries out of range or not
finite are refused with EINVAL, without being used as indices.
"""
import numpy as np
import pytest

import paper_1511_02433_amd.ccdpp as C
from oracle import Oracle
from paper_1511_02433_amd import synth
from paper_1511_02433_amd.ccdpp import CCDPP

pytestmark = pytest.mark.gpu


def _device(a, dtype):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).cuda()


def test_rmse_noalloc_matches_rmse_on_two_calls():
    import torch
    torch.cuda.set_device(0)
    ds = synth.load("tiny")
    w = ds.workload
    g = CCDPP(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val)
    g.set_factors(np.zeros((w.m, w.k), np.float32), ds.H0)
    g.run(2, w.inner)
    o = Oracle(w.m, w.n, w.k, w.lam, ds.row, ds.col, ds.val, ds.H0)
    o.run(2, w.inner)
    # Held-out triplets plus training ones, so that every block of the kernel has work.
    r = np.concatenate([ds.test_row, ds.row[:40_000]])
    c = np.concatenate([ds.test_col, ds.col[:40_000]])
    v = np.concatenate([ds.test_val, ds.val[:40_000]])
    for size in (r.size, 3_001):  # the second call on a smaller input
        dr, dc, dv = _device(r[:size], np.int32), _device(c[:size], np.int32), _device(v[:size], np.float32)
        torch.cuda.synchronize()
        C.ccdpp_debug_inject(0, 0)  # the next device allocation of the library fails
        try:
            got = g.rmse_noalloc(size, dr.data_ptr(), dc.data_ptr(), dv.data_ptr())
            with pytest.raises(C.CCDPPError) as ei:  # still armed: nothing was allocated
                g.rmse(r[:size], c[:size], v[:size])
            assert ei.value.code == C.CCDPP_ENOMEM
        finally:
            C.ccdpp_debug_inject(0, -1)
        ref = g.rmse(r[:size], c[:size], v[:size])
        orc = o.test_rmse(r[:size], c[:size], v[:size])
        print(f"size {size}: noalloc {got!r}, rmse {ref!r}, oracle {orc!r}", flush=True)
        assert got == ref
        assert abs(got - orc) <= 1e-4
    g.close()
    o.close()


def test_rmse_noalloc_refuses_bad_triplets():
    import torch
    torch.cuda.set_device(0)
    row, col, val, H0 = synth.small_random(300, 200, 5_000, 3, seed=8)
    g = CCDPP(300, 200, 3, 0.1, row, col, val)
    g.run(1, 1)
    # (the tensors are kept alive while the library reads them)
    dr, dc, dv = _device(row, np.int32), _device(col, np.int32), _device(val, np.float32)
    torch.cuda.synchronize()
    good = g.rmse_noalloc(row.size, dr.data_ptr(), dc.data_ptr(), dv.data_ptr())
    assert good == g.rmse(row, col, val)
    for bad in ("row", "col", "val"):
        r, c, v = row.copy(), col.copy(), val.copy()
        if bad == "row":
            r[17] = 300
        elif bad == "col":
            c[4_000] = -1
        else:
            v[2_500] = np.inf
        br, bc, bv = _device(r, np.int32), _device(c, np.int32), _device(v, np.float32)
        torch.cuda.synchronize()
        with pytest.raises(C.CCDPPError) as ei:
            g.rmse_noalloc(r.size, br.data_ptr(), bc.data_ptr(), bv.data_ptr())
        assert ei.value.code == C.CCDPP_EINVAL
        assert "1 held-out entries" in str(ei.value)
    with pytest.raises(C.CCDPPError) as ei:
        g.rmse_noalloc(0, 0, 0, 0)
    assert ei.value.code == C.CCDPP_EINVAL
    # still usable, and the scratch serves the next call
    assert g.rmse_noalloc(row.size, dr.data_ptr(), dc.data_ptr(), dv.data_ptr()) == good
    g.close()
