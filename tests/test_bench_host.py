"""Host-side logic of bench.py (no GPU): kernel names, stored traffic lookup, and
the refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# ccdpp_info fields of the large layouts: user-major tiled with one tile (streaming),
# item-major tiled with 36 tiles (write-back stores).
INFO = {"value_bytes": 4, "u_gather": 2, "u_tiles": 1, "u_tile_width": 17770, "u_cache": 1,
        "v_gather": 2, "v_tiles": 36, "v_tile_width": 13376, "v_cache": 2}


def test_kernel_symbols_follow_the_layout_and_cache_policy():
    k = bench.kernel_symbol
    assert k(0, INFO, 0) == "void ccdk::ccd_pass_fused<true, true, true, 0, float>(ccdk::PassArgs<float>)"
    assert k(0, INFO, 1) == "void ccdk::ccd_pass_fused<true, true, false, 1, float>(ccdk::PassArgs<float>)"
    # the plain pass stores no residual: the streaming kernel
    assert k(1, INFO, 0) == "void ccdk::ccd_pass<true, true, true, 0, float>(ccdk::PassArgs<float>)"
    assert k(1, INFO, 1) == "void ccdk::ccd_pass<true, true, false, 0, float>(ccdk::PassArgs<float>)"
    assert k(4, INFO, 1) == "void ccdk::ccd_flush<true, true, false, 1, float>(ccdk::PassArgs<float>)"
    # automatic write-back stores apply to CCD++ with two or more inner iterations only
    assert k(0, INFO, 1, wb_stores=False) == \
        "void ccdk::ccd_pass_fused<true, true, false, 0, float>(ccdk::PassArgs<float>)"
    wb_user = dict(INFO, u_cache=2, v_cache=1)
    assert k(0, wb_user, 0) == "void ccdk::ccd_pass_fused<true, true, true, 1, float>(ccdk::PassArgs<float>)"
    assert k(4, wb_user, 1) == "void ccdk::ccd_flush<true, true, false, 0, float>(ccdk::PassArgs<float>)"
    hot = dict(INFO, v_gather=3, v_tiles=1, v_tile_width=40768, value_bytes=8)
    assert k(1, hot, 1) == "void ccdk::ccd_pass<true, false, true, 0, double>(ccdk::PassArgs<double>)"
    assert k(2, INFO, 1) == "void ccdk::ccd_combine<16, float>(ccdk::CombineArgs<float>)"
    # A split item-major copy: its tiled part's kernel, then its hot part's.
    split = dict(INFO, v_tiles=75, v_tile_width=13504, v_cache=1, v_split_rows=36620,
                 v2_gather=3, v2_tile_width=40768, v2_cache=1)
    assert k(1, split, 1) == ("void ccdk::ccd_pass<true, true, false, 0, float>(ccdk::PassArgs<float>)"
                              " + void ccdk::ccd_pass<true, false, true, 0, float>(ccdk::PassArgs<float>)")


def test_stored_traffic_only_for_the_sources_it_was_taken_on():
    # The committed counters carry the digest of the kernel sources they were taken on;
    # bench.py reports them only while the sources are unchanged.
    for wl in ("large", "vlarge"):
        with open(os.path.join(ROOT, "profiles", f"traffic_{wl}.json")) as f:
            t = json.load(f)
        assert len(t["source_digest"]) == 16
        for key, v in t["kernels"].items():
            assert v["bytes_per_launch"] > 0 and v["stored_bytes_per_launch"] > 0
            got = bench.stored_traffic(key, wl)
            if t["source_digest"] == bench.source_digest():
                assert got == v["bytes_per_launch"]
            else:
                assert got is None
    assert bench.stored_traffic("ccd_pass/rows", "no_such_workload") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr)


LARGE = dict(INFO, m=480_189, n=17_770, nnz=100_480_507)


def test_model_bytes_follow_the_byte_model():
    # Plain pass over the user-major copy of the large matrix: 8 B per entry (4-byte
    # index, 4-byte value), row pointers, coordinates, one gathered vector.
    N, m, n = 100_480_507, 480_189, 17_770
    assert bench.model_bytes(1, 0, LARGE) == 8 * N + 4 * (m + 1) + 4 * m + 4 * n
    assert abs(bench.model_bytes(1, 0, LARGE) / 1e6 - 807.8) < 0.05
    # A first pass writes the residual back (12 B per entry), reads two per-row scalars
    # and gathers two (user-major) or three (item-major) vectors.
    assert bench.model_bytes(0, 0, LARGE) == 12 * N + 4 * (m + 1) + 4 * m + 8 * m + 8 * n
    assert bench.model_bytes(0, 1, LARGE) == 12 * N + 4 * (n + 1) + 4 * n + 8 * n + 12 * m
    # The flush reads and writes the residual, one per-row scalar and one vector.
    assert bench.model_bytes(4, 1, LARGE) == 12 * N + 4 * (n + 1) + 4 * n + 4 * m
    # Doubles: 8-byte values and factor entries, still 4-byte indices.
    d = dict(LARGE, value_bytes=8)
    assert bench.model_bytes(1, 1, d) == 12 * N + 4 * (n + 1) + 8 * n + 8 * m
    assert bench.model_bytes(2, 1, LARGE) is None  # the combine is not a pass


def test_host_threads_reports_the_host():
    h = bench.host_threads()
    assert h["cores_all"] == os.cpu_count()
    assert 1 <= h["threads"] <= h["affinity"] <= h["cores_all"]
    assert h["cpu_model"] is None or isinstance(h["cpu_model"], str)
