"""Host logic of bench.py (no GPU): the rocprofv3 counter summaries that the
profiles and the bench line's `traffic` come from, and the refusal of more
than one GPU."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]


def _write(path, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=FIELDS)
        wr.writeheader()
        for r in rows:
            wr.writerow(dict(zip(FIELDS, r)))


SWEEP = "void bgmfk::(anonymous namespace)::k_sgd_lds<64, false>(bgmfk::SgdParams)"
RMSE = "void bgmfk::(anonymous namespace)::k_rmse_lds<64>(...)"
FILL = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>(...)"


def test_pmc_summary_scales_by_the_calibration_copy(tmp_path):
    # a 1 MiB calibration copy (the first copy after the fill) reads 512 KiB
    # of FETCH_SIZE and writes 1024 KiB of WRITE_SIZE: scales 2.0 and 1.0
    f, w = tmp_path / "f.csv", tmp_path / "w.csv"
    _write(f, [(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 7),      # before the fill: ignored
               (2, FILL, "FETCH_SIZE", 0),
               (3, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 512),
               (4, SWEEP, "FETCH_SIZE", 100), (5, SWEEP, "FETCH_SIZE", 300),
               (6, RMSE, "FETCH_SIZE", 10)])
    _write(w, [(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 3),
               (2, FILL, "WRITE_SIZE", 0),
               (3, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024),
               (4, SWEEP, "WRITE_SIZE", 50), (5, SWEEP, "WRITE_SIZE", 150),
               (6, RMSE, "WRITE_SIZE", 0)])
    s = bench.pmc_summary(str(f), str(w), 1)
    assert s["fetch_scale"] == 2.0 and s["write_scale"] == 1.0
    k = s["kernels"][SWEEP]
    assert k["dispatches"] == 2
    assert k["fetch_bytes"] == 200 * 2.0 * 1024      # mean 200 KiB, scaled
    assert k["write_bytes"] == 100 * 1.0 * 1024
    assert k["bytes"] == k["fetch_bytes"] + k["write_bytes"]
    assert "__amd_rocclr_copyBuffer" not in s["kernels"]  # library kernels only


def test_pmc_summary_needs_the_calibration_copy(tmp_path):
    f = tmp_path / "f.csv"
    _write(f, [(1, SWEEP, "FETCH_SIZE", 100)])
    with pytest.raises(ValueError, match="calibration"):
        bench.pmc_summary(str(f), str(f), 1)


def test_pmc_l2_hit_rate(tmp_path):
    c = tmp_path / "l2.csv"
    _write(c, [(1, SWEEP, "TCC_HIT_sum", 90), (1, SWEEP, "TCC_MISS_sum", 10),
               (2, SWEEP, "TCC_HIT_sum", 70), (2, SWEEP, "TCC_MISS_sum", 30),
               (3, "__amd_rocclr_copyBuffer", "TCC_HIT_sum", 5),
               (3, "__amd_rocclr_copyBuffer", "TCC_MISS_sum", 5)])
    out = bench.pmc_l2(str(c))
    assert list(out) == [SWEEP]
    assert out[SWEEP]["dispatches"] == 2
    assert out[SWEEP]["hits"] == 80 and out[SWEEP]["misses"] == 20
    assert out[SWEEP]["hit_rate"] == pytest.approx(0.8)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]
