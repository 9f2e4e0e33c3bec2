"""Host-side checks of the two measurement scripts: their argument handling and the
work model's launch lists (no GPU)."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import sweep  # noqa: E402
from paper_2106_12736_amd import inputs  # noqa: E402


def _run(*args):
    return subprocess.run([sys.executable, *args], cwd=ROOT, capture_output=True, text=True, timeout=120)


def test_bench_refuses_more_than_one_gpu():
    r = _run("bench.py", "--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_sweep_help_and_table():
    r = _run("sweep.py", "--help")
    assert r.returncode == 0 and "--batch" in r.stdout
    t = sweep.table("t", "k", [("a", {"x": 1.0, "y": None})], ["x", "y"])
    assert "| a | 1.000 | — |" in t


@pytest.mark.parametrize("n,m", [(1024, 512), (512, 256), (64, 32), (256, 256)])
def test_pooled_rfft2_work_model(n, m):
    # fdc_rfft2_pooled_ws: the row pass writes m/2+1 bins of every row (to the
    # workspace), the column pass reads those columns and writes the m kept rows; with no
    # pooling the bytes of the full transform; small planes in one launch
    planes = 8
    got = bench.pooled_rfft2_launches(n, m, planes)
    full = bench.fft2_launches(n, planes, inverse=False)
    if n <= 64:
        assert got == full
        return
    assert [k for k, _ in got] == [f"row_r2c_{n}", f"col_fft_keep_{n}"]
    L = m // 2 + 1
    assert got[0][1] == 4 * planes * n * n + 8 * planes * n * L
    assert got[1][1] == 8 * planes * (n + m) * L
    if m == n:
        assert [b for _, b in got] == [b for _, b in full]
    else:
        assert sum(b for _, b in got) < sum(b for _, b in full)


def test_chain_work_model_starts_with_the_pooled_transform():
    wl = inputs.STACK1024
    launches = bench.chain_step_launches(wl)
    assert launches[:2] == bench.pooled_rfft2_launches(1024, 512, wl.batch * wl.channels[0])
