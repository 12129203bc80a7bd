"""The decode kernels' slice geometry (fp32 estimate + one integer correction,
no 64-bit division) against its exact integer definition, on the host.

The same header the kernels include is compiled host-only with hipcc; the
program checks every slice boundary of several thousand (W, n) pairs, with and
without the per-XCD slice weights."""
import os
import subprocess

import pytest

from paper_2411_01142_amd import _build as B

HERE = os.path.dirname(os.path.abspath(__file__))


def test_slice_geometry_matches_integer_definition(tmp_path):
    try:
        cc = B.hipcc()
    except RuntimeError as e:
        pytest.skip(str(e))
    exe = str(tmp_path / "slice_geom_check")
    subprocess.run([cc, "-x", "hip", "--offload-host-only", "-O2", "-std=c++17",
                    "-I" + B.INCLUDE, "-I" + B.CSRC, os.path.join(HERE, "slice_geom_check.cpp"),
                    "-o", exe], check=True, capture_output=True, text=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.startswith("ok"), res.stdout
