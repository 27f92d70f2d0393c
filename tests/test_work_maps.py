"""The kernels' workgroup -> work maps (XCD-contiguous ranges, and the
(tile group, token block) order of the matrix-core kernels) are bijections:
every output tile is computed by exactly one workgroup.  The maps are the
kernels' own header functions, compiled for the host by hipcc; the check runs
on the CPU over every grid size up to 4200 workgroups and every (group,
token block) grid up to 180 x 40.  Full-size parity tests sample outputs, so
a map that skipped or repeated a tile could hide there."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _hipcc():
    for p in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if p and os.path.exists(p):
            return p
    pytest.skip("hipcc not found")


def test_workgroup_maps_are_bijections(tmp_path):
    exe = str(tmp_path / "work_maps")
    src = os.path.join(HERE, "host", "work_maps.hip")
    cmd = [_hipcc(), "-O2", "-std=c++17", "--offload-arch=gfx950", "-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(ROOT, "paper_2406_13868_amd", "csrc"), src, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "work maps ok" in r.stdout, r.stdout + r.stderr
