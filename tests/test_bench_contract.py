"""CPU checks of bench.py's contract: one GPU only, and the algorithmic bytes
the roofline divides by (read x and ref, write the wire and the fp32
reconstruction once; decode reads the wire and ref and writes the
reconstruction), at the headline and uplink shapes."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import paper_2608_04991_amd as rac

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.fixture(scope="module")
def lib():
    try:
        return rac.library()
    except (OSError, RuntimeError) as e:
        pytest.skip(f"librac.so not loadable here: {e}")


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_exits_with_a_message(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env=dict(os.environ, **env), timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _per_elem(b, ga, gq, k, d):
    # x, ref, codes, scale, coefficient pair, outlier entries, fp32 x-hat
    return 2 + 2 + b / 8 + 2 / gq + 4 / ga + 4 * k / d + 4


@pytest.mark.parametrize("T,d,g,b,k,enc,dec", [
    (65536, 3584, 128, 4, 4, 2_008_547_584, 1_538_785_536),  # the headline step's encode and decode
    (4096, 4096, 128, 4, 8, 143_524_096, None),             # the uplink encode
])
def test_algorithmic_bytes(lib, T, d, g, b, k, enc, dec):
    wb = rac.rac_wire_size(rac.RacConfig(T, d, g, g, b, k))
    e = bench.algorithmic_bytes(T, d, wb)
    assert e == enc
    # the wire is the packed fields plus a 256-byte header and section padding
    assert abs(e - T * d * _per_elem(b, g, g, k, d)) <= 256 * 5
    if dec is not None:
        assert bench.algorithmic_bytes(T, d, wb, encode=False) == dec == e - 2 * T * d


def test_fraction_of_peak():
    # 8 TB/s moves 8e12 bytes a second, so 8e6 bytes take 1 us
    assert bench.frac(8_000_000, 1.0) == 1.0
    assert bench.frac(2_008_547_584, 348.5) == round(2_008_547_584 / 348.5e-6 / 8e12, 4)
