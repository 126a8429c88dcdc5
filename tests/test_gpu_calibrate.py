"""GPU parity of the offline calibration: the error reduction against the
oracle's correctly rounded binary64 sums, and the native search against the
oracle-driven search on uplink (outlier mode: g_a, g_q, q, k_g) and
decode-phase (g_a, g_q, q) samples.

The GPU sums take a fixed pairwise order, the oracle's are correctly rounded;
both add the same binary64 squares, so they agree to a few units of 1e-16
relative (the bar below is 1e-12).  The maximum is exact on both sides.  The
chosen configuration must be the same, and the costs equal rac_wire_size.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import paper_2608_04991_amd as rac
from oracle import calibrate as ocal
from paper_2608_04991_amd import workloads as wl
from tests.gpu_util import cfgd, say, to_dev

pytestmark = pytest.mark.gpu
GRP = rac.RAC_FLAG_GROUP_OUTLIERS
RTOL = 1e-12


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rac.library()


def _gpu_error(xb, xhat, flags=0):
    import torch
    T, d = xb.shape
    x = to_dev(xb)
    h = np.ascontiguousarray(xhat)
    h = torch.from_numpy(h.view(np.int16) if h.dtype == np.uint16 else h).cuda()
    st = torch.full((3,), -1.0, dtype=torch.float64, device="cuda")
    ws = torch.empty(max(rac.rac_recon_error_workspace(T), 8), dtype=torch.uint8, device="cuda")
    rac.rac_recon_error(T, d, x, h, st, ws, flags)
    torch.cuda.synchronize()
    return st.cpu().numpy().tolist()


def _close(a, b):
    return abs(a - b) <= RTOL * abs(b)


@pytest.mark.parametrize("T,d,bf16", [(4096, 4096, False), (37, 520, False), (1, 8, False), (29, 4096, True),
                                      (0, 512, False)])
def test_error_sums_match_the_oracle(T, d, bf16):
    say(f"[gpu] error reduction {T}x{d} bf16={bf16}")
    if T:
        src = wl.prefill_uplink(0, rows=(0, T), hidden=d) if d % 128 == 0 else \
            wl.affine_pair(wl.AffineRecipe(T, d, 8), 0)
        xb, rb = src[0], src[1]
    else:
        xb = np.zeros((0, d), np.uint16)
        rb = xb
    c = cfgd(T, d, 128 if d % 128 == 0 else 8, 128 if d % 128 == 0 else 8, 4, 4 if d >= 4 else 0,
             rac.RAC_FLAG_XHAT_BF16 if bf16 else 0)
    rc, _, xhat = oracle.encode(xb, rb, **c)
    assert rc == 0
    se, sx, mx = _gpu_error(xb, xhat, c["flags"])
    ose, osx, omx = ocal.error_stats(xb, xhat, bf16)
    assert _close(se, ose) and _close(sx, osx) and mx == omx, ((se, sx, mx), (ose, osx, omx))


def _target_between(nmses):
    """A target strictly between two neighbouring distinct candidate errors
    near the middle, far (relative 1e-3) from every candidate's."""
    v = sorted(set(nmses))
    i = len(v) // 2
    t = math.sqrt(v[i - 1] * v[i])
    assert all(abs(t - e) > 1e-3 * e for e in v)
    return t


def _run(xb, rb, configs, label):
    say(f"[gpu] calibration {label}: {len(configs)} candidates, oracle first")
    odicts = [dict(tokens=c.tokens, hidden=c.hidden, group_align=c.group_align, group_quant=c.group_quant,
                   bits=c.bits, outlier_k=c.outlier_k, flags=c.flags) for c in configs]
    ores = [ocal.evaluate(xb, rb, c) for c in odicts]
    target = _target_between([r["nmse"] for r in ores])
    for r in ores:
        r["feasible"] = r["nmse"] <= target
    ochosen = ocal.choose(ores, target)
    chosen, gres = rac.rac_calibrate(to_dev(xb), None if rb is None else to_dev(rb), configs, target)
    for c, g, o in zip(configs, gres, ores):
        assert g["wire_bytes"] == rac.rac_wire_size(c) == o["wire_bytes"]
        assert _close(g["sq_err"], o["sq_err"]) and _close(g["sq_x"], o["sq_x"]) and g["max_abs"] == o["max_abs"]
        assert g["feasible"] == o["feasible"]
    assert chosen == ochosen, (configs[chosen], configs[ochosen])
    say(f"[gpu] calibration {label}: chose {configs[chosen]} ({gres[chosen]['wire_bytes']} B, "
        f"nmse {gres[chosen]['nmse']:.3e}, target {target:.3e})")
    # no target: the cheapest wire of all
    chosen, gres = rac.rac_calibrate(to_dev(xb), None if rb is None else to_dev(rb), configs, math.inf)
    assert chosen == ocal.choose(ores, math.inf)
    return chosen


def test_calibration_on_uplink_rows_in_outlier_mode():
    T, d = 128, 4096
    xb, rb, _ = wl.prefill_uplink(0, rows=(1000, 1000 + T))
    configs = [rac.RacConfig(T, d, ga, gq, b, kg, GRP if kg else 0)
               for ga in (64, 128, 256) for gq in (64, 128, 256) for b in (2, 3, 4, 8) for kg in (0, 1, 2)]
    _run(xb, rb, configs, "uplink 128x4096")


def test_calibration_on_decode_phase_batches():
    B, d = 64, 4096
    xb, rb = wl.decode_step(B)
    configs = [rac.RacConfig(B, d, ga, gq, b) for ga in (128, 256, 512, 4096) for gq in (128, 512, 4096)
               for b in (2, 3, 4, 8)]
    _run(xb, rb, configs, "decode step 64x4096")


def test_calibration_with_bf16_reconstructions_and_zero_reference():
    T, d = 48, 1024
    xb, _, _ = wl.prefill_uplink(3, rows=(0, T), hidden=d)
    configs = [rac.RacConfig(T, d, g, g, b, 2, rac.RAC_FLAG_XHAT_BF16) for g in (64, 128) for b in (3, 4, 8)]
    _run(xb, None, configs, "zero reference, bf16 H-hat")
