"""GPU parity of the saturation marks: rows built so that exactly one kind
of fp16 overflow happens in known rows (an alignment coefficient, a scale, an
outlier value), through every encode kernel path (the per-token outlier
kernel, the one-wavefront-per-chunk kernel with and without outliers,
per-group outliers, groups wider than a chunk, the fixed step table, the
pooled fit).  The marked fields hold +-infinity; the whole wire must be
bit-identical to the oracle's, the reconstruction finite and equal to the
decode's, and the marked rows the expected ones.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2608_04991_amd as rac
from paper_2608_04991_amd import workloads as wl
from tests import wirefmt
from tests.gpu_util import assert_parity, cfgd, gpu_run, oracle_run, say, to_dev

pytestmark = pytest.mark.gpu
GRP = rac.RAC_FLAG_GROUP_OUTLIERS
BF16 = lambda a: wl.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rac.library()


def _base(T, d, seed):
    """Ordinary rows (no overflow anywhere) to put the planted blocks in."""
    return wl.affine_pair(wl.AffineRecipe(T, d, 64), seed)[0].astype(np.uint16)


def _scale_rows(T, d):
    # zero reference: a +-2^20 group has beta = 0 and |E| = 2^20 > 65504 * 7
    x = wl.bf16_bits_to_f32(_base(T, d, 1)).copy()
    x[0, 0:128] = np.tile([2.0 ** 20, -2.0 ** 20], 64)
    x[T - 1, d - 128:d] = np.tile([2.0 ** 20, -2.0 ** 20], 64)
    return BF16(x), None


def _beta_rows(T, d):
    # group means 65516 (rounds to 65504) and 65520 (overflows)
    x = wl.bf16_bits_to_f32(_base(T, d, 2)).copy()
    for row, c0, j in ((0, 0, 59), (0, 512, 60), (T - 1, d - 64, 60)):
        v = np.full(64, 65280.0, np.float32)
        v[:j] = 65536.0
        x[row, c0:c0 + 64] = v
    return BF16(x), None


def _beta_wide_rows(T, d):
    # row 2, channels 1024-2047 (chunks 2 and 3): mean 65536
    x = wl.bf16_bits_to_f32(_base(T, d, 6)).copy()
    x[2, 1024:2048] = 65536.0
    return BF16(x), None


def _alpha_rows(T, d):
    rng = np.random.default_rng(3)
    r = rng.standard_normal((T, d)).astype(np.float32)
    x = r * 0.5 + rng.standard_normal((T, d)).astype(np.float32) * 0.01
    r[1, 512:640] = np.tile([2.0 ** -10, -2.0 ** -10], 64)
    x[1, 512:640] = np.tile([1024.0, -1024.0], 64)
    return BF16(x), BF16(r)


def _outlier_rows(T, d):
    x = np.zeros((T, d), np.float32)
    x[:] = wl.bf16_bits_to_f32(_base(T, d, 4))
    x[0, 600], x[0, 601] = 131072.0, -131072.0
    x[T - 1, 5], x[T - 1, 6] = -131072.0, 131072.0
    return BF16(x), None


CASES = {
    # bit 2, the per-token outlier kernel (k > 0: two of the +-2^20 values
    # become outliers, which overflow as well) and the chunk kernel (k = 0)
    "scale_rows_kernel_5x1024_b4_k2": (cfgd(5, 1024, 128, 128, 4, 2), _scale_rows, [(0, 0, 6), (4, 1, 6)]),
    "scale_chunk_kernel_5x1024_b4_k0": (cfgd(5, 1024, 128, 128, 4, 0), _scale_rows, [(0, 0, 2), (4, 1, 2)]),
    "scale_8bit_covers_5x1024_b8": (cfgd(5, 1024, 128, 128, 8, 0), _scale_rows, []),
    # a quantization group of 1024 channels (two chunks) is reported in its first chunk
    "scale_wide_group_5x2048_gq1024_b4": (cfgd(5, 2048, 128, 1024, 4, 0), _scale_rows, [(0, 0, 2), (4, 2, 2)]),
    # bit 1 from beta (the 65520 threshold), both kernels and per-group outliers
    "beta_rows_kernel_5x1024_g64_k1": (cfgd(5, 1024, 64, 64, 4, 1), _beta_rows, [(0, 1, 1), (4, 1, 1)]),
    "beta_chunk_kernel_5x1024_g64_k0": (cfgd(5, 1024, 64, 64, 4, 0), _beta_rows, [(0, 1, 1), (4, 1, 1)]),
    "beta_group_outliers_5x1024_g64_kg1": (cfgd(5, 1024, 64, 64, 4, 1, GRP), _beta_rows, [(0, 1, 1), (4, 1, 1)]),
    # an alignment group of 1024 channels: reported in the group's first chunk
    "beta_wide_align_5x2048_ga1024_b4": (cfgd(5, 2048, 1024, 128, 4, 0), _beta_wide_rows, [(2, 2, 1)]),
    # bit 1 from alpha
    "alpha_rows_kernel_3x1024_k4": (cfgd(3, 1024, 128, 128, 4, 4), _alpha_rows, [(1, 1, 1)]),
    "alpha_chunk_kernel_3x1024_k0": (cfgd(3, 1024, 128, 128, 4, 0), _alpha_rows, [(1, 1, 1)]),
    # bit 4: per-token outliers (rows kernel), per-group outliers, and the
    # fixed step table (the chunk kernel's per-token selection)
    "outlier_rows_kernel_4x1024_b8_k3": (cfgd(4, 1024, 128, 128, 8, 3), _outlier_rows, [(0, 1, 4), (3, 0, 4)]),
    "outlier_group_mode_4x1024_b8_kg1": (cfgd(4, 1024, 128, 128, 8, 1, GRP), _outlier_rows, [(0, 1, 4), (3, 0, 4)]),
}


@pytest.mark.parametrize("name", list(CASES))
def test_saturation_report_parity(name):
    c, gen, expect = CASES[name]
    xb, rb = gen(c["tokens"], c["hidden"])
    say(f"[gpu] saturation {name}")
    ow, ox = oracle_run(c, xb, rb)
    gw, gx, gd, gr = gpu_run(c, xb, rb)
    assert_parity(c, gw, gx, ow, ox)
    assert np.array_equal(gx.view(np.uint8), gd.view(np.uint8))
    assert np.isfinite(gx).all()
    marks = wirefmt.saturation_marks(gw)
    want = np.zeros_like(marks)
    for row, _, bit in expect:
        want[row] |= bit
    assert np.array_equal(marks, want), f"marks {marks.tolist()} != {want.tolist()}"
    rows, bits = rac.rac_saturation_summary(rac.RacConfig(**c), gw)
    assert rows == int((marks != 0).sum()) and bits == int(np.bitwise_or.reduce(marks))


def test_saturation_with_fixed_steps_and_outliers():
    """The fixed step table takes the chunk kernel's per-token selection:
    outlier overflow is reported, scale saturation never (codes clip by
    design with a step table)."""
    T, d = 4, 1024
    c = cfgd(T, d, 128, 128, 4, 2, rac.RAC_FLAG_FIXED_STEP)
    xb, rb = _outlier_rows(T, d)
    steps = np.full(d // 128, 0.01, np.float32)
    ow, ox = oracle_run(c, xb, rb, steps)
    gw, gx, gd, _ = gpu_run(c, xb, rb, steps)
    assert_parity(c, gw, gx, ow, ox)
    assert wirefmt.saturation_marks(gw).tolist() == [4, 0, 0, 4]


def test_pooled_fit_reports_every_row_of_a_saturated_segment():
    import torch
    T, d = 9, 1024
    x = np.full((T, d), 1.0, np.float32)
    x[:, 0:64] = 65536.0          # rows 0-5 below: pooled beta* = 65536 in group 0
    x[6:, 0:64] = 65280.0         # rows 6-8: no overflow
    xb = BF16(x + np.random.default_rng(5).standard_normal((T, d)).astype(np.float32) * (x < 2))
    seg = np.array([0, 6, 9], np.int32)
    c = cfgd(T, d, 64, 64, 4, 2)
    rc, ow, ox = oracle.encode_pooled(xb, None, seg, **c)
    assert rc == 0
    cfg = rac.RacConfig(**c)
    wire = torch.full((rac.rac_wire_size(cfg),), 0xCD, dtype=torch.uint8, device="cuda")
    xh = torch.empty(T, d, dtype=torch.float32, device="cuda")
    rac.rac_encode_pooled(cfg, to_dev(xb), None, torch.from_numpy(seg).cuda(), None, wire, xh)
    torch.cuda.synchronize()
    gw = wire.cpu().numpy()
    assert np.array_equal(gw, ow)
    assert np.array_equal(xh.cpu().numpy().view(np.uint32), ox.view(np.uint32))
    assert wirefmt.saturation_marks(gw).tolist() == [1] * 6 + [0] * 3
