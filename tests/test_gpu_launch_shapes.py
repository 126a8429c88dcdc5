"""GPU: the launch hints change how rows are spread over workgroups, never a
byte of the output.  Above 256 rows a launch runs either on the strided grid
(the workgroups the device holds at once, each taking rows in strides with
its next row prefetched) or on one workgroup per row; the default picks by
rows per workgroup.  Each case runs the default, RAC_FLAG_LAUNCH_STRIDED and
RAC_FLAG_LAUNCH_PER_ROW and requires identical wires and reconstructions; the
default is also held to the oracle.  The cases cover the outlier modes, the
bf16 reconstruction and a step table.
"""
from __future__ import annotations

import numpy as np
import pytest

import paper_2608_04991_amd as rac
from paper_2608_04991_amd import workloads as wl
from tests.gpu_util import assert_parity, cfgd, gpu_run, oracle_run, say, to_dev

pytestmark = pytest.mark.gpu
GRP = rac.RAC_FLAG_GROUP_OUTLIERS
HINTS = (0, rac.RAC_FLAG_LAUNCH_STRIDED, rac.RAC_FLAG_LAUNCH_PER_ROW)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rac.library()


def _bytes(a):
    return np.ascontiguousarray(a).view(np.uint8)


CASES = {
    # per-token outliers (the rows kernel and the per-token decode)
    "per_token_3000x1024_g128_b4_k8": (cfgd(3000, 1024, 128, 128, 4, 8), 0),
    # per-group outliers (one wavefront per chunk)
    "per_group_2999x1024_ga64_gq128_b3_kg2": (cfgd(2999, 1024, 64, 128, 3, 2, GRP), 1),
    # no outliers, bf16 reconstruction, a ragged chunk (1536 = 3 chunks)
    "none_bf16_2600x1536_g128_b8": (cfgd(2600, 1536, 128, 128, 8, 0, rac.RAC_FLAG_XHAT_BF16), 2),
    "per_token_1000x4096_g64_b2_k16": (cfgd(1000, 4096, 64, 64, 2, 16), 3),
    # 16 < k <= 48: the two-value threshold variant of the rows kernel
    "per_token_1500x2048_g128_b4_k32": (cfgd(1500, 2048, 128, 128, 4, 32), 5),
    # k > 48: the four-value threshold and the list of 128 candidates
    "per_token_2100x4096_g128_b4_k64": (cfgd(2100, 4096, 128, 128, 4, 64), 6),
    # bf16 reconstruction from the rows kernel (one and two threshold values)
    "per_token_bf16_2000x2048_g128_b4_k8": (cfgd(2000, 2048, 128, 128, 4, 8, rac.RAC_FLAG_XHAT_BF16), 7),
    "per_token_bf16_1100x4096_g128_b3_k32": (cfgd(1100, 4096, 128, 128, 3, 32, rac.RAC_FLAG_XHAT_BF16), 8),
    # a step table (the chunk kernel's per-token and per-group selections;
    # codes clip by design)
    "fixed_step_per_token_1800x2048_g128_b4_k4": (cfgd(1800, 2048, 128, 128, 4, 4, rac.RAC_FLAG_FIXED_STEP), 9),
    "fixed_step_per_group_1500x1024_g64_b4_kg2": (cfgd(1500, 1024, 64, 64, 4, 2, rac.RAC_FLAG_FIXED_STEP | GRP), 10),
}


def _steps(c, seed):
    """A step per quantization group for the step-table cases (None otherwise)."""
    if not c["flags"] & rac.RAC_FLAG_FIXED_STEP:
        return None
    return np.random.default_rng(seed).uniform(0.01, 0.2, c["hidden"] // c["group_quant"]).astype(np.float32)


@pytest.mark.parametrize("name", list(CASES))
def test_launch_shapes_give_identical_bytes(name):
    c, seed = CASES[name]
    T, d = c["tokens"], c["hidden"]
    xb, rb, _ = wl.prefill_uplink(seed, tokens=T, hidden=d)
    steps = _steps(c, seed)
    outs = []
    for hint in HINTS:
        say(f"[gpu] launch shapes {name}: hint {hint}")
        outs.append(gpu_run(dict(c, flags=c["flags"] | hint), xb, rb, steps))
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(_bytes(a), _bytes(b))
    ow, ox = oracle_run(c, xb, rb, steps)
    assert_parity(c, outs[0][0], outs[0][1], ow, ox)


def test_launch_shapes_gathered_and_pooled():
    """The gathered reference (at most 64 rows per workgroup on the strided
    grid) and the pooled fit's encode launch under every hint."""
    import torch
    T, d = 3000, 1024
    c = cfgd(T, d, 128, 128, 4, 4)
    xb, rb, _ = wl.prefill_uplink(4, tokens=T, hidden=d)
    rng = np.random.default_rng(8)
    S = T + 500
    store = wl.f32_to_bf16_bits(rng.standard_normal((S, d)).astype(np.float32))
    pos = rng.permutation(S)[:T]
    store[pos] = rb
    idx = pos.astype(np.int32)
    idx[rng.random(T) < 0.2] = -1
    cuts = np.unique(np.concatenate([[0, T], np.cumsum(rng.integers(1, 300, 20))]))
    seg = cuts[cuts <= T].astype(np.int32)
    x, st, ref = to_dev(xb), to_dev(store), to_dev(rb)
    ix, sg = torch.from_numpy(idx).cuda(), torch.from_numpy(seg).cuda()
    res = []
    for hint in HINTS:
        say(f"[gpu] launch shapes gathered/pooled {T}x{d}: hint {hint}")
        cfg = rac.RacConfig(**dict(c, flags=hint))
        wb = rac.rac_wire_size(cfg)
        w1, w2 = (torch.full((wb,), 0xAB, dtype=torch.uint8, device="cuda") for _ in range(2))
        h1, h2, d1 = (torch.full((T, d), -1.0, dtype=torch.float32, device="cuda") for _ in range(3))
        rac.rac_encode_gather(cfg, x, st, ix, None, w1, h1, store_rows=S)
        rac.rac_decode_gather(cfg, w1, st, ix, None, d1, store_rows=S)
        rac.rac_encode_pooled(cfg, x, ref, sg, None, w2, h2)
        torch.cuda.synchronize()
        res.append([t.cpu().numpy() for t in (w1, h1, d1, w2, h2)])
    for r in res[1:]:
        for a, b in zip(res[0], r):
            assert np.array_equal(_bytes(a), _bytes(b))
    assert np.array_equal(_bytes(res[0][1]), _bytes(res[0][2]))
    gref = np.zeros_like(rb)
    ok = idx >= 0
    gref[ok] = store[idx[ok]]
    ow, ox = oracle_run(c, xb, gref)
    assert_parity(c, res[0][0], res[0][1], ow, ox)


def test_more_rows_than_one_dispatch_holds():
    """17,000,000 rows of 8 channels: one workgroup per row would exceed the
    2^32 work-items of a dispatch for the 256-thread outlier encode, so its
    grid stops at 16,777,215 workgroups and some take a second row.  Sampled
    rows (the ends of the grid and past it) must equal the oracle's, decode
    and reconstruct the sender's on every row, and a gathered call with a
    fifth of its rows missing the same bytes as the materialized call."""
    import torch
    from tests.gpu_util import gpu_run_rows
    T, d = 17_000_000, 8
    c = cfgd(T, d, 8, 8, 4, 2)
    say(f"[gpu] {T}x{d} k2: generating")
    # the tiny recipe's distribution, drawn in bulk: x = a ref + b + noise with
    # (a, b) per row, a fifth of the rows against a zero reference
    rng = np.random.default_rng(11)
    ref = rng.standard_normal((T, d), dtype=np.float32)
    x = (rng.uniform(0.8, 1.2, (T, 1)).astype(np.float32) * ref
         + (0.1 * rng.standard_normal((T, 1))).astype(np.float32)
         + np.float32(0.05) * rng.standard_normal((T, d), dtype=np.float32))
    ref[rng.random(T) < 0.2] = 0.0
    xb, rb = wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(ref)
    del x, ref
    cap = 0xFFFFFFFF // 256
    rows = np.unique(np.concatenate([[0, 1, cap - 1, cap, cap + 1, T - 2, T - 1],
                                     rng.choice(T, 40, replace=False)]))
    say(f"[gpu] {T}x{d} k2: encode, decode, reconstruct")
    gw, gx = gpu_run_rows(c, xb, rb, rows)
    ow, ox = oracle_run(dict(c, tokens=rows.size), xb[rows], rb[rows])
    assert_parity(c, gw, gx, ow, ox, g_rows=rows, o_rows=slice(None), g_xhat_sampled=True)
    # gathered: the store is the reference itself, and a fifth of the rows
    # name no row (their reference is zero in the materialized call)
    miss = rng.random(T) < 0.2
    idx = np.arange(T, dtype=np.int32)
    idx[miss] = -1
    rz = rb.copy()
    rz[miss] = 0
    say(f"[gpu] {T}x{d} k2: gathered against materialized")
    cfg = rac.RacConfig(**c)
    x, st, ix = to_dev(xb), to_dev(rb), torch.from_numpy(idx).cuda()
    wg = torch.empty(rac.rac_wire_size(cfg), dtype=torch.uint8, device="cuda")
    rac.rac_encode_gather(cfg, x, st, ix, None, wg, None, store_rows=T)
    torch.cuda.synchronize()
    del st
    wm = torch.empty_like(wg)
    rac.rac_encode(cfg, x, to_dev(rz), None, wm, None)
    torch.cuda.synchronize()
    assert torch.equal(wg, wm)
    del x, ix, wg, wm
    torch.cuda.empty_cache()
