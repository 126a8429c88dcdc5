"""GPU parity of rac_encode_pooled (the affine fit pooled over segments of
rows) against the oracle's pooled encode, through the C ABI; the wire decodes
with the unchanged rac_decode to the sender's reconstruction.  Segment lengths
cover one row, partial and full 64-row blocks and a segment deep enough for
the block stack; the full 4096 x 4096 shape is compared on every row."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2608_04991_amd as rac
from paper_2608_04991_amd import workloads as wl
from tests.gpu_util import assert_parity, cfgd, gpu_run, say, to_dev

pytestmark = pytest.mark.gpu
GRP = rac.RAC_FLAG_GROUP_OUTLIERS


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rac.library()


def _gpu_pooled(c, xb, rb, seg):
    import torch
    cfg = rac.RacConfig(**c)
    T, d = c["tokens"], c["hidden"]
    seg = np.asarray(seg, np.int32)
    assert xb.shape == (T, d) and seg[0] == 0 and seg[-1] == T and np.all(np.diff(seg) > 0)
    x = to_dev(xb)
    ref = to_dev(rb) if rb is not None else None
    st = torch.from_numpy(seg).cuda()
    wire = torch.full((rac.rac_wire_size(cfg),), 0xAB, dtype=torch.uint8, device="cuda")
    bf16 = bool(c["flags"] & rac.RAC_FLAG_XHAT_BF16)
    dt = torch.int16 if bf16 else torch.float32
    xh = torch.full((T, d), -1, dtype=dt, device="cuda")
    xd = torch.full((T, d), -1, dtype=dt, device="cuda")
    rac.rac_encode_pooled(cfg, x, ref, st, None, wire, xh)
    rac.rac_decode(cfg, wire, ref, None, xd)
    torch.cuda.synchronize()
    view = (lambda a: a.view(np.uint16)) if bf16 else (lambda a: a)
    return wire.cpu().numpy(), view(xh.cpu().numpy()), view(xd.cpu().numpy())


def _oracle_pooled(c, xb, rb, seg):
    rc, w, xh = oracle.encode_pooled(xb, rb, np.asarray(seg, np.int32), **c)
    assert rc == 0, rc
    return w, xh


CASES = {
    "uplink_37x4096_g128_b4_k8": (cfgd(37, 4096, 128, 128, 4, 8), [0, 5, 6, 37],
                                  lambda: wl.prefill_uplink(0, rows=(0, 37))[:2]),
    "blocks_300x512_g128_b2": (cfgd(300, 512, 128, 128, 2), [0, 1, 64, 128, 193, 300],
                               lambda: wl.prefill_uplink(1, rows=(0, 300), hidden=512)[:2]),
    "one_segment_200x1024_ga64_gq128_b4": (cfgd(200, 1024, 64, 128, 4), [0, 200],
                                           lambda: wl.prefill_uplink(2, rows=(0, 200), hidden=1024)[:2]),
    "deep_stack_4100x512_g64_b8": (cfgd(4100, 512, 64, 64, 8), [0, 4100],
                                   lambda: wl.long_context(0, rows=(0, 4100), group=64, hidden=512)[:2]),
    "group_outliers_50x4096_g128_b4_kg2": (cfgd(50, 4096, 128, 128, 4, 2, GRP), [0, 17, 18, 50],
                                           lambda: wl.prefill_uplink(3, rows=(0, 50))[:2]),
    "zero_reference_40x2048_g128_b4_k4": (cfgd(40, 2048, 128, 128, 4, 4), [0, 20, 40],
                                          lambda: (wl.prefill_uplink(4, rows=(0, 40), hidden=2048)[0], None)),
    "bf16_out_66x4096_g128_b4_k8": (cfgd(66, 4096, 128, 128, 4, 8, rac.RAC_FLAG_XHAT_BF16), [0, 64, 65, 66],
                                    lambda: wl.prefill_uplink(5, rows=(0, 66))[:2]),
    "ragged_chunk_23x2880_ga64_gq32_b4": (cfgd(23, 2880, 64, 32, 4), [0, 7, 23],
                                          lambda: wl.affine_pair(wl.AffineRecipe(23, 2880, 64), 0)[:2]),
    # the outlier encode finds each row's segment 64 starts at a time: about
    # 100 segments take two levels of that search, 4100 one-row segments three
    "many_segments_300x1024_g128_b4_k4": (cfgd(300, 1024, 128, 128, 4, 4),
                                          np.unique(np.concatenate([[0, 300], np.cumsum(
                                              np.random.default_rng(21).integers(1, 6, 120))]))[:None],
                                          lambda: wl.prefill_uplink(7, rows=(0, 300), hidden=1024)[:2]),
    "one_row_segments_4100x512_g64_b4_k2": (cfgd(4100, 512, 64, 64, 4, 2), np.arange(4101),
                                            lambda: wl.long_context(1, rows=(0, 4100), group=64, hidden=512)[:2]),
}
_c, _s, _g = CASES["many_segments_300x1024_g128_b4_k4"]
CASES["many_segments_300x1024_g128_b4_k4"] = (_c, _s[_s <= 300], _g)


@pytest.mark.parametrize("name", list(CASES))
def test_pooled_parity(name):
    c, seg, gen = CASES[name]
    xb, rb = gen()
    say(f"[gpu] pooled {name}: segments {np.diff(seg).tolist()[:8]}")
    ow, ox = _oracle_pooled(c, xb, rb, seg)
    gw, gx, gd = _gpu_pooled(c, xb, rb, seg)
    assert_parity(c, gw, gx, ow, ox)
    assert np.array_equal(gx.view(np.uint8), gd.view(np.uint8))


def test_one_row_segments_equal_the_per_token_encode():
    c = cfgd(29, 4096, 128, 128, 4, 8)
    xb, rb, _ = wl.prefill_uplink(6, rows=(0, 29))
    say("[gpu] pooled with one-row segments vs the per-token encode")
    gw, gx, _ = _gpu_pooled(c, xb, rb, np.arange(30))
    tw, tx, _, _ = gpu_run(c, xb, rb)
    assert gw[6] == tw[6] | 16
    gw = gw.copy()
    gw[6] = tw[6]
    assert np.array_equal(gw, tw) and np.array_equal(gx.view(np.uint32), tx.view(np.uint32))


def test_more_segment_groups_than_one_dispatch_holds():
    """4,300,000 one-row segments of 32 channels (one alignment group each):
    more (segment, group) pairs than merge workgroups one dispatch holds
    (2^32 work-items over 1024 per workgroup), so some workgroups merge a
    second pair.  One-row segments must still give the per-token encode's
    bytes (header flag aside) and reconstruction."""
    T, d = 4_300_000, 32
    c = cfgd(T, d, 32, 32, 4, 2)
    say(f"[gpu] pooled, {T} one-row segments of {d} channels: generating")
    rng = np.random.default_rng(21)
    ref = rng.standard_normal((T, d), dtype=np.float32)
    x = (rng.uniform(0.8, 1.2, (T, 1)).astype(np.float32) * ref
         + (0.1 * rng.standard_normal((T, 1))).astype(np.float32)
         + np.float32(0.05) * rng.standard_normal((T, d), dtype=np.float32))
    xb, rb = wl.f32_to_bf16_bits(x), wl.f32_to_bf16_bits(ref)
    del x, ref
    assert T > 0xFFFFFFFF // 1024
    say(f"[gpu] pooled, {T} one-row segments: encode and decode")
    gw, gx, gd = _gpu_pooled(c, xb, rb, np.arange(T + 1))
    assert np.array_equal(gx.view(np.uint32), gd.view(np.uint32))
    tw, tx, _, _ = gpu_run(c, xb, rb)
    assert gw[6] == tw[6] | 16
    gw = gw.copy()
    gw[6] = tw[6]
    assert np.array_equal(gw, tw) and np.array_equal(gx.view(np.uint32), tx.view(np.uint32))


def test_full_prefill_uplink_4096x4096_pooled_over_spans():
    """The benchmark shape with segments standing for retrieved spans (random
    lengths between 1 and 600 rows), every row compared with the oracle."""
    import torch
    c = cfgd(4096, 4096, 128, 128, 4, 8)
    rng = np.random.default_rng(12)
    cuts = np.unique(np.concatenate([[0, 4096], np.cumsum(rng.integers(1, 600, 40))]))
    seg = cuts[cuts <= 4096]
    say(f"[gpu] full 4096x4096 pooled over {seg.size - 1} segments: generating")
    xb, rb, _ = wl.prefill_uplink(0)
    gw, gx, gd = _gpu_pooled(c, xb, rb, seg)
    assert np.array_equal(gx, gd)
    ow, ox = _oracle_pooled(c, xb, rb, seg)
    assert_parity(c, gw, gx, ow, ox)
    torch.cuda.empty_cache()


def test_pooled_with_fixed_steps_and_group_outliers():
    import torch
    c = cfgd(64, 512, 64, 64, 4, 2, rac.RAC_FLAG_FIXED_STEP | GRP)
    xb, rb, _ = wl.tiny(0)
    steps = np.linspace(0.02, 0.2, 512 // 64).astype(np.float32)
    seg = np.array([0, 10, 11, 40, 64], np.int32)
    say("[gpu] pooled with a calibrated step table and per-group outliers")
    rc, ow, ox = oracle.encode_pooled(xb, rb, seg, steps, **c)
    assert rc == 0
    cfg = rac.RacConfig(**c)
    x, ref = to_dev(xb), to_dev(rb)
    st = torch.from_numpy(steps).cuda()
    wire = torch.full((rac.rac_wire_size(cfg),), 0xAB, dtype=torch.uint8, device="cuda")
    xh = torch.full((64, 512), -1.0, dtype=torch.float32, device="cuda")
    xd = torch.full((64, 512), -1.0, dtype=torch.float32, device="cuda")
    rac.rac_encode_pooled(cfg, x, ref, torch.from_numpy(seg).cuda(), st, wire, xh)
    rac.rac_decode(cfg, wire, ref, st, xd)
    torch.cuda.synchronize()
    assert_parity(c, wire.cpu().numpy(), xh.cpu().numpy(), ow, ox)
    assert torch.equal(xh, xd)
