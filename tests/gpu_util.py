"""Shared helpers of the GPU parity tests: run the HIP codec through the C ABI
and compare its wire and reconstruction with the CPU oracle's."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import paper_2608_04991_amd as rac
from tests import wirefmt

QMAX = {2: 1, 3: 3, 4: 7, 8: 127}


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def cfgd(T, d, ga, gq, b, k=0, flags=0):
    return dict(tokens=T, hidden=d, group_align=ga, group_quant=gq, bits=b, outlier_k=k,
                flags=flags)


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).cuda()


def check_shapes(c, xb, rb, steps):
    """Host-side check, before any launch, that buffers match the config."""
    T, d = c["tokens"], c["hidden"]
    assert xb.shape == (T, d) and xb.dtype == np.uint16
    assert rb is None or (rb.shape == (T, d) and rb.dtype == np.uint16)
    if c["flags"] & rac.RAC_FLAG_FIXED_STEP:
        assert steps is not None and steps.shape == (d // c["group_quant"],)


def gpu_run(c, xb, rb, steps=None, *, stream=None, want_xhat=True, garbage=0xAB):
    """Encode (fused reconstruction), then decode and reconstruct from the
    wire.  Returns numpy (wire, xhat_sender, xhat_decode, xhat_reconstruct)."""
    import torch
    check_shapes(c, xb, rb, steps)
    cfg = rac.RacConfig(**c)
    T, d = c["tokens"], c["hidden"]
    size = rac.rac_wire_size(cfg)
    x = to_dev(xb)
    ref = to_dev(rb) if rb is not None else None
    st = torch.from_numpy(np.asarray(steps, np.float32)).cuda() if steps is not None else None
    wire = torch.full((size,), garbage, dtype=torch.uint8, device="cuda")
    bf16 = bool(c["flags"] & rac.RAC_FLAG_XHAT_BF16)
    dt = torch.int16 if bf16 else torch.float32
    outs = [torch.full((T, d), -1, dtype=dt, device="cuda") for _ in range(3)]
    rac.rac_encode(cfg, x, ref, st, wire, outs[0] if want_xhat else None, stream=stream)
    rac.rac_decode(cfg, wire, ref, st, outs[1], stream=stream)
    rac.rac_reconstruct(cfg, wire, ref, st, outs[2], stream=stream)
    torch.cuda.synchronize()
    res = [wire.cpu().numpy()]
    for o in outs:
        a = o.cpu().numpy()
        res.append(a.view(np.uint16) if bf16 else a)
    return tuple(res)


def oracle_run(c, xb, rb, steps=None):
    rc, wire, xhat = oracle.encode(xb, rb, steps, **c)
    assert rc == 0, rc
    return wire, xhat


def row_sections(wire: np.ndarray, rows) -> dict:
    s = wirefmt.sections(wire)
    out = {}
    for k in ("coef", "scale", "codes", "outl", "gval", "goff"):
        out[k] = None if s[k] is None else s[k][rows]
    return out


def assert_parity(c, g_wire, g_xhat, o_wire, o_xhat, g_rows=None, o_rows=None, strict=True,
                  g_xhat_sampled=False):
    """Compare GPU and oracle outputs.

    The bar (per element): header, coefficients, scales, outlier channels and
    values identical; codes equal except at most +-1 on at most 0.01% of
    elements (rounding ties); reconstruction within 1e-5 relative / 1e-6
    absolute where codes agree and off by exactly one step where they do not.
    With strict=True the wire and reconstruction must also be bit-identical,
    which is what the fixed evaluation order guarantees.  g_xhat_sampled: the
    GPU reconstruction holds only the rows g_rows, in that order.
    """
    T, d, b, gq = c["tokens"], c["hidden"], c["bits"], c["group_quant"]
    if g_rows is None:
        assert np.array_equal(g_wire[:256], o_wire[:256]), "header differs"
        assert wirefmt.padding_is_zero(g_wire), "padding not zero"
        gs, os_ = row_sections(g_wire, slice(None)), row_sections(o_wire, slice(None))
        gx, ox = g_xhat, o_xhat
    else:
        gs, os_ = row_sections(g_wire, g_rows), row_sections(o_wire, o_rows)
        gx = g_xhat if g_xhat_sampled else g_xhat[g_rows]
        ox = o_xhat[o_rows]
    n = gs["codes"].shape[0]
    assert np.array_equal(gs["coef"], os_["coef"]), \
        f"coef differ at {np.argwhere(gs['coef'] != os_['coef'])[:5].tolist()}"
    if os_["scale"] is not None:
        assert np.array_equal(gs["scale"], os_["scale"]), \
            f"scales differ at {np.argwhere(gs['scale'] != os_['scale'])[:5].tolist()}"
    assert (gs["outl"] is None) == (os_["outl"] is None) and (gs["gval"] is None) == (os_["gval"] is None)
    if os_["outl"] is not None:
        assert np.array_equal(gs["outl"], os_["outl"]), "outliers differ"
    if os_["gval"] is not None:
        assert np.array_equal(gs["goff"], os_["goff"]), \
            f"group outlier offsets differ at {np.argwhere(gs['goff'] != os_['goff'])[:5].tolist()}"
        assert np.array_equal(gs["gval"], os_["gval"]), \
            f"group outlier values differ at {np.argwhere(gs['gval'] != os_['gval'])[:5].tolist()}"
    gc = wirefmt.unpack_codes(gs["codes"], d, b)
    oc = wirefmt.unpack_codes(os_["codes"], d, b)
    diff = gc != oc
    assert np.abs(gc - oc).max(initial=0) <= 1
    assert diff.sum() <= 1e-4 * gc.size, f"{diff.sum()} code mismatches"
    if gx is not None and gx.dtype == np.float32:
        same = ~diff
        tol = 1e-5 * np.abs(ox) + 1e-6
        bad = same & ~(np.abs(gx - ox) <= tol)
        assert not bad.any(), f"xhat mismatch at {np.argwhere(bad)[:5].tolist()}"
    if strict:
        assert np.array_equal(gs["codes"], os_["codes"]), f"codes differ at {np.argwhere(diff)[:5].tolist()}"
        if gx is not None:
            assert np.array_equal(gx.view(np.uint8), ox.view(np.uint8)), \
                f"xhat not bitwise at {np.argwhere(gx.view(np.uint32 if gx.dtype == np.float32 else np.uint16) != ox.view(np.uint32 if ox.dtype == np.float32 else np.uint16))[:5].tolist()}"
    return n


def gpu_run_rows(c, xb, rb, rows, steps=None):
    """Full-size encode (fused reconstruction), decode and reconstruct on the
    GPU; asserts on the device that the three reconstructions are bitwise
    equal, then returns the whole wire and only the given rows of the
    sender's reconstruction (numpy), so shapes of several GB stay on the
    device."""
    import torch
    check_shapes(c, xb, rb, steps)
    cfg = rac.RacConfig(**c)
    T, d = c["tokens"], c["hidden"]
    x = to_dev(xb)
    ref = to_dev(rb) if rb is not None else None
    st = torch.from_numpy(np.asarray(steps, np.float32)).cuda() if steps is not None else None
    wire = torch.full((rac.rac_wire_size(cfg),), 0xAB, dtype=torch.uint8, device="cuda")
    bf16 = bool(c["flags"] & rac.RAC_FLAG_XHAT_BF16)
    dt = torch.int16 if bf16 else torch.float32
    xh = torch.full((T, d), -1, dtype=dt, device="cuda")
    rac.rac_encode(cfg, x, ref, st, wire, xh)
    del x
    xo = torch.full((T, d), -1, dtype=dt, device="cuda")
    rac.rac_decode(cfg, wire, ref, st, xo)
    torch.cuda.synchronize()
    assert torch.equal(xh, xo), "receiver decode differs from the sender reconstruction"
    xo.fill_(-1)
    rac.rac_reconstruct(cfg, wire, ref, st, xo)
    torch.cuda.synchronize()
    assert torch.equal(xh, xo), "rac_reconstruct differs from the sender reconstruction"
    del xo
    sel = xh.index_select(0, torch.from_numpy(np.asarray(rows, np.int64)).cuda()).cpu().numpy()
    out = wire.cpu().numpy()
    del xh, wire, ref
    torch.cuda.empty_cache()
    return out, (sel.view(np.uint16) if bf16 else sel)
