"""Pins of the predictor oracle (oracle/predictor.py) against what does not
come from it: torch's float64 library routines for each layer (rms_norm,
scaled-dot-product attention, silu), an independent torch forward over
several steps, and structural facts of the definition (a zero output
projection returns the input exactly, a one-input window attends only the
current input, inputs older than the window do not matter, and the rotary
pairing of channels, whose scores depend on relative positions only).
Planted mistakes in a copy of the oracle's source must fail a pin."""
from __future__ import annotations

import sys
import types

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import predictor as P
from paper_2608_04991_amd import workloads as wl

D, M, H, FF = 512, 128, 2, 256


def _pred(window=4, batch=3, seed=0):
    return P.Predictor(wl.predictor_weights(D, M, FF, seed), D, M, H, FF, window, batch)


def _seq(batch, steps, seed=0):
    return wl.decode_sequence(batch, steps, seed, hidden=D)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(1)
    h, g = rng.standard_normal((5, M)) * 3, 1 + 0.1 * rng.standard_normal(M)
    want = F.rms_norm(torch.from_numpy(h), (M,), weight=torch.from_numpy(g), eps=P.EPS).numpy()
    np.testing.assert_allclose(P.rmsnorm(h, g), want, rtol=1e-13, atol=0)


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(2)
    for n in (1, 2, 7, 64):
        q, k, v = rng.standard_normal(64), rng.standard_normal((n, 64)), rng.standard_normal((n, 64))
        want = F.scaled_dot_product_attention(torch.from_numpy(q)[None, None, None], torch.from_numpy(k)[None, None],
                                              torch.from_numpy(v)[None, None]).numpy().ravel()
        np.testing.assert_allclose(P.attend(q, k, v), want, rtol=1e-12, atol=1e-14)


def test_silu_matches_torch():
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(P.silu(z), F.silu(torch.from_numpy(z)).numpy(), rtol=1e-13, atol=1e-300)


def test_rotary_turns_channel_pairs_and_scores_depend_on_relative_position():
    # channel 2i, 2i+1 of a head turned by pos * 10000^(-2i/64)
    for i, p in ((0, 5), (1, 3), (31, 1000)):
        e = np.zeros((1, 128))
        e[0, 64 + 2 * i] = 1.0                     # head 1
        r = P.rope(e, np.array([p]))[0]
        ang = p * 10000.0 ** (-2.0 * i / 64)
        assert abs(r[64 + 2 * i] - np.cos(ang)) < 1e-12 and abs(r[65 + 2 * i] - np.sin(ang)) < 1e-12
        assert np.count_nonzero(np.abs(r) > 1e-15) <= 2
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal((1, 64)), rng.standard_normal((1, 64))
    s = lambda a, b: float(P.rope(q, np.array([a]))[0] @ P.rope(k, np.array([b]))[0])
    assert abs(s(9, 4) - s(109, 104)) < 1e-12 and abs(s(9, 4) - s(5, 0)) < 1e-12


def _torch_forward(W, xs, window):
    """An independent forward with torch's float64 ops (linear, rms_norm,
    scaled-dot-product attention with a window mask, silu) and bf16 casts at
    the same storage points; xs bf16 [steps][B][D]; returns R [steps][B][D]
    as float64 values."""
    t = {k: torch.from_numpy(v.astype(np.float64)) for k, v in W.items()}
    bfr = lambda a: a.to(torch.bfloat16).to(torch.float64)
    theta = 10000.0 ** (-2.0 * torch.arange(32, dtype=torch.float64) / 64)
    steps, B, _ = xs.shape
    ks, vs, out = [[] for _ in range(B)], [[] for _ in range(B)], []
    for step in range(steps):
        x = torch.from_numpy(P.bf16_to_f64(xs[step]))
        h0 = F.linear(x, t["w_in"])
        n1 = bfr(F.rms_norm(h0, (M,), weight=t["g1"], eps=P.EPS))
        q, k, v = F.linear(n1, t["w_qkv"]).split(M, dim=1)

        def rot(a):
            c, s = torch.cos(step * theta), torch.sin(step * theta)
            pr = a.reshape(B, H, 32, 2)
            return torch.stack([pr[..., 0] * c - pr[..., 1] * s, pr[..., 0] * s + pr[..., 1] * c], -1).reshape(B, M)
        q, k = rot(q), bfr(rot(k))
        v = bfr(v)
        o = torch.zeros(B, M, dtype=torch.float64)
        for b in range(B):
            ks[b].append(k[b])
            vs[b].append(v[b])
            kk = torch.stack(ks[b][-window:]).reshape(-1, H, 64).transpose(0, 1)
            vv = torch.stack(vs[b][-window:]).reshape(-1, H, 64).transpose(0, 1)
            o[b] = F.scaled_dot_product_attention(q[b].reshape(H, 1, 64), kk, vv).reshape(M)
        h1 = h0 + F.linear(bfr(o), t["w_o"])
        n2 = bfr(F.rms_norm(h1, (M,), weight=t["g2"], eps=P.EPS))
        gu = F.linear(n2, t["w_gu"])
        h2 = h1 + F.linear(bfr(F.silu(gu[:, 0::2]) * gu[:, 1::2]), t["w_down"])
        n3 = bfr(F.rms_norm(h2, (M,), weight=t["g3"], eps=P.EPS))
        out.append((x + F.linear(n3, t["w_out"])).numpy())
    return np.stack(out)


def test_steps_match_an_independent_torch_forward():
    window, B, steps = 3, 2, 6
    pr = _pred(window, B)
    xs = _seq(B, steps)
    want = _torch_forward({k: P.bf16_to_f64(v) for k, v in wl.predictor_weights(D, M, FF, 0).items()}, xs, window)
    for s in range(steps):
        _, inter = pr.step(xs[s], np.full(B, s))
        # torch casts float64 to bf16 through float32; a rare double rounding
        # moves one bf16 activation by an ulp, so the bar is relative 1e-6
        np.testing.assert_allclose(inter["r"], want[s], rtol=1e-6, atol=1e-6 * np.abs(want[s]).max())


def test_zero_output_projection_returns_the_input_exactly():
    w = wl.predictor_weights(D, M, FF, 0)
    w["w_out"] = np.zeros_like(w["w_out"])
    pr = P.Predictor(w, D, M, H, FF, 4, 2)
    xs = _seq(2, 2)
    for s in range(2):
        r, _ = pr.step(xs[s], [s, s])
        assert np.array_equal(r, xs[s])


def test_a_window_of_one_attends_only_the_current_input():
    pr = _pred(window=1, batch=2)
    xs = _seq(2, 3)
    for s in range(3):
        _, inter = pr.step(xs[s], [s, s])
        np.testing.assert_array_equal(inter["o"], P.to_bf16(inter["v"]))


def test_inputs_older_than_the_window_do_not_matter():
    window, steps = 3, 6
    a, b = _pred(window, 1), _pred(window, 1)
    xa, xb = _seq(1, steps, seed=1), _seq(1, steps, seed=1).copy()
    xb[:steps - window] = _seq(1, steps - window, seed=9)     # different old history
    for s in range(steps):
        ra, _ = a.step(xa[s], [s])
        rb, _ = b.step(xb[s], [s])
    assert np.array_equal(ra, rb)


PLANTED = [
    ("score_scale_1_over_64", "s = keys @ q / np.sqrt(HEAD)", "s = keys @ q / HEAD"),
    ("window_one_too_long", "span = range(max(0, p - win + 1), p + 1)", "span = range(max(0, p - win), p + 1)"),
    ("residual_dropped", "h1 = h0 + o @ W[\"w_o\"].T", "h1 = o @ W[\"w_o\"].T"),
    ("rotary_sign", "out = np.stack([a * c - b * s, a * s + b * c], axis=-1)",
     "out = np.stack([a * c + b * s, a * s + b * c], axis=-1)"),
    ("gate_and_up_swapped", "g = to_bf16(silu(gu[:, 0::2]) * gu[:, 1::2])", "g = to_bf16(silu(gu[:, 1::2]) * gu[:, 0::2])"),
    ("norm_without_gain", "return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + EPS) * gain",
     "return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + EPS)"),
]


@pytest.mark.parametrize("name,old,new", PLANTED, ids=[p[0] for p in PLANTED])
def test_planted_predictor_mistake_fails_a_pin(monkeypatch, name, old, new):
    src = open(P.__file__).read()
    assert src.count(old) == 1, name
    mod = types.ModuleType("mutant_predictor")
    exec(compile(src.replace(old, new), "mutant_predictor", "exec"), mod.__dict__)
    monkeypatch.setattr(sys.modules[__name__], "P", mod)
    caught = 0
    for pin in (test_rmsnorm_matches_torch, test_attention_matches_torch_sdpa,
                test_rotary_turns_channel_pairs_and_scores_depend_on_relative_position,
                test_steps_match_an_independent_torch_forward, test_inputs_older_than_the_window_do_not_matter):
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught, f"no pin caught {name}"
