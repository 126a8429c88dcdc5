"""Seeded synthetic boundary activations for the RAC codec.

This module only draws inputs: it holds none of the codec's arithmetic, so both
the HIP library's tests and the CPU oracle can consume the same arrays.  The
paper measures on model activations of WikiText-2 / HellaSwag / GSM8K /
MATH-500 / ShareGPT prompts (Evaluation, "Datasets"); none of those are used.
Seeded stand-ins with the shapes of the evaluated models' boundary states and
the value structure the codec cares about (per-channel scale spread, affine
relation to a reference, outlier channels, rows without a reference) take
their place.

Arrays are numpy; bf16 tensors are uint16 bit patterns (round-to-nearest-even
from float32).  Rows are drawn in blocks of ``BLOCK`` rows, each block from its
own generator seeded with ``[seed, tag, block]``, so any row subset can be
regenerated without drawing the whole tensor.  Per-channel quantities (the
channel scale spread, outlier channels, which rows lack a reference) come from
one generator seeded with ``[seed, tag]``.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

BLOCK = 256


def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((u + (((u >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class AffineRecipe:
    """x = a * ref + b + noise per (token, group), ref = N(0,1) * s_c."""
    tokens: int
    hidden: int
    group: int
    a_lo: float = 0.8
    a_hi: float = 1.2
    b_sigma: float = 0.1
    noise: str = "normal"        # "normal" or "student_t3"
    noise_scale: float = 0.05
    outlier_frac: float = 0.0    # fraction of channels scaled in x only
    outlier_scale: float = 20.0
    zero_ref_frac: float = 0.0   # fraction of rows whose reference is zero
    tag: int = 0                 # separates recipes that share a seed


def _rows(tokens: int, rows) -> np.ndarray:
    if rows is None:
        return np.arange(tokens, dtype=np.int64)
    if isinstance(rows, tuple):
        return np.arange(rows[0], rows[1], dtype=np.int64)
    return np.asarray(rows, dtype=np.int64)


def _channel_state(rc: AffineRecipe, seed: int):
    g = np.random.default_rng([seed, rc.tag])
    s_c = g.lognormal(0.0, 0.5, size=rc.hidden).astype(np.float32)
    n_out = int(round(rc.outlier_frac * rc.hidden))
    out_ch = np.sort(g.choice(rc.hidden, n_out, replace=False)) if n_out else np.zeros(0, np.int64)
    zero_rows = np.zeros(rc.tokens, dtype=bool)
    n_zero = int(round(rc.zero_ref_frac * rc.tokens))
    if n_zero:
        zero_rows[g.permutation(rc.tokens)[:n_zero]] = True
    return s_c, out_ch, zero_rows


def _block(rc: AffineRecipe, seed: int, blk: int, s_c):
    n = min(BLOCK, rc.tokens - blk * BLOCK)
    g = np.random.default_rng([seed, rc.tag, 1 + blk])
    ngrp = rc.hidden // rc.group
    ref = g.standard_normal((n, rc.hidden), dtype=np.float32) * s_c
    a = g.uniform(rc.a_lo, rc.a_hi, size=(n, ngrp)).astype(np.float32)
    b = g.standard_normal((n, ngrp), dtype=np.float32) * np.float32(rc.b_sigma)
    if rc.noise == "normal":
        eps = g.standard_normal((n, rc.hidden), dtype=np.float32)
    elif rc.noise == "student_t3":
        eps = g.standard_t(3.0, size=(n, rc.hidden)).astype(np.float32)
    else:
        raise ValueError(rc.noise)
    return ref, a, b, eps * np.float32(rc.noise_scale)


def affine_pair(rc: AffineRecipe, seed: int = 0, rows=None):
    """Return (x_bits, ref_bits, zero_ref_mask) for the requested rows."""
    idx = _rows(rc.tokens, rows)
    s_c, out_ch, zero_rows = _channel_state(rc, seed)
    x_out = np.empty((idx.size, rc.hidden), dtype=np.uint16)
    r_out = np.empty((idx.size, rc.hidden), dtype=np.uint16)
    blocks = np.unique(idx // BLOCK)
    for blk in blocks:
        ref, a, b, eps = _block(rc, seed, int(blk), s_c)
        want = np.nonzero(idx // BLOCK == blk)[0]
        local = idx[want] - blk * BLOCK
        ref_b = f32_to_bf16_bits(ref[local])
        ref_f = bf16_bits_to_f32(ref_b)
        x = (np.repeat(a[local], rc.group, axis=1) * ref_f
             + np.repeat(b[local], rc.group, axis=1) + eps[local])
        if out_ch.size:
            x[:, out_ch] *= np.float32(rc.outlier_scale)
        x_out[want] = f32_to_bf16_bits(x)
        zr = zero_rows[idx[want]]
        ref_b[zr] = 0
        r_out[want] = ref_b
    return x_out, r_out, zero_rows[idx]


# ---- The benchmark shapes ------------------------------------------------

def tiny(seed: int = 0, rows=None):
    """64 tokens x 512 hidden, group 64: x = a*ref + b + N(0, 0.05^2)."""
    return affine_pair(AffineRecipe(64, 512, 64), seed, rows)


def prefill_uplink(seed: int = 0, rows=None, tokens: int = 4096, hidden: int = 4096):
    """Llama-3-8B-shaped prefill uplink, 4096 x 4096, group 128: the tiny
    recipe plus 0.1% outlier channels scaled x20 in x only, and 20% of rows
    without a reference (ref = 0)."""
    rc = AffineRecipe(tokens, hidden, 128, outlier_frac=0.001, zero_ref_frac=0.2, tag=1)
    return affine_pair(rc, seed, rows)


def prefill_downlink_uplink(seed: int = 0, rows=None, tokens: int = 65536, hidden: int = 3584):
    """Uplink state whose reconstruction becomes the downlink reference
    (Qwen2-7B-shaped, 8 x 8192 tokens x 3584 hidden, group 128)."""
    return affine_pair(AffineRecipe(tokens, hidden, 128, tag=2), seed, rows)


def prefill_downlink(ref_bits, seed: int = 0, rows=None, tokens: int = 65536,
                     hidden: int = 3584):
    """Downlink x for the given rows from the (reconstructed uplink) reference:
    x = a*ref + b + N(0, 0.1^2), a ~ U(0.7, 1.3), b ~ N(0, 0.1^2) per group."""
    idx = _rows(tokens, rows)
    ref_f = bf16_bits_to_f32(ref_bits)
    assert ref_f.shape == (idx.size, hidden)
    ngrp = hidden // 128
    x = np.empty((idx.size, hidden), dtype=np.uint16)
    for blk in np.unique(idx // BLOCK):
        n = min(BLOCK, tokens - blk * BLOCK)
        g = np.random.default_rng([seed, 3, 1 + int(blk)])
        a = g.uniform(0.7, 1.3, size=(n, ngrp)).astype(np.float32)
        b = g.standard_normal((n, ngrp), dtype=np.float32) * np.float32(0.1)
        eps = g.standard_normal((n, hidden), dtype=np.float32) * np.float32(0.1)
        want = np.nonzero(idx // BLOCK == blk)[0]
        local = idx[want] - blk * BLOCK
        xf = (np.repeat(a[local], 128, axis=1) * ref_f[want]
              + np.repeat(b[local], 128, axis=1) + eps[local])
        x[want] = f32_to_bf16_bits(xf)
    return x


def decode_step(batch: int, seed: int = 0, hidden: int = 4096):
    """GLM-4-9B-shaped decode step: `batch` sequences x 1 token x 4096.
    P = N(0,1)*s_c is the previous token's state; ref = 0.9 P + N(0, 0.3^2)
    stands for the predictor output and x = P + N(0, 0.2^2)."""
    g = np.random.default_rng([seed, 4, batch])
    s_c = np.random.default_rng([seed, 4]).lognormal(0.0, 0.5, size=hidden).astype(np.float32)
    p = g.standard_normal((batch, hidden), dtype=np.float32) * s_c
    ref = np.float32(0.9) * p + g.standard_normal((batch, hidden), dtype=np.float32) * np.float32(0.3)
    x = p + g.standard_normal((batch, hidden), dtype=np.float32) * np.float32(0.2)
    return f32_to_bf16_bits(x), f32_to_bf16_bits(ref)


def long_context(seed: int = 0, rows=None, group: int = 128, tokens: int = 32768,
                 hidden: int = 4096):
    """32768 x 4096: x = a*ref + b + 0.05 t_3 (Student-t, 3 degrees of
    freedom), half of the rows without a reference."""
    rc = AffineRecipe(tokens, hidden, group, noise="student_t3", noise_scale=0.05,
                      zero_ref_frac=0.5, tag=5)
    return affine_pair(rc, seed, rows)


# ---- Decode-phase reference predictor -------------------------------------

PREDICTOR_SECTIONS = ("w_in", "g1", "w_qkv", "w_o", "g2", "w_gu", "w_down", "g3", "w_out")


def predictor_weights(hidden: int, model: int, ffn: int, seed: int = 0) -> dict:
    """Random weights of the one-layer predictor (the trained ones are not
    available), as bf16 patterns: every matrix [outputs][inputs] drawn
    N(0, 1/inputs), every RMSNorm gain 1 + N(0, 0.1^2).  W_gu interleaves the
    gate (even rows) and up (odd rows) projections."""
    g = np.random.default_rng([seed, 6])
    mat = lambda o, i: f32_to_bf16_bits(g.standard_normal((o, i), dtype=np.float32) / np.float32(np.sqrt(i)))
    gain = lambda n: f32_to_bf16_bits(1.0 + 0.1 * g.standard_normal(n, dtype=np.float32))
    return {"w_in": mat(model, hidden), "g1": gain(model), "w_qkv": mat(3 * model, model),
            "w_o": mat(model, model), "g2": gain(model), "w_gu": mat(2 * ffn, model),
            "w_down": mat(model, ffn), "g3": gain(model), "w_out": mat(hidden, model)}


def decode_sequence(batch: int, steps: int, seed: int = 0, hidden: int = 4096):
    """Boundary states of `batch` sequences over `steps` decode steps
    (GLM-4-9B-shaped, 4096 hidden): a per-channel scale s_c ~ LogNormal(0, 0.5)
    and a state that drifts, x_t = 0.95 x_{t-1} + 0.3 N(0, 1) s_c, as bf16
    [steps][batch][hidden]."""
    g = np.random.default_rng([seed, 7, batch])
    s_c = g.lognormal(0.0, 0.5, size=hidden).astype(np.float32)
    x = g.standard_normal((batch, hidden), dtype=np.float32) * s_c
    out = np.empty((steps, batch, hidden), dtype=np.uint16)
    for t in range(steps):
        if t:
            x = np.float32(0.95) * x + np.float32(0.3) * g.standard_normal((batch, hidden), dtype=np.float32) * s_c
        out[t] = f32_to_bf16_bits(x)
    return out
