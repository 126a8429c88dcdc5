"""Oracle of the decode-phase reference predictor.  TEST INFRASTRUCTURE ONLY:
only the tests, the smoke check and the benchmark's CPU baseline may call it;
it shares no code with the HIP library.

Subsection "Predicted References for Decode", Eq. decode-predictor: from the
second decode step on, a one-layer causal Transformer with a key-value cache
over a bounded history maps the previous reconstruction H-hat^{t-1} of a
sequence to the reference of step t.  The paper gives neither the block's
sizes nor its weights; the reading here (also the library's) is a pre-norm
block between a projection from and a residual projection back to the
boundary width:

    h0 = x W_in^T
    q, k, v = RMSNorm(h0; g1) W_qkv^T, rotary positions on q and k
    o  = softmax(q k^T / sqrt(64)) v over the last `window` inputs
    h1 = h0 + o W_o^T
    h2 = h1 + (silu(n2 W_gate^T) * (n2 W_up^T)) W_down^T,  n2 = RMSNorm(h1; g2)
    R  = x + RMSNorm(h2; g3) W_out^T

Arithmetic in binary64, with values rounded to bf16 where the definition
stores them in bf16 (the normalized activations, the attention output, the
SwiGLU output, the cached keys and values, R); x and the weights are bf16.
"""
from __future__ import annotations

import numpy as np

HEAD = 64
EPS = 1e-6


def bf16_to_f64(bits) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def to_bf16(a) -> np.ndarray:
    """Nearest bf16 (ties to even) of binary64 values, as binary64."""
    a = np.asarray(a, dtype=np.float64)
    f = a.astype(np.float32)
    # one rounding to bf16 from the binary64 value: pick the nearer of the two
    # bf16 neighbours of the float32 truncation's bracket
    u = f.view(np.uint32).astype(np.uint64)
    lo = (u & 0xFFFF0000)
    hi = lo + 0x10000
    v_lo = (lo.astype(np.uint32)).view(np.float32).astype(np.float64)
    v_hi = (hi.astype(np.uint32)).view(np.float32).astype(np.float64)
    # for negative values the truncation is toward zero as well (sign-magnitude)
    d_lo, d_hi = np.abs(a - v_lo), np.abs(a - v_hi)
    even_lo = ((lo >> 16) & 1) == 0
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ~even_lo)
    return np.where(pick_hi, v_hi, v_lo)


def bf16_bits(a) -> np.ndarray:
    v = to_bf16(a).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def rmsnorm(h, gain) -> np.ndarray:
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + EPS) * gain


def rope(v, pos) -> np.ndarray:
    """Rotary positions on [..., heads*64] rows at positions pos[...]: the
    channel pair (2i, 2i+1) of every head turned by pos * 10000^(-2i/64)."""
    out = np.array(v, dtype=np.float64, copy=True)
    i = np.arange(HEAD // 2)
    theta = 10000.0 ** (-2.0 * i / HEAD)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * theta       # [..., 32]
    c, s = np.cos(ang), np.sin(ang)
    sh = v.shape[:-1] + (v.shape[-1] // HEAD, HEAD // 2, 2)
    pr = np.asarray(v, dtype=np.float64).reshape(sh)
    a, b = pr[..., 0], pr[..., 1]
    c, s = c[..., None, :], s[..., None, :]
    out = np.stack([a * c - b * s, a * s + b * c], axis=-1)
    return out.reshape(v.shape)


def attend(q, keys, values) -> np.ndarray:
    """softmax(q . keys^T / 8) . values for one head: q [64], keys/values [n][64]."""
    s = keys @ q / np.sqrt(HEAD)
    p = np.exp(s - s.max())
    return (p / p.sum()) @ values


def silu(z) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


class Predictor:
    """Weights (bf16 patterns, as from workloads.predictor_weights) and a
    key-value cache [max_batch][window][2][model] of bf16 values."""

    def __init__(self, weights: dict, hidden: int, model: int, heads: int, ffn: int, window: int, max_batch: int):
        assert heads * HEAD == model
        self.W = {k: bf16_to_f64(v) for k, v in weights.items()}
        self.d, self.m, self.h, self.f, self.win = hidden, model, heads, ffn, window
        self.cache = np.zeros((max_batch, window, 2, model), dtype=np.float64)

    def step(self, x_bits, pos):
        """One decode step for rows b < len(pos): x_bits bf16 [B][hidden] (the
        previous reconstructions), pos [B] the input positions.  Updates the
        cache; returns (R as bf16 patterns [B][hidden], intermediates)."""
        W, m, win = self.W, self.m, self.win
        x = bf16_to_f64(x_bits)
        B = x.shape[0]
        pos = np.maximum(np.asarray(pos, dtype=np.int64), 0)
        h0 = x @ W["w_in"].T
        n1 = to_bf16(rmsnorm(h0, W["g1"]))
        qkv = n1 @ W["w_qkv"].T
        q, k, v = qkv[:, :m], qkv[:, m:2 * m], qkv[:, 2 * m:]
        q, k = rope(q, pos), rope(k, pos)
        kb, vb = to_bf16(k), to_bf16(v)
        o = np.zeros((B, m))
        for b in range(B):
            p = int(pos[b])
            self.cache[b, p % win, 0] = kb[b]
            self.cache[b, p % win, 1] = vb[b]
            span = range(max(0, p - win + 1), p + 1)
            keys = np.stack([self.cache[b, pp % win, 0] for pp in span])
            vals = np.stack([self.cache[b, pp % win, 1] for pp in span])
            for hh in range(self.h):
                c = slice(hh * HEAD, (hh + 1) * HEAD)
                o[b, c] = attend(q[b, c], keys[:, c], vals[:, c])
        o = to_bf16(o)
        h1 = h0 + o @ W["w_o"].T
        n2 = to_bf16(rmsnorm(h1, W["g2"]))
        gu = n2 @ W["w_gu"].T
        g = to_bf16(silu(gu[:, 0::2]) * gu[:, 1::2])
        h2 = h1 + g @ W["w_down"].T
        n3 = to_bf16(rmsnorm(h2, W["g3"]))
        y = n3 @ W["w_out"].T
        r = x + y
        return bf16_bits(r), dict(h0=h0, h1=h1, h2=h2, q=q, k=k, v=v, o=o, g=g, y=y, r=r)
