"""Oracle of the codec's offline calibration.  TEST INFRASTRUCTURE ONLY: only
the tests, the smoke check and the benchmark's CPU baseline may call it; the
product path never imports it, and it shares no code with the HIP library.

The paper's calibration (subsection "Quality- and Cost-Constrained Aligned
Residual Encoding", its opening paragraph; the last sentence of "Grouped
Residual Quantization"; "Outlier Metadata and Calibration") runs the
sender's reconstruction path offline over candidate configurations, the
groupings g_a and g_q, the bit width q and, in outlier mode, the outlier
count k_g, and keeps one that meets a quality target while accounting for
the bytes of the packed values, scales, alignment coefficients and outlier
metadata.  The paper fixes neither the quality measure nor the tie rules;
this oracle reads them as follows:

  - quality: the normalized squared reconstruction error of the sender's
    reconstruction over the calibration sample,
        NMSE = sum (x - H-hat)^2 / sum x^2,
    with each difference formed in binary64 (exact for any realistic pair of
    a bf16 input and its fp32 reconstruction), each square rounded once in
    binary64 and the sum of the squares correctly rounded (math.fsum);
  - cost: the whole wire of the configuration in bytes (values, scales,
    coefficient pairs, outlier entries, the header, section padding and the
    saturation report), from the oracle's own layout;
  - choice: among candidates with NMSE <= target, the fewest bytes, ties to
    the smaller squared error, then the earlier candidate; when no candidate
    meets the target, the smallest squared error, ties to fewer bytes, then
    the earlier candidate.

The paper also names selection time among the calibration's inputs; timing
is not a quantity the oracle can fix, so the choice here is time-blind (the
benchmark reports encode times next to a calibration run).
"""
from __future__ import annotations

import math

import numpy as np

import oracle


def _bf16_to_f64(bits) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def error_stats(x_bits, xhat, xhat_bf16: bool = False):
    """(sum of squared errors, sum of x^2, max |x - H-hat|) of a
    reconstruction (fp32 array, or bf16 patterns with xhat_bf16) against the
    bf16 input x."""
    x = _bf16_to_f64(x_bits).ravel()
    h = (_bf16_to_f64(xhat) if xhat_bf16 else np.asarray(xhat, dtype=np.float32).astype(np.float64)).ravel()
    d = x - h
    sq = d * d
    return (math.fsum(sq.tolist()), math.fsum((x * x).tolist()),
            float(np.max(np.abs(d))) if d.size else 0.0)


def nmse(sq_err: float, sq_x: float) -> float:
    return sq_err / sq_x if sq_x > 0.0 else 0.0


def wire_bytes(cfg: dict) -> int:
    return oracle.layout(**cfg)["total"]


def choose(results, target: float) -> int:
    """Index of the chosen candidate; results: dicts with wire_bytes, sq_err
    and nmse, in candidate order."""
    feasible = [i for i, r in enumerate(results) if r["nmse"] <= target]
    if feasible:
        return min(feasible, key=lambda i: (results[i]["wire_bytes"], results[i]["sq_err"], i))
    return min(range(len(results)), key=lambda i: (results[i]["sq_err"], results[i]["wire_bytes"], i))


def evaluate(x_bits, ref_bits, cfg: dict) -> dict:
    """Encode the sample with one configuration and measure its
    reconstruction (the sender's, which the receiver's decode equals)."""
    rc, _, xhat = oracle.encode(x_bits, ref_bits, **cfg)
    if rc != 0:
        raise ValueError(f"oracle rejects {cfg}: status {rc}")
    se, sx, mx = error_stats(x_bits, xhat, bool(cfg.get("flags", 0) & oracle.FLAG_XHAT_BF16))
    return dict(cfg=dict(cfg), wire_bytes=wire_bytes(cfg), sq_err=se, sq_x=sx, max_abs=mx, nmse=nmse(se, sx))


def calibrate(x_bits, ref_bits, candidates, target: float):
    """Run every candidate configuration (dicts with the sample's tokens and
    hidden) over the sample; returns (chosen index, per-candidate results)."""
    results = [evaluate(x_bits, ref_bits, c) for c in candidates]
    for r in results:
        r["feasible"] = r["nmse"] <= target
    return choose(results, target), results
