"""GPU parity of the decode-phase reference predictor against its binary64
oracle, through the C ABI.

The bar, per output element: |R_gpu - r| <= 2^-8 |r| + 2^-6 rms(y), with r
the oracle's unrounded x + y and y its predicted update, and on average
mean|R_gpu - r| <= 2^-9 mean|r| + 2^-10 rms(y).  Where it comes from: R is
bf16 (at most half an ulp, 2^-9 |r|, a quarter ulp on average);
the GPU accumulates in binary32 in another order than the binary64 oracle,
so the bf16 rounding of an intermediate activation (the normalized inputs,
the attention output, the SwiGLU output, the cached keys and values) lands on
the other neighbour where the exact value sits next to a rounding boundary,
which moves that activation by one bf16 ulp and the outputs it feeds by a
small fraction of rms(y).  A wrong lane layout, weight section, rotation or
window would be off by about rms(y).  The cached keys and values are checked
the same way against the oracle's cache.
"""
from __future__ import annotations

import numpy as np
import pytest

import paper_2608_04991_amd as rac
from oracle import predictor as P
from paper_2608_04991_amd import workloads as wl
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rac.library()


def _run(cfg, batch, steps, pos_of, seed=0, check_every=1):
    import torch
    weights = wl.predictor_weights(cfg.hidden, cfg.model, cfg.ffn, seed)
    blob = torch.from_numpy(rac.predictor_pack(cfg, weights)).cuda()
    cache = torch.zeros(rac.rac_predictor_cache_bytes(cfg) // 2, dtype=torch.int16, device="cuda")
    ws = torch.empty(rac.rac_predictor_workspace_bytes(cfg), dtype=torch.uint8, device="cuda")
    ref = P.Predictor(weights, cfg.hidden, cfg.model, cfg.heads, cfg.ffn, cfg.window, cfg.max_batch)
    xs = wl.decode_sequence(batch, steps, seed, hidden=cfg.hidden)
    out = torch.empty(batch, cfg.hidden, dtype=torch.int16, device="cuda")
    worst = 0.0
    for s in range(steps):
        pos = np.asarray([pos_of(s, b) for b in range(batch)], np.int32)
        x = torch.from_numpy(xs[s].view(np.int16)).cuda()
        rac.rac_predictor_step(cfg, blob, cache, torch.from_numpy(pos).cuda(), x, out, ws, batch)
        _, inter = ref.step(xs[s], pos)
        if s % check_every and s != steps - 1:
            continue
        torch.cuda.synchronize()
        g = P.bf16_to_f64(out.cpu().numpy().view(np.uint16))
        r, y = inter["r"], inter["y"]
        ry = np.sqrt(np.mean(y * y))
        err = np.abs(g - r)
        assert np.all(err <= 2.0 ** -8 * np.abs(r) + 2.0 ** -6 * ry), \
            f"step {s}: worst {np.max(err / (2.0 ** -8 * np.abs(r) + 2.0 ** -6 * ry)):.3f} of the bar"
        assert err.mean() <= 2.0 ** -9 * np.abs(r).mean() + 2.0 ** -10 * ry, (s, err.mean() / ry)
        worst = max(worst, float((err / ry).max()))
        # (for the record: elements whose bf16 differs from the oracle's rounding of r)
        off = float(np.mean(g != P.to_bf16(r)))
        say(f"[gpu]   step {s}: max |R - r| {err.max() / ry:.2e} rms(y), mean {err.mean() / ry:.2e}, "
            f"{off:.2%} of elements off the oracle's bf16")
    torch.cuda.synchronize()
    gc = P.bf16_to_f64(cache.cpu().numpy().view(np.uint16)).reshape(ref.cache.shape)
    used = np.zeros(ref.cache.shape[:2], dtype=bool)
    for b in range(batch):
        for s in range(steps):
            used[b, pos_of(s, b) % cfg.window] = True
    oc = ref.cache[used]
    rc = np.sqrt(np.mean(oc * oc))
    assert np.all(np.abs(gc[used] - oc) <= 2.0 ** -7 * np.abs(oc) + 2.0 ** -7 * rc)
    return worst


def test_predictor_glm_shape_70_steps_window_wraps():
    cfg = rac.PredictorConfig(4096, 512, 8, 2048, 64, 64)
    say("[gpu] predictor 4096/512/8/2048, window 64, batch 16, 70 steps")
    worst = _run(cfg, 16, 70, lambda s, b: s, check_every=7)
    say(f"[gpu] predictor: worst |R - r| = {worst:.2e} rms(y)")


def test_predictor_ragged_batch_with_staggered_and_restarted_positions():
    cfg = rac.PredictorConfig(512, 128, 2, 256, 5, 40)
    # sequence b starts at position 7 (b % 3); every fifth restarts at step 6
    pos = lambda s, b: (s - 6 if (b % 5 == 0 and s >= 6) else s + 7 * (b % 3))
    say("[gpu] predictor 512/128/2/256, window 5, batch 37, 12 steps")
    _run(cfg, 37, 12, pos)


@pytest.mark.parametrize("batch", [1, 100, 256])
def test_predictor_single_and_full_batches(batch):
    # (100: the wide products with a ragged second tile of 64 rows)
    cfg = rac.PredictorConfig(4096, 512, 8, 2048, 64, 256)
    say(f"[gpu] predictor batch {batch}, 3 steps")
    _run(cfg, batch, 3, lambda s, b: s + 100 * (b % 2), seed=1)


@pytest.mark.parametrize("window,start", [(300, 400), (1024, 1500)])
def test_predictor_windows_longer_than_one_pass_of_64_positions(window, start):
    # sequences start deep into their positions, so the window reaches back
    # over slots never written (zero on both sides) and spans several passes
    # of 64 positions in the score loop
    cfg = rac.PredictorConfig(512, 128, 2, 256, window, 8)
    say(f"[gpu] predictor 512/128/2/256, window {window}, batch 8, 4 steps from position {start}")
    _run(cfg, 8, 4, lambda s, b: start + s + 37 * b, seed=2)



@pytest.mark.parametrize("hidden,model,heads,ffn,window,batch", [
    (4096, 512, 8, 2048, 64, 2), (4096, 512, 8, 2048, 64, 4),
    (1024, 2048, 32, 512, 16, 3), (512, 128, 2, 256, 5, 4)])
def test_predictor_small_batches_fold_the_norms(hidden, model, heads, ffn, window, batch):
    # batches of at most four rows form each norm inside the product that
    # consumes it; widths 128 to 2048, including a down projection of one
    # K range (ffn 256 and 512)
    cfg = rac.PredictorConfig(hidden, model, heads, ffn, window, 4)
    say(f"[gpu] predictor {hidden}/{model}/{heads}/{ffn}, window {window}, batch {batch}, 6 steps")
    _run(cfg, batch, 6, lambda s, b: s + 3 * b, seed=4)
