"""Benchmark of the RAC codec hot path on one MI355X.

One step = one pass of the whole hot path over one batch of the prefill-uplink
workload (Llama-3-8B-shaped boundary state: 4096 tokens x 4096 hidden bf16,
alignment/quantization group 128, 4-bit codes, top-8 outliers per token):
rac_encode with the fused sender reconstruction, then the receiver's
rac_decode, on one stream.  Inputs are resident in HBM before timing starts;
batches rotate through enough buffer sets (> 1 GB) that no step finds its
inputs in the 256 MB Infinity Cache.  Untimed steps run for --warm-ms first:
the GPU clock climbs over the first ~20 ms of sustained load, and the timed
steps measure the steady state.

Prints ONE JSON line:
  value       bf16 activation bytes processed per second (2*T*d per step), GB/s
  roofline    the encode kernel (the dominant one): algorithmic bytes per
              launch / its average HIP-event duration, against 8 TB/s
  cpu_baseline the CPU oracle (single thread) on the same step
  extras      encode-only and decode-only rates, decode-phase µs per call at
              batch 1/16/64/256 (GLM-4-9B-shaped, 4096 hidden), and the same
              4096 x 4096 inputs coded with k_g outliers per quantization
              group instead of per token (and with none, for comparison)
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "rac_encode_prefill_uplink_4096x4096_traffic.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(T, d, wire_bytes, xhat_bytes_per_elem=4, encode=True):
    """Minimum bytes one launch must move: encode reads x and ref and writes
    the wire and x-hat; decode reads the wire and ref and writes x-hat."""
    elems = T * d
    if encode:
        return elems * 2 + elems * 2 + wire_bytes + elems * xhat_bytes_per_elem
    return wire_bytes + elems * 2 + elems * xhat_bytes_per_elem


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--warm-ms", type=float, default=50.0,
                    help="after the warmup steps, keep running untimed steps for this long: the GPU clock "
                         "climbs for the first ~20 ms of sustained load")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true")
    ap.add_argument("--all-configs", action="store_true",
                    help="also time every other workload at full size (tiny 64 x 512; prefill downlink "
                         "65536 x 3584; long context 32768 x 4096 at groups 64 and 128 and 2/3/4/8 bits) "
                         "into extras.all_configs; adds about a minute")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run plain device copies of MIB MiB (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the codec shards by token rows with no "
              "exchange between GPUs, so multi-GPU runs are not part of this benchmark.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_04991_amd as rac
    from paper_2608_04991_amd import workloads as wl
    from paper_2608_04991_amd import rocprof_summary

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copied {n} bytes 5 times")
        return
    rac.library()
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()

    T, d, g, b, k = 4096, 4096, 128, 4, 8
    cfg = rac.RacConfig(T, d, g, g, b, k)
    wbytes = rac.rac_wire_size(cfg)
    log("[bench] generating the prefill-uplink workload")
    xb, rb, _ = wl.prefill_uplink(0)
    x0, r0 = dev(xb), dev(rb)
    set_bytes = 2 * T * d * 2 + 2 * T * d * 4 + wbytes
    nsets = max(2, int(np.ceil(1.2e9 / set_bytes)))
    sets = []
    for i in range(nsets):
        sets.append(dict(x=x0.clone(), ref=r0.clone(),
                         wire=torch.empty(wbytes, dtype=torch.uint8, device="cuda"),
                         xhat=torch.empty(T, d, dtype=torch.float32, device="cuda"),
                         xdec=torch.empty(T, d, dtype=torch.float32, device="cuda")))
    stream = torch.cuda.current_stream()

    def encode(i):
        s = sets[i % nsets]
        rac.rac_encode(cfg, s["x"], s["ref"], None, s["wire"], s["xhat"], stream=stream)

    def decode(i):
        s = sets[i % nsets]
        rac.rac_decode(cfg, s["wire"], s["ref"], None, s["xdec"], stream=stream)

    log(f"[bench] warmup {args.warmup} steps, then {args.warm_ms:g} ms ({nsets} rotating buffer sets)")
    for i in range(args.warmup):
        encode(i)
        decode(i)
    torch.cuda.synchronize()
    t_warm, i = time.perf_counter(), 0
    while (time.perf_counter() - t_warm) * 1e3 < args.warm_ms:
        for _ in range(10):
            encode(i)
            decode(i)
            i += 1
        torch.cuda.synchronize()
    # The timed steps: encode + decode per step, back to back on one stream.
    log(f"[bench] timing {args.steps} steps")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        encode(i)
        decode(i)
    ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    gpu_ms_per_step = ev[0].elapsed_time(ev[1]) / args.steps
    # Per-launch durations of each kernel on the same stream, as in the timed
    # steps (back to back, rotating buffers): the encodes of the timed steps
    # again, then their decodes, each run bracketed by HIP events.
    ev[2].record(stream)
    for i in range(args.steps):
        encode(i)
    ev[3].record(stream)
    for i in range(args.steps):
        decode(i)
    ev[4].record(stream)
    torch.cuda.synchronize()
    enc_ms = ev[2].elapsed_time(ev[3]) / args.steps
    dec_ms = ev[3].elapsed_time(ev[4]) / args.steps
    act_bytes = T * d * 2
    value = act_bytes / (ms_per_step * 1e-3) / 1e9

    # parity spot check of the timed configuration (first rows) vs the sender
    s0 = sets[0]
    assert torch.equal(s0["xhat"], s0["xdec"]), "sender and receiver reconstructions differ"

    enc_alg = algorithmic_bytes(T, d, wbytes)
    dec_alg = algorithmic_bytes(T, d, wbytes, encode=False)
    enc_avg_s = enc_ms * 1e-3
    dec_avg_s = dec_ms * 1e-3
    achieved = enc_alg / enc_avg_s / 1e9
    # HBM bytes per launch from the committed rocprofv3 counter runs, valid
    # only for the kernel source they were taken on
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        t = json.load(open(TRAFFIC_FILE))
        if t.get("kernel_source_sha256_16") == rocprof_summary.source_hash():
            traffic = round(t["bytes_per_launch"])
    out = {
        "metric": "encode+reconstruct GB/s of bf16 activation & % HBM peak; decode-step µs/call",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "prefill uplink, Llama-3-8B-shaped: x,ref bf16 4096 tokens x 4096 hidden, "
                               "group 128, 4-bit, top-8 outliers/token; step = rac_encode (fused sender "
                               "reconstruction, fp32) + rac_decode",
                   "tokens": T, "hidden": d, "group": g, "bits": b, "outlier_k": k,
                   "wire_bytes": wbytes, "rotating_buffer_sets": nsets},
        "roofline": {"kernel": "rac_encode_rows_kernel<4,4,4,4,2,false>", "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": enc_alg,
                     "avg_launch_us": round(enc_avg_s * 1e6, 3)},
    }
    extras = {
        "encode_recon_GBps_activation": round(act_bytes / enc_avg_s / 1e9, 1),
        "encode_us": round(enc_avg_s * 1e6, 2),
        "decode_us": round(dec_avg_s * 1e6, 2),
        "decode_GBps_activation": round(act_bytes / dec_avg_s / 1e9, 1),
        "decode_hbm_frac": round(dec_alg / dec_avg_s / 1e9 / HBM_PEAK_GBPS, 4),
        "gpu_ms_per_step": round(gpu_ms_per_step, 5),
    }
    if not args.no_extras:
        extras["decode_step"] = decode_step_latency(torch, rac, wl, dev, stream)
        # graph-replayed encode + decode pair, µs, across the bit widths and
        # with one scale per token row (quantization group = hidden)
        extras["decode_step_graph_pair_us"] = {
            f"b{bits}_gq{gq}": decode_step_latency(torch, rac, wl, dev, stream, bits, gq, detail=False)
            for bits, gq in ((2, 128), (8, 128), (4, 4096))}
        extras["outlier_modes_4096x4096_g128_b4"] = outlier_mode_rates(
            torch, rac, sets, nsets, stream, args.steps)
        extras["gathered_reference"] = gather_rates(torch, rac, cfg, rb, sets, nsets, stream, args.steps)
        extras["span_selection"] = span_selection_cost(rac, T)
        extras["pooled_fit"] = pooled_rates(torch, rac, cfg, sets, nsets, stream, args.steps)
    if args.all_configs:
        del sets
        torch.cuda.empty_cache()
        extras["all_configs"] = all_config_rates(torch, rac, wl, dev, stream)
    out["extras"] = extras

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(xb, rb, cfg)
    print(json.dumps(out), flush=True)


def outlier_mode_rates(torch, rac, sets, nsets, stream, steps):
    """Average launch time (HIP events around `steps` back-to-back launches
    over the rotating buffer sets) of rac_encode and of rac_decode on the
    benchmark inputs with other outlier settings: k_g = 1, 2, 4 outliers per
    quantization group (u8 offsets), and none.  Each entry gives µs, the
    fraction of 8 TB/s by algorithmic bytes, and the wire size relative to
    the bf16 tensor."""
    res = {}
    variants = {"none": (0, 0), "per_group_kg1": (1, rac.RAC_FLAG_GROUP_OUTLIERS),
                "per_group_kg2": (2, rac.RAC_FLAG_GROUP_OUTLIERS),
                "per_group_kg4": (4, rac.RAC_FLAG_GROUP_OUTLIERS)}
    T, d = 4096, 4096
    for name, (k, flags) in variants.items():
        cfg = rac.RacConfig(T, d, 128, 128, 4, k, flags)
        wb = rac.rac_wire_size(cfg)
        wires = [torch.empty(wb, dtype=torch.uint8, device="cuda") for _ in range(nsets)]

        def enc(i):
            s = sets[i % nsets]
            rac.rac_encode(cfg, s["x"], s["ref"], None, wires[i % nsets], s["xhat"], stream=stream)

        def dec(i):
            s = sets[i % nsets]
            rac.rac_decode(cfg, wires[i % nsets], s["ref"], None, s["xdec"], stream=stream)

        for i in range(2 * nsets):
            enc(i)
            dec(i)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for i in range(steps):
            enc(i)
        ev[1].record(stream)
        for i in range(steps):
            dec(i)
        ev[2].record(stream)
        torch.cuda.synchronize()
        assert torch.equal(sets[0]["xhat"], sets[0]["xdec"]), name
        e_us = ev[0].elapsed_time(ev[1]) / steps * 1e3
        d_us = ev[1].elapsed_time(ev[2]) / steps * 1e3
        res[name] = {"encode_us": round(e_us, 2),
                     "encode_hbm_frac": round(algorithmic_bytes(T, d, wb) / e_us / 1e3 / HBM_PEAK_GBPS, 4),
                     "decode_us": round(d_us, 2),
                     "decode_hbm_frac": round(algorithmic_bytes(T, d, wb, encode=False) / d_us / 1e3
                                              / HBM_PEAK_GBPS, 4),
                     "wire_over_bf16": round(wb / (T * d * 2), 4)}
        del wires
    return res


def time_pair(torch, rac, cfg, sets, stream, iters=20):
    """Average µs of rac_encode (fused fp32 reconstruction), of rac_decode,
    and of encode + decode on one stream, each over `iters` back-to-back
    launches rotating over `sets` (inputs and outputs per set), after at
    least 60 ms of untimed launches."""
    n = len(sets)

    def enc(i):
        s = sets[i % n]
        rac.rac_encode(cfg, s["x"], s["ref"], None, s["wire"], s["xhat"], stream=stream)

    def dec(i):
        s = sets[i % n]
        rac.rac_decode(cfg, s["wire"], s["ref"], None, s["xdec"], stream=stream)

    # untimed launches for at least 60 ms first: the data of each workload is
    # generated on the host while the GPU idles, and its clock drops meanwhile
    t0, i = time.perf_counter(), 0
    while (time.perf_counter() - t0) < 0.06 or i < 2 * n:
        enc(i)
        dec(i)
        i += 1
        if i % 4 == 0:
            torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(iters):
        enc(i)
    ev[1].record(stream)
    for i in range(iters):
        dec(i)
    ev[2].record(stream)
    for i in range(iters):
        enc(i)
        dec(i)
    ev[3].record(stream)
    torch.cuda.synchronize()
    assert torch.equal(sets[0]["xhat"], sets[0]["xdec"])
    return [ev[j].elapsed_time(ev[j + 1]) / iters * 1e3 for j in range(3)]


def all_config_rates(torch, rac, wl, dev, stream):
    """Every other workload at its full size, on its own synthetic data: µs
    per call of encode, decode and the encode + decode round trip on one
    stream, with the fraction of 8 TB/s by algorithmic bytes (the tiny case
    is launch-bound and reports µs only).  Two buffer sets rotate (each set of
    the large shapes is far above the 256 MB last-level cache; the tiny case
    uses 64)."""
    out = {}

    def run(name, cfg, xb, rb, nsets, report_frac=True):
        T, d = cfg.tokens, cfg.hidden
        wb = rac.rac_wire_size(cfg)
        x, r = dev(xb), dev(rb)
        sets = [dict(x=x if i == 0 else x.clone(), ref=r if i == 0 else r.clone(),
                     wire=torch.empty(wb, dtype=torch.uint8, device="cuda"),
                     xhat=torch.empty(T, d, dtype=torch.float32, device="cuda"),
                     xdec=torch.empty(T, d, dtype=torch.float32, device="cuda")) for i in range(nsets)]
        e, dcd, rt = time_pair(torch, rac, cfg, sets, stream)
        res = {"encode_us": round(e, 2), "decode_us": round(dcd, 2), "round_trip_us": round(rt, 2),
               "wire_over_bf16": round(wb / (T * d * 2), 4)}
        if report_frac:
            res["encode_hbm_frac"] = round(algorithmic_bytes(T, d, wb) / e / 1e3 / HBM_PEAK_GBPS, 4)
            res["decode_hbm_frac"] = round(algorithmic_bytes(T, d, wb, encode=False) / dcd / 1e3 / HBM_PEAK_GBPS, 4)
            res["activation_GBps_round_trip"] = round(T * d * 2 / rt / 1e3, 1)
        out[name] = res
        log(f"[bench] {name}: {res}")
        del sets
        torch.cuda.empty_cache()

    xb, rb, _ = wl.tiny(0)
    run("tiny_64x512_g64_b4", rac.RacConfig(64, 512, 64, 64, 4, 0), xb, rb, 64, report_frac=False)
    # prefill downlink: the reference is the sender reconstruction (bf16) of a
    # synthetic uplink, made here by the GPU encode (bit-identical to the
    # oracle's, which the GPU tests check on sampled rows)
    T, d = 65536, 3584
    cfg = rac.RacConfig(T, d, 128, 128, 4, 4)
    log("[bench] generating the prefill-downlink workload")
    xu, ru, _ = wl.prefill_downlink_uplink(0)
    xh = torch.empty(T, d, dtype=torch.float32, device="cuda")
    w = torch.empty(rac.rac_wire_size(cfg), dtype=torch.uint8, device="cuda")
    rac.rac_encode(cfg, dev(xu), dev(ru), None, w, xh, stream=stream)
    torch.cuda.synchronize()
    ref = wl.f32_to_bf16_bits(xh.cpu().numpy())
    del xh, w, xu, ru
    torch.cuda.empty_cache()
    xd = wl.prefill_downlink(ref, 0)
    run("prefill_downlink_65536x3584_g128_b4_k4", cfg, xd, ref, 2)
    del xd, ref
    for g in (64, 128):
        log(f"[bench] generating the long-context workload, group {g}")
        xb, rb, _ = wl.long_context(0, group=g)
        for bits in (2, 3, 4, 8):
            run(f"long_context_32768x4096_g{g}_b{bits}_k16", rac.RacConfig(32768, 4096, g, g, bits, 16), xb, rb, 2)
    return out


def pooled_rates(torch, rac, cfg, sets, nsets, stream, steps):
    """rac_encode_pooled on the benchmark inputs, with segments standing for
    retrieved spans (random lengths of 1 to 600 rows): average time of the
    whole call (its three launches) over `steps` back-to-back calls, and the
    fraction of 8 TB/s by the per-token encode's algorithmic bytes (the
    pooled call also reads x and ref a second time for the moments)."""
    T, d = cfg.tokens, cfg.hidden
    rng = np.random.default_rng(12)
    cuts = np.unique(np.concatenate([[0, T], np.cumsum(rng.integers(1, 600, 40))]))
    seg = torch.from_numpy(cuts[cuts <= T].astype(np.int32)).cuda()
    wb = rac.rac_wire_size(cfg)
    wires = [torch.empty(wb, dtype=torch.uint8, device="cuda") for _ in range(nsets)]

    def enc(i):
        s = sets[i % nsets]
        rac.rac_encode_pooled(cfg, s["x"], s["ref"], seg, None, wires[i % nsets], s["xhat"], stream=stream)

    for i in range(2 * nsets):
        enc(i)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(steps):
        enc(i)
    ev[1].record(stream)
    torch.cuda.synchronize()
    us = ev[0].elapsed_time(ev[1]) / steps * 1e3
    del wires
    return {"segments": int(seg.numel()) - 1, "encode_us": round(us, 2),
            "hbm_frac_by_encode_bytes": round(algorithmic_bytes(T, d, wb) / us / 1e3 / HBM_PEAK_GBPS, 4)}


def span_selection_cost(rac, T, window=16, n_hist=7):
    """Host cost of the reference selection (librac's span index, one CPU
    thread) for a T-token prompt against n_hist earlier T-token requests of a
    synthetic agent session: a shared system prompt, stretches copied from
    earlier requests, fresh tokens.  Index build time for the history, then
    the selection time for the prompt, and the fraction of positions
    covered."""
    rng = np.random.default_rng(3)
    system = rng.integers(0, 32000, T // 4).tolist()
    reqs = []
    for _ in range(n_hist + 1):
        r = list(system)
        while len(r) < T:
            if reqs and rng.random() < 0.6:
                src = reqs[rng.integers(0, len(reqs))]
                a = int(rng.integers(0, len(src)))
                r += src[a:a + int(rng.integers(16, 400))]
            else:
                r += rng.integers(0, 32000, int(rng.integers(1, 64))).tolist()
        reqs.append(r[:T])
    reqs = [np.asarray(r, np.int32) for r in reqs]
    t0 = time.perf_counter()
    ix = rac.SpanIndex(window)
    for i in range(n_hist):
        ix.add(reqs[i], i * T)
    t1 = time.perf_counter()
    reps = 20
    for _ in range(reps):
        idx, cov = ix.select(reqs[n_hist])
    t2 = time.perf_counter()
    ix.close()
    return {"window": window, "history_tokens": n_hist * T, "prompt_tokens": T,
            "index_build_ms": round((t1 - t0) * 1e3, 2), "select_us": round((t2 - t1) / reps * 1e6, 1),
            "covered_fraction": round(cov / T, 4)}


def gather_rates(torch, rac, cfg, rb, sets, nsets, stream, steps):
    """rac_encode_gather / rac_decode_gather on the benchmark configuration:
    each row's reference sits at a random row of an 8192-row bf16 store of
    earlier rows (one store per buffer set), a fifth of the rows name no row
    (zero reference).  Average launch time over `steps` back-to-back launches,
    next to the same calls with the reference materialized."""
    T, d = cfg.tokens, cfg.hidden
    rng = np.random.default_rng(11)
    pos = rng.permutation(2 * T)[:T].astype(np.int32)
    pos[rng.random(T) < 0.2] = -1
    idx = torch.from_numpy(pos).cuda()
    stores = []
    for i in range(nsets):
        st = torch.zeros(2 * T, d, dtype=torch.int16, device="cuda")
        ok = idx >= 0
        st[idx[ok].long()] = sets[i]["ref"][ok]
        stores.append(st)
    wb = rac.rac_wire_size(cfg)
    wires = [torch.empty(wb, dtype=torch.uint8, device="cuda") for _ in range(nsets)]

    def enc(i):
        s = sets[i % nsets]
        rac.rac_encode_gather(cfg, s["x"], stores[i % nsets], idx, None, wires[i % nsets], s["xhat"], stream=stream)

    def dec(i):
        s = sets[i % nsets]
        rac.rac_decode_gather(cfg, wires[i % nsets], stores[i % nsets], idx, None, s["xdec"], stream=stream)

    for i in range(2 * nsets):
        enc(i)
        dec(i)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(steps):
        enc(i)
    ev[1].record(stream)
    for i in range(steps):
        dec(i)
    ev[2].record(stream)
    torch.cuda.synchronize()
    assert torch.equal(sets[0]["xhat"], sets[0]["xdec"])
    del stores, wires
    return {"store_rows": 2 * T, "miss_fraction": round(float((pos < 0).mean()), 4),
            "encode_us": round(ev[0].elapsed_time(ev[1]) / steps * 1e3, 2),
            "decode_us": round(ev[1].elapsed_time(ev[2]) / steps * 1e3, 2)}


def decode_step_latency(torch, rac, wl, dev, stream, bits=4, gq=128, detail=True):
    """µs per call of rac_encode and rac_decode for decode-phase batches
    (1 token per sequence, 4096 hidden, alignment group 128, quantization
    group gq, no outliers): wall time per call with back-to-back launches,
    kernel time from HIP events (with detail), and the time per encode +
    decode pair when 20 pairs are captured in one HIP graph and replayed."""
    res = {}
    for B in (1, 16, 64, 256):
        cfg = rac.RacConfig(B, 4096, 128, gq, bits, 0)
        xb, rb = wl.decode_step(B)
        x, ref = dev(xb), dev(rb)
        wire = torch.empty(rac.rac_wire_size(cfg), dtype=torch.uint8, device="cuda")
        xh = torch.empty(B, 4096, dtype=torch.float32, device="cuda")
        xd = torch.empty_like(xh)
        for _ in range(20):
            rac.rac_encode(cfg, x, ref, None, wire, xh, stream=stream)
            rac.rac_decode(cfg, wire, ref, None, xd, stream=stream)
        torch.cuda.synchronize()
        n = 200 if detail else 20
        t0 = time.perf_counter()
        for _ in range(n):
            rac.rac_encode(cfg, x, ref, None, wire, xh, stream=stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(n):
            rac.rac_decode(cfg, wire, ref, None, xd, stream=stream)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ke, kd = [], []
        for _ in range(20 if detail else 0):
            e[0].record(stream)
            rac.rac_encode(cfg, x, ref, None, wire, xh, stream=stream)
            e[1].record(stream)
            rac.rac_decode(cfg, wire, ref, None, xd, stream=stream)
            e[2].record(stream)
            torch.cuda.synchronize()
            ke.append(e[0].elapsed_time(e[1]))
            kd.append(e[1].elapsed_time(e[2]))
        # the same pair captured in a HIP graph (20 pairs per graph), replayed
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(20):
                rac.rac_encode(cfg, x, ref, None, wire, xh)
                rac.rac_decode(cfg, wire, ref, None, xd)
        g.replay()
        torch.cuda.synchronize()
        e[0].record(stream)
        for _ in range(10):
            g.replay()
        e[1].record(stream)
        torch.cuda.synchronize()
        pair = round(e[0].elapsed_time(e[1]) * 1e3 / 200, 2)
        if not detail:
            res[f"B{B}"] = pair
            continue
        res[f"B{B}"] = {"encode_us_per_call": round((t1 - t0) / n * 1e6, 2),
                        "decode_us_per_call": round((t2 - t1) / n * 1e6, 2),
                        "encode_event_us": round(float(np.median(ke)) * 1e3, 2),
                        "decode_event_us": round(float(np.median(kd)) * 1e3, 2),
                        "graph_pair_us": pair}
    return res


def cpu_baseline(xb, rb, cfg):
    """The CPU oracle, single-threaded, on the same step (all rows: encode
    with sender reconstruction, then decode), repeated until at least 10 s of
    CPU time have been spent (at most 30 s)."""
    import oracle
    c = dict(tokens=cfg.tokens, hidden=cfg.hidden, group_align=cfg.group_align,
             group_quant=cfg.group_quant, bits=cfg.bits, outlier_k=cfg.outlier_k, flags=cfg.flags)
    log("[bench] CPU oracle baseline (full steps, single thread)")
    reps, dt = 0, 0.0
    while dt < 10.0 and reps < 30:
        t0 = time.perf_counter()
        rc, wire, _ = oracle.encode(xb, rb, **c)
        rc2, _ = oracle.decode(wire, rb, **c)
        dt += time.perf_counter() - t0
        reps += 1
        assert rc == 0 and rc2 == 0
        log(f"[bench] oracle step {reps}: {dt:.1f} s so far")
    return {"value": round(reps * cfg.tokens * cfg.hidden * 2 / dt / 1e9, 5), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{reps} full steps of the benchmark workload ({cfg.tokens}x{cfg.hidden} encode with "
                      f"sender reconstruction + decode), {dt:.1f} s, single thread on a host with "
                      f"{os.cpu_count()} visible cores"}


if __name__ == "__main__":
    main()
