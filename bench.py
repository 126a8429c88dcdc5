"""Benchmark of the RAC codec hot path on one MI355X.

One step = one pass of the whole hot path over one batch of the prefill
downlink workload, the largest one-GPU configuration (Qwen2-7B-shaped boundary
state: 8 sequences x 8192 tokens = 65536 tokens x 3584 hidden bf16, group 128,
4-bit codes, top-4 outliers per token; the reference is the bf16 sender
reconstruction of a synthetic uplink state): rac_encode with the fused fp32
sender reconstruction of one batch, and rac_decode of the batch encoded in the
step before, on one stream.  Three buffer sets of 2.9 GB rotate, so no launch
reads what the launch just before it touched: the decode reads a wire and
reference that the previous step wrote, with 3 GB of other traffic since, and
the encode reads inputs no launch has touched for two steps.  Nothing is served
from the 256 MB Infinity Cache.
Inputs are resident in HBM before timing starts.  Untimed steps run for
--warm-ms first: the GPU clock climbs over the first ~20 ms of sustained load.

Prints ONE JSON line:
  value        bf16 activation bytes processed per second (2*T*d per step), GB/s
  roofline     the encode kernel (the dominant one): algorithmic bytes per
               launch / its average duration from HIP events around each encode
               of the timed steps, against 8 TB/s; traffic from the committed
               rocprofv3 counter runs (null once the kernel source changed)
  cpu_baseline the CPU oracle, one thread pinned to one core, on a row sample
               of the same workload
  extras       encode-only and decode-only rates of the headline workload; the
               prefill uplink (4096 x 4096, k = 8), the long context
               (32768 x 4096 at groups 64/128 and 2/3/4/8 bits, k = 16) and the
               tiny case, each with its fraction of 8 TB/s; decode-phase
               microseconds per call at batch 1/16/64/256; the decode-phase
               reference predictor's step time at the same batches; the
               per-group outlier modes, gathered reference, span selection and
               pooled fit on the uplink inputs; the headline and uplink
               workloads under each launch shape (the launch hints); a plain
               1 GiB device copy as the memory system's reference.

--profile WORKLOAD runs only that workload's launches (back-to-back encodes,
then back-to-back decodes, over rotating buffers) and prints their event
timings: the command the rocprofv3 kernel traces and counter runs under
profiles/ were taken with.  --profile launch_shapes instead times encode and
decode under each launch shape over 2048 to 65536 rows of random inputs.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
# calibrated HBM traffic per launch of the headline encode, from rocprofv3
# FETCH_SIZE / WRITE_SIZE runs (see paper_2608_04991_amd/rocprof_summary.py)
LLC_BYTES = 256 << 20    # MI355X last-level (Infinity) cache
TRAFFIC_FILE = os.path.join(PROFILES, "rac_encode_prefill_downlink_65536x3584_traffic.json")
HEADLINE_KERNEL = "rac_encode_rows_kernel<4, 4, 4, 4, 2, false, false, false>"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(T, d, wire_bytes, xhat_bytes_per_elem=4, encode=True):
    """Minimum bytes one launch must move: encode reads x and ref and writes
    the wire and x-hat; decode reads the wire and ref and writes x-hat."""
    elems = T * d
    if encode:
        return elems * 2 + elems * 2 + wire_bytes + elems * xhat_bytes_per_elem
    return wire_bytes + elems * 2 + elems * xhat_bytes_per_elem


def frac(nbytes, us):
    return round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)


class Codec:
    """Buffer sets of one configuration and its encode / decode calls."""

    def __init__(self, torch, rac, cfg, x, ref, nsets, stream):
        self.torch, self.rac, self.cfg, self.stream = torch, rac, cfg, stream
        T, d = cfg.tokens, cfg.hidden
        self.wbytes = rac.rac_wire_size(cfg)
        self.sets = [dict(x=x if i == 0 else x.clone(), ref=ref if i == 0 else ref.clone(),
                          wire=torch.empty(self.wbytes, dtype=torch.uint8, device="cuda"),
                          xhat=torch.empty(T, d, dtype=torch.float32, device="cuda"),
                          xdec=torch.empty(T, d, dtype=torch.float32, device="cuda"))
                     for i in range(nsets)]
        self.n = nsets

    def enc(self, i):
        s = self.sets[i % self.n]
        self.rac.rac_encode(self.cfg, s["x"], s["ref"], None, s["wire"], s["xhat"], stream=self.stream)

    def dec(self, i):
        s = self.sets[i % self.n]
        self.rac.rac_decode(self.cfg, s["wire"], s["ref"], None, s["xdec"], stream=self.stream)

    def alg(self, encode=True):
        return algorithmic_bytes(self.cfg.tokens, self.cfg.hidden, self.wbytes, encode=encode)

    def warm(self, ms=60.0):
        """Untimed encode + decode pairs for at least `ms` (and every set
        encoded twice): the GPU clock drops while the host generates data."""
        t0, i = time.perf_counter(), 0
        while (time.perf_counter() - t0) * 1e3 < ms or i < 2 * self.n:
            self.enc(i)
            self.dec(i)
            i += 1
            if i % 4 == 0:
                self.torch.cuda.synchronize()
        self.torch.cuda.synchronize()

    def back_to_back(self, iters):
        """Average µs of `iters` back-to-back encodes, then of as many
        decodes, rotating over the sets (HIP events on the launch stream)."""
        torch = self.torch
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        torch.cuda.synchronize()
        ev[0].record(self.stream)
        for i in range(iters):
            self.enc(i)
        ev[1].record(self.stream)
        for i in range(iters):
            self.dec(i)
        ev[2].record(self.stream)
        torch.cuda.synchronize()
        s0 = self.sets[(iters - 1) % self.n]
        assert torch.equal(s0["xhat"], s0["xdec"]), "sender and receiver reconstructions differ"
        return [ev[j].elapsed_time(ev[j + 1]) / iters * 1e3 for j in range(2)]

    def steady(self, iters, reps=5):
        """Medians over `reps` back_to_back blocks: after a pause the first
        blocks run while the GPU clock ramps back up (up to 20% slower)."""
        r = np.asarray([self.back_to_back(iters) for _ in range(reps)])
        return float(np.median(r[:, 0])), float(np.median(r[:, 1]))

    def round_trip(self, iters):
        """Average µs of an encode followed by the decode of the same set."""
        torch = self.torch
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(self.stream)
        for i in range(iters):
            self.enc(i)
            self.dec(i)
        ev[1].record(self.stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / iters * 1e3

    def free(self):
        del self.sets
        self.torch.cuda.empty_cache()


SHAPE_REPS = 3  # back-to-back blocks per launch shape (their median is reported)


def launch_shape_rates(torch, rac, C, iters):
    """Encode and decode times of one workload under each launch shape: the
    default choice and the two shapes forced by the launch hints (the strided
    grid of resident workgroups, one workgroup per row).  The outputs are
    identical under every hint (checked by the GPU tests); medians of
    back-to-back blocks."""
    base = C.cfg
    out = {}
    C.warm(100)
    for name, hint in (("default", 0), ("strided", rac.RAC_FLAG_LAUNCH_STRIDED),
                       ("per_row", rac.RAC_FLAG_LAUNCH_PER_ROW)):
        C.cfg = dataclasses.replace(base, flags=base.flags | hint)
        C.warm(30)
        e, d = C.steady(iters, reps=SHAPE_REPS)
        out[name] = {"encode_us": round(e, 2), "decode_us": round(d, 2)}
    C.cfg = base
    return out


def launch_shape_sweep(torch, rac, stream, iters):
    """Encode and decode µs under each launch shape over 2048 to 65536 rows at
    4096 channels (k = 8) and 3584 channels (k = 4), group 128, 4-bit, on
    random inputs (x ~ N(0, 0.25) with every 97th channel scaled x12, ref = x
    plus N(0, 0.0025)), generated on the device."""
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    out = {}
    for d, k in ((4096, 8), (3584, 4)):
        for T in (2048, 4096, 8192, 16384, 32768, 65536):
            cfg = rac.RacConfig(T, d, 128, 128, 4, k)
            x = torch.randn(T, d, device="cuda", generator=g) * 0.5
            x[:, ::97] *= 12.0
            ref = (x + 0.05 * torch.randn(T, d, device="cuda", generator=g)).bfloat16().view(torch.int16)
            x = x.bfloat16().view(torch.int16)
            nsets = max(2, int(np.ceil(2 * LLC_BYTES / (T * d * 8))))
            C = Codec(torch, rac, cfg, x, ref, nsets, stream)
            res = launch_shape_rates(torch, rac, C, iters)
            out[f"{T}x{d}_k{k}"] = res
            log(f"[bench] launch shapes {T}x{d}: {res}")
            C.free()
            del C, x, ref
            torch.cuda.empty_cache()
    return out


def to_dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def downlink_workload(torch, rac, wl, stream):
    """Prefill downlink inputs on the device: the reference is the bf16 sender
    reconstruction of a synthetic uplink (made by the GPU encode, which the
    GPU tests check bit for bit against the oracle on sampled rows); x is
    drawn from it on the host.  Returns (cfg, x_dev, ref_dev, x_bits, ref_bits)."""
    T, d = 65536, 3584
    cfg = rac.RacConfig(T, d, 128, 128, 4, 4)
    log("[bench] generating the prefill-downlink workload (uplink state)")
    xu, ru, _ = wl.prefill_downlink_uplink(0)
    xh = torch.empty(T, d, dtype=torch.float32, device="cuda")
    w = torch.empty(rac.rac_wire_size(cfg), dtype=torch.uint8, device="cuda")
    rac.rac_encode(cfg, to_dev(torch, xu), to_dev(torch, ru), None, w, xh, stream=stream)
    torch.cuda.synchronize()
    ref = wl.f32_to_bf16_bits(xh.cpu().numpy())
    del xh, w, xu, ru
    torch.cuda.empty_cache()
    log("[bench] generating the prefill-downlink workload (downlink state)")
    xd = wl.prefill_downlink(ref, 0)
    return cfg, to_dev(torch, xd), to_dev(torch, ref), xd, ref


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--warm-ms", type=float, default=60.0,
                    help="after the warmup steps, keep running untimed steps for this long: the GPU clock "
                         "climbs for the first ~20 ms of sustained load")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true")
    ap.add_argument("--profile", choices=["downlink", "uplink", "long_context", "decode_step", "tiny", "predictor",
                                            "launch_shapes"],
                    help="run only this workload's back-to-back encodes and decodes and print their timings")
    ap.add_argument("--iters", type=int, default=20, help="back-to-back launches per kernel in --profile runs")
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
    stream = torch.cuda.current_stream()
    if args.profile:
        print(json.dumps(profile_run(torch, rac, wl, stream, args.profile, args.iters)), flush=True)
        return

    cfg, x0, r0, xd_bits, ref_bits = downlink_workload(torch, rac, wl, stream)
    T, d = cfg.tokens, cfg.hidden
    C = Codec(torch, rac, cfg, x0, r0, 3, stream)

    # one step: encode batch i into set i % 3, decode the batch of step i - 1.
    # With three sets no launch reads what the launch before it touched: the
    # decode of set i - 1 follows the encode of set i, and the next encode
    # (set i + 1) follows the decode of set i - 1.
    def step(i):
        C.enc(i)
        C.dec(i - 1)

    log(f"[bench] warmup {args.warmup} steps, then {args.warm_ms:g} ms")
    C.enc(-1)  # the first step decodes the other set
    for i in range(max(args.warmup, 2)):
        step(i)
    torch.cuda.synchronize()
    t_warm, i = time.perf_counter(), 0
    while (time.perf_counter() - t_warm) * 1e3 < args.warm_ms:
        for _ in range(4):
            step(i)
            i += 1
        torch.cuda.synchronize()
    # The timed steps, back to back on one stream; HIP events on that stream
    # bracket every encode, which gives the dominant kernel's launch time.
    log(f"[bench] timing {args.steps} steps")
    ea = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    eb = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(args.steps):
        ea[i].record(stream)
        C.enc(i)
        eb[i].record(stream)
        C.dec(i - 1)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    gpu_ms_per_step = e0.elapsed_time(e1) / args.steps
    enc_us = float(np.mean([a.elapsed_time(b) for a, b in zip(ea, eb)])) * 1e3
    act_bytes = T * d * 2
    value = act_bytes / (ms_per_step * 1e-3) / 1e9
    # sender and receiver agree on the last batch decoded in the timed steps
    s = C.sets[(args.steps - 2) % 3]
    assert torch.equal(s["xhat"], s["xdec"]), "sender and receiver reconstructions differ"

    enc_alg = C.alg()
    achieved = enc_alg / (enc_us * 1e-6) / 1e9
    # HBM bytes per launch from the committed counter runs of this workload,
    # while they were taken on the current kernel source
    traffic = rocprof_summary.block_traffic(TRAFFIC_FILE, "downlink_65536x3584_g128_b4_k4 encode")
    traffic = round(traffic) if traffic is not None else None
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
        "config": {"workload": "prefill downlink reuse, Qwen2-7B-shaped: x,ref bf16 8 x 8192 = 65536 tokens x "
                               "3584 hidden, group 128, 4-bit, top-4 outliers/token, ref = bf16 sender "
                               "reconstruction of a synthetic uplink; step = rac_encode of one batch (fused fp32 "
                               "sender reconstruction) + rac_decode of the previous step's batch",
                   "tokens": T, "hidden": d, "group": 128, "bits": 4, "outlier_k": 4,
                   "wire_bytes": C.wbytes, "buffer_sets": 3},
        "roofline": {"kernel": HEADLINE_KERNEL, "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": enc_alg,
                     "avg_launch_us": round(enc_us, 3)},
    }
    log(f"[bench] step {ms_per_step * 1e3:.1f} us, encode {enc_us:.1f} us ({achieved / HBM_PEAK_GBPS:.4f})")
    extras = {"gpu_ms_per_step": round(gpu_ms_per_step, 5), "decode_kernel": "rac_decode_kernel<4, 1, false>"}
    if not args.no_extras:
        # (after the timed steps, so that without extras the last launches of
        # the encode kernel in a kernel trace are those of the timed steps)
        C.warm()
        e_us, d_us = C.steady(args.steps)
        extras["launch_shapes"] = launch_shape_rates(torch, rac, C, args.steps)
        extras.update({"encode_us_back_to_back": round(e_us, 2),
                       "encode_hbm_frac_back_to_back": frac(enc_alg, e_us),
                       "decode_us_back_to_back": round(d_us, 2),
                       "decode_hbm_frac_back_to_back": frac(C.alg(False), d_us)})
    C.free()
    del C, x0, r0
    torch.cuda.empty_cache()
    if not args.no_extras:
        extras.update(all_extras(torch, rac, wl, stream))
    out["extras"] = extras
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(xd_bits, ref_bits, cfg)
    print(json.dumps(out), flush=True)


def prefill_uplink(torch, rac, wl, stream):
    """The 4096 x 4096 uplink on rotating buffer sets: enough of them that a
    pass of decodes (each reading its wire and reference) and a pass of
    encodes (each reading x and the reference) read at least twice the
    256 MiB last-level cache, so no set is still cached when it comes round
    again (the reconstruction stores are non-temporal and do not evict it)."""
    T, d = 4096, 4096
    cfg = rac.RacConfig(T, d, 128, 128, 4, 8)
    xb, rb, _ = wl.prefill_uplink(0)
    dec_read = T * d * 2 + rac.rac_wire_size(cfg)
    nsets = max(2, int(np.ceil(2 * LLC_BYTES / dec_read)))
    return Codec(torch, rac, cfg, to_dev(torch, xb), to_dev(torch, rb), nsets, stream), rb


def copy_reference(torch, stream, nbytes=1 << 30, iters=10, reps=5):
    """What the memory system gives a plain copy: a 1 GiB device-to-device
    copy (the HIP runtime's copy kernel, through torch), timed back to back;
    bytes moved = read + write.  The median of `reps` blocks."""
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(iters):
            dst.copy_(src)
        ev[1].record(stream)
        torch.cuda.synchronize()
        times.append(ev[0].elapsed_time(ev[1]) / iters * 1e3)
    us = float(np.median(times))
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes_per_copy": 2 * nbytes, "us": round(us, 1), "GBps": round(2 * nbytes / us / 1e3, 1),
            "hbm_frac": frac(2 * nbytes, us)}


def all_extras(torch, rac, wl, stream):
    ex = {}
    ex["copy_reference_1GiB"] = copy_reference(torch, stream)
    log(f"[bench] device copy: {ex['copy_reference_1GiB']}")
    log("[bench] prefill uplink 4096 x 4096")
    U, rb = prefill_uplink(torch, rac, wl, stream)
    U.warm()
    e, dcd = U.steady(50)
    ex["prefill_uplink_4096x4096_g128_b4_k8"] = {
        "encode_us": round(e, 2), "encode_hbm_frac": frac(U.alg(), e),
        "decode_us": round(dcd, 2), "decode_hbm_frac": frac(U.alg(False), dcd),
        "wire_over_bf16": round(U.wbytes / (4096 * 4096 * 2), 4),
        "encode_kernel": "rac_encode_rows_kernel<4, 4, 4, 4, 2, false, false, false>"}
    log(f"[bench] uplink: {ex['prefill_uplink_4096x4096_g128_b4_k8']}")
    ex["launch_shapes_4096x4096_g128_b4_k8"] = launch_shape_rates(torch, rac, U, 50)
    ex["outlier_modes_4096x4096_g128_b4"] = outlier_mode_rates(torch, rac, U, 50)
    ex["gathered_reference"] = gather_rates(torch, rac, U, 50)
    ex["pooled_fit"] = pooled_rates(torch, rac, U, 50)
    ex["span_selection"] = span_selection_cost(rac, 4096)
    ex["calibration"] = calibration_rates(torch, rac, wl, U)
    U.free()
    del U
    ex["long_context_32768x4096_k16"] = long_context_rates(torch, rac, wl, stream)
    ex["tiny_64x512_g64_b4"] = tiny_rates(torch, rac, wl, stream)
    ex["decode_step"] = decode_step_latency(torch, rac, wl, stream)
    ex["decode_predictor"] = predictor_latency(torch, rac, wl, stream)
    # graph-replayed encode + decode pair, µs, across the bit widths and with
    # one scale per token row (quantization group = hidden)
    ex["decode_step_graph_pair_us"] = {
        f"b{bits}_gq{gq}": decode_step_latency(torch, rac, wl, stream, bits, gq, detail=False)
        for bits, gq in ((2, 128), (8, 128), (4, 4096))}
    return ex


def long_context_rates(torch, rac, wl, stream, iters=20):
    """32768 x 4096 at groups 64 and 128 and 2/3/4/8 bits, k = 16, each on
    its own data: encode, decode (back to back over two sets, each far above
    the last-level cache) and the encode + decode round trip on one stream."""
    out = {}
    T, d = 32768, 4096
    for g in (64, 128):
        log(f"[bench] generating the long-context workload, group {g}")
        xb, rb, _ = wl.long_context(0, group=g)
        x, r = to_dev(torch, xb), to_dev(torch, rb)
        for bits in (2, 3, 4, 8):
            cfg = rac.RacConfig(T, d, g, g, bits, 16)
            C = Codec(torch, rac, cfg, x, r, 2, stream)
            C.warm()
            e, dcd = C.steady(iters)
            rt = C.round_trip(iters)
            res = {"encode_us": round(e, 2), "encode_hbm_frac": frac(C.alg(), e),
                   "decode_us": round(dcd, 2), "decode_hbm_frac": frac(C.alg(False), dcd),
                   "round_trip_us": round(rt, 2), "activation_GBps_round_trip": round(T * d * 2 / rt / 1e3, 1),
                   "wire_over_bf16": round(C.wbytes / (T * d * 2), 4)}
            out[f"g{g}_b{bits}"] = res
            log(f"[bench] long context g{g} b{bits}: {res}")
            C.free()
            del C
        del x, r
        torch.cuda.empty_cache()
    return out


def tiny_rates(torch, rac, wl, stream, iters=200):
    """64 x 512, group 64, 4-bit: launch-bound, µs per call only (64 sets)."""
    xb, rb, _ = wl.tiny(0)
    C = Codec(torch, rac, rac.RacConfig(64, 512, 64, 64, 4, 0), to_dev(torch, xb), to_dev(torch, rb), 64, stream)
    C.warm()
    e, dcd = C.steady(iters)
    C.free()
    return {"encode_us": round(e, 2), "decode_us": round(dcd, 2)}


def outlier_mode_rates(torch, rac, U, steps):
    """Average launch time (HIP events around `steps` back-to-back launches
    over the rotating buffer sets) of rac_encode and of rac_decode on the
    uplink inputs with other outlier settings: k = 16, 32, 64 per token,
    k_g = 1, 2, 4 outliers per quantization group (u8 offsets), and none.  Each entry gives µs, the
    fraction of 8 TB/s by algorithmic bytes, and the wire size relative to
    the bf16 tensor."""
    res = {}
    variants = {"none": (0, 0), "per_token_k16": (16, 0), "per_token_k32": (32, 0), "per_token_k64": (64, 0),
                "per_group_kg1": (1, rac.RAC_FLAG_GROUP_OUTLIERS),
                "per_group_kg2": (2, rac.RAC_FLAG_GROUP_OUTLIERS),
                "per_group_kg4": (4, rac.RAC_FLAG_GROUP_OUTLIERS)}
    T, d = 4096, 4096
    sets, nsets, stream = U.sets, U.n, U.stream
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
                     "encode_hbm_frac": frac(algorithmic_bytes(T, d, wb), e_us),
                     "decode_us": round(d_us, 2),
                     "decode_hbm_frac": frac(algorithmic_bytes(T, d, wb, encode=False), d_us),
                     "wire_over_bf16": round(wb / (T * d * 2), 4)}
        del wires
    return res


def pooled_rates(torch, rac, U, steps, reps=5):
    """rac_encode_pooled on the uplink inputs, with segments standing for
    retrieved spans (random lengths of 1 to 600 rows): average time of the
    whole call (its three launches) over `steps` back-to-back calls (the
    median of `reps` such timings), and the fraction of 8 TB/s by the
    per-token encode's algorithmic bytes and by the pooled call's own (the
    moments pass reads x and ref a second time)."""
    cfg, sets, nsets, stream = U.cfg, U.sets, U.n, U.stream
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
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        ev[0].record(stream)
        for i in range(steps):
            enc(i)
        ev[1].record(stream)
        torch.cuda.synchronize()
        times.append(ev[0].elapsed_time(ev[1]) / steps * 1e3)
    us = float(np.median(times))
    del wires
    own = algorithmic_bytes(T, d, wb) + T * d * 4
    return {"segments": int(seg.numel()) - 1, "encode_us": round(us, 2),
            "hbm_frac_by_encode_bytes": frac(algorithmic_bytes(T, d, wb), us),
            "hbm_frac_by_own_bytes": frac(own, us)}


def calibration_rates(torch, rac, wl, U, steps=20):
    """The offline calibration's two costs.  rac_recon_error over the
    uplink's 4096 x 4096 reconstruction (reads x, bf16, and the fp32
    reconstruction once: 6 bytes per element), back to back over the rotating
    buffer sets; and one rac_calibrate over a grid of 108 candidates
    (g_a, g_q in {64, 128, 256}, b in {2, 3, 4, 8}, k_g in {0, 1, 2}) on 1024
    uplink rows, host time of the whole call (it synchronizes to read its
    results back)."""
    T, d = U.cfg.tokens, U.cfg.hidden
    ws = torch.empty(rac.rac_recon_error_workspace(T), dtype=torch.uint8, device="cuda")
    stats = torch.empty(3, dtype=torch.float64, device="cuda")
    for i in range(U.n):
        U.enc(i)
    for i in range(2 * U.n):
        s = U.sets[i % U.n]
        rac.rac_recon_error(T, d, s["x"], s["xhat"], stats, ws, stream=U.stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev[0].record(U.stream)
    for i in range(steps):
        s = U.sets[i % U.n]
        rac.rac_recon_error(T, d, s["x"], s["xhat"], stats, ws, stream=U.stream)
    ev[1].record(U.stream)
    torch.cuda.synchronize()
    err_us = ev[0].elapsed_time(ev[1]) / steps * 1e3
    n = 1024
    xs, rs = U.sets[0]["x"][:n].contiguous(), U.sets[0]["ref"][:n].contiguous()
    grp = rac.RAC_FLAG_GROUP_OUTLIERS
    configs = [rac.RacConfig(n, d, ga, gq, b, kg, grp if kg else 0)
               for ga in (64, 128, 256) for gq in (64, 128, 256) for b in (2, 3, 4, 8) for kg in (0, 1, 2)]
    wsc = torch.empty(rac.rac_calibrate_workspace(configs), dtype=torch.uint8, device="cuda")
    rac.rac_calibrate(xs, rs, configs, 1e-3, workspace=wsc, stream=U.stream)
    times = []
    for _ in range(3):
        t0 = time.perf_counter()
        chosen, res = rac.rac_calibrate(xs, rs, configs, 1e-3, workspace=wsc, stream=U.stream)
        times.append(time.perf_counter() - t0)
    c = configs[chosen]
    return {"recon_error_4096x4096_us": round(err_us, 2),
            "recon_error_hbm_frac": frac(T * d * 6, err_us),
            "calibrate_1024x4096_108_candidates_ms": round(min(times) * 1e3, 2),
            "chosen_for_nmse_1e-3": {"g_a": c.group_align, "g_q": c.group_quant, "bits": c.bits, "k_g": c.outlier_k,
                                     "wire_bytes": res[chosen]["wire_bytes"], "nmse": res[chosen]["nmse"]}}


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


def gather_rates(torch, rac, U, steps, reps=7):
    """rac_encode_gather / rac_decode_gather on the uplink configuration,
    each row's reference read from an 8192-row bf16 store of earlier rows
    (one store per buffer set), for two index patterns: span runs (what
    repeated-span retrieval hands over: spans of 32 to 512 tokens, each read
    from consecutive store rows at a disjoint random place) and random rows
    (every row at a random store row: the worst case for locality).  The
    workload's rows without a reference name no row (a zero reference), the
    others a store row holding their own reference, so the codec sees the
    materialized call's data.  Average launch time over `steps` back-to-back
    launches, for the materialized calls on the same inputs and the two
    patterns in turn, `reps` times over; each figure is the median of its
    repetitions (the clock drifts under sustained load, so a single timing
    of each, taken one after the other, would mostly measure that drift)."""
    cfg, sets, nsets, stream = U.cfg, U.sets, U.n, U.stream
    T, d = cfg.tokens, cfg.hidden
    # the rows without a reference (ref = 0 in the workload, a fifth of
    # them) name no store row; every other row names one holding its own
    # reference, so the data are those of the materialized call
    miss = (sets[0]["ref"] == 0).all(dim=1).cpu().numpy()
    rng = np.random.default_rng(11)
    rand = rng.permutation(2 * T)[:T].astype(np.int32)
    # spans of 32 to 512 tokens, each read from a contiguous store region;
    # the regions are disjoint, in random order with random gaps
    lens = []
    while sum(lens) < T:
        lens.append(min(int(rng.integers(32, 513)), T - sum(lens)))
    order = rng.permutation(len(lens))
    gaps = rng.multinomial(T, np.ones(len(lens) + 1) / (len(lens) + 1))
    place, at = {}, 0
    for k, g in zip(order, gaps):
        at += int(g)
        place[int(k)] = at
        at += lens[k]
    runs = np.concatenate([np.arange(place[k], place[k] + n) for k, n in enumerate(lens)]).astype(np.int32)
    assert runs.size == T and np.unique(runs).size == T and runs.max() < 2 * T
    rand[miss], runs[miss] = -1, -1
    wb = rac.rac_wire_size(cfg)
    wires = [torch.empty(wb, dtype=torch.uint8, device="cuda") for _ in range(nsets)]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]

    def timed(enc, dec):
        for i in range(nsets):
            enc(i)
            dec(i)
        torch.cuda.synchronize()
        ev[0].record(stream)
        for i in range(steps):
            enc(i)
        ev[1].record(stream)
        for i in range(steps):
            dec(i)
        ev[2].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps * 1e3, ev[1].elapsed_time(ev[2]) / steps * 1e3

    def gathered(pos):
        idx = torch.from_numpy(pos).cuda()
        ok = idx >= 0
        stores = []
        for i in range(nsets):
            st = torch.zeros(2 * T, d, dtype=torch.int16, device="cuda")
            st[idx[ok].long()] = sets[i]["ref"][ok]
            stores.append(st)

        def enc(i):
            s = sets[i % nsets]
            rac.rac_encode_gather(cfg, s["x"], stores[i % nsets], idx, None, wires[i % nsets], s["xhat"],
                                  stream=stream)

        def dec(i):
            s = sets[i % nsets]
            rac.rac_decode_gather(cfg, wires[i % nsets], stores[i % nsets], idx, None, s["xdec"], stream=stream)
        return enc, dec

    calls = {"materialized": (U.enc, U.dec), "span_runs": gathered(runs), "random_rows": gathered(rand)}
    times = {name: [] for name in calls}
    for _ in range(reps):
        for name, (enc, dec) in calls.items():
            times[name].append(timed(enc, dec))
            if name != "materialized":
                assert torch.equal(sets[0]["xhat"], sets[0]["xdec"])
    out = {"store_rows": 2 * T, "repetitions": reps}
    for name, tv in times.items():
        a = np.asarray(tv)
        out[name] = {"encode_us": round(float(np.median(a[:, 0])), 2),
                     "decode_us": round(float(np.median(a[:, 1])), 2)}
        if name != "materialized":
            out[name]["miss_fraction"] = round(float(((runs if name == "span_runs" else rand) < 0).mean()), 4)
    del calls, wires
    return out


def decode_step_latency(torch, rac, wl, stream, bits=4, gq=128, detail=True):
    """µs per call of rac_encode and rac_decode for decode-phase batches
    (1 token per sequence, 4096 hidden, alignment group 128, quantization
    group gq, no outliers): wall time per call with back-to-back launches,
    per-call HIP-event time (with detail; events add their own dispatch
    overhead, the rocprofv3 kernel trace under profiles/ gives kernel-only
    time per batch), and the time per encode + decode pair when 20 pairs are
    captured in one HIP graph and replayed."""
    res = {}
    for B in (1, 16, 64, 256):
        cfg = rac.RacConfig(B, 4096, 128, gq, bits, 0)
        xb, rb = wl.decode_step(B)
        x, ref = to_dev(torch, xb), to_dev(torch, rb)
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


def profile_run(torch, rac, wl, stream, workload, iters):
    """One workload alone, for rocprofv3: warm, then `iters` back-to-back
    encodes and `iters` back-to-back decodes over rotating buffer sets, per
    configuration of the workload.  Returns the event timings."""
    out = {"profile": workload, "iters": iters}
    if workload == "downlink":
        cfg, x, r, _, _ = downlink_workload(torch, rac, wl, stream)
        C = Codec(torch, rac, cfg, x, r, 3, stream)
        C.warm()
        e, dcd = C.back_to_back(iters)
        out["downlink_65536x3584_g128_b4_k4"] = {"encode_us": round(e, 2), "encode_hbm_frac": frac(C.alg(), e),
                                                 "decode_us": round(dcd, 2),
                                                 "decode_hbm_frac": frac(C.alg(False), dcd),
                                                 "encode_alg_bytes": C.alg(), "decode_alg_bytes": C.alg(False)}
    elif workload == "uplink":
        U, _ = prefill_uplink(torch, rac, wl, stream)
        U.warm()
        e, dcd = U.back_to_back(iters)
        out["uplink_4096x4096_g128_b4_k8"] = {"encode_us": round(e, 2), "encode_hbm_frac": frac(U.alg(), e),
                                              "decode_us": round(dcd, 2), "decode_hbm_frac": frac(U.alg(False), dcd),
                                              "encode_alg_bytes": U.alg(), "decode_alg_bytes": U.alg(False)}
    elif workload == "long_context":
        out.update(long_context_rates(torch, rac, wl, stream, iters))
    elif workload == "tiny":
        out.update(tiny_rates(torch, rac, wl, stream, iters))
    elif workload == "predictor":
        out.update(predictor_latency(torch, rac, wl, stream, iters=iters))
    elif workload == "launch_shapes":
        out["reps"] = SHAPE_REPS
        out.update(launch_shape_sweep(torch, rac, stream, iters))
    else:
        for bits, gq in ((2, 128), (4, 128), (8, 128), (4, 4096)):
            for B, v in decode_step_latency(torch, rac, wl, stream, bits, gq, detail=True).items():
                out[f"b{bits}_gq{gq}_{B}"] = v
    log(f"[bench] profile {workload} done")
    return out


def predictor_latency(torch, rac, wl, stream, batches=(1, 16, 64, 256), iters=50):
    """Decode-phase reference predictor (one-layer causal Transformer, width
    512, 8 heads, SwiGLU 2048, window 64, on 4096-wide boundary states):
    microseconds per step with back-to-back launches (HIP events) and per
    step replayed from a HIP graph of 20 steps; the weight stream (bytes per
    step / time) and the matrix-core rate (2 * batch * parameters / time)."""
    cfg = rac.PredictorConfig(4096, 512, 8, 2048, 64, 256)
    weights = wl.predictor_weights(cfg.hidden, cfg.model, cfg.ffn, 0)
    blob = torch.from_numpy(rac.predictor_pack(cfg, weights)).cuda()
    params = sum(int(v.size) for v in weights.values())
    cache = torch.zeros(rac.rac_predictor_cache_bytes(cfg) // 2, dtype=torch.int16, device="cuda")
    ws = torch.empty(rac.rac_predictor_workspace_bytes(cfg), dtype=torch.uint8, device="cuda")
    out = {"config": "hidden 4096, model 512, 8 heads, ffn 2048, window 64", "weight_bytes": params * 2}
    for B in batches:
        x = torch.from_numpy(wl.decode_sequence(B, 1, 0)[0].view(np.int16)).cuda()
        r = torch.empty_like(x)
        pos = torch.arange(B, dtype=torch.int32, device="cuda") % 64 + 63
        step = lambda: rac.rac_predictor_step(cfg, blob, cache, pos, x, r, ws, B, stream=stream)
        for _ in range(20):
            step()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(iters):
            step()
        ev[1].record(stream)
        torch.cuda.synchronize()
        eager = ev[0].elapsed_time(ev[1]) / iters * 1e3
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(20):
                rac.rac_predictor_step(cfg, blob, cache, pos, x, r, ws, B)
        g.replay()
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(5):
            g.replay()
        ev[1].record(stream)
        torch.cuda.synchronize()
        graph = ev[0].elapsed_time(ev[1]) * 1e3 / 100
        out[f"B{B}"] = {"eager_us_per_step": round(eager, 2), "graph_us_per_step": round(graph, 2),
                        "weight_GBps_graph": round(params * 2 / graph / 1e3, 1),
                        "mfma_TFLOPs_graph": round(2 * B * params / graph / 1e6, 2)}
        log(f"[bench] predictor B{B}: {out[f'B{B}']}")
    return out


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(xb, rb, cfg, rows=1024, min_s=10.0, max_s=30.0):
    """The CPU oracle on a sample of the headline workload: its first `rows`
    token rows (encode with sender reconstruction, then decode), repeated
    until at least `min_s` seconds have passed, on one thread pinned to one
    core (the calling thread's affinity is restored afterwards)."""
    import oracle
    c = dict(tokens=rows, hidden=cfg.hidden, group_align=cfg.group_align,
             group_quant=cfg.group_quant, bits=cfg.bits, outlier_k=cfg.outlier_k, flags=cfg.flags)
    xs, rs = np.ascontiguousarray(xb[:rows]), np.ascontiguousarray(rb[:rows])
    allowed = os.sched_getaffinity(0)
    core = max(allowed)
    os.sched_setaffinity(0, {core})
    log(f"[bench] CPU oracle baseline on core {core} ({rows} rows per pass)")
    try:
        reps, dt = 0, 0.0
        while dt < min_s and dt < max_s:
            t0 = time.perf_counter()
            rc, wire, _ = oracle.encode(xs, rs, **c)
            rc2, _ = oracle.decode(wire, rs, **c)
            dt += time.perf_counter() - t0
            reps += 1
            assert rc == 0 and rc2 == 0
    finally:
        os.sched_setaffinity(0, allowed)
    return {"value": round(reps * rows * cfg.hidden * 2 / dt / 1e9, 5), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{reps} passes over the first {rows} token rows of the headline workload "
                      f"({rows}x{cfg.hidden}: encode with sender reconstruction + decode), {dt:.1f} s, "
                      f"one thread pinned to core {core} of {len(allowed)} allowed ({os.cpu_count()} visible)",
            "cpu_model": cpu_model()}


if __name__ == "__main__":
    main()
