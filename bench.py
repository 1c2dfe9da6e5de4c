#!/usr/bin/env python3
"""Decode-step benchmark on one MI355X.

One step = one decode step of the whole model (embedding, all decoder layers,
final norm + LM head) for every sequence of the batch, on seeded synthetic
weights and KV cache already resident in HBM.  The headline is the looped
(kernel-looping) schedule; the per-layer schedule is timed beside it.

Prints ONE JSON line with tokens/s, step latency, achieved HBM bandwidth of
the step kernel (algorithmic bytes / mean launch duration, HIP events on the
launch stream) against the 8 TB/s peak, and the CPU oracle timed on a
bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tok/s + achieved HBM TB/s vs peak, 8B-shape batch 1 ctx 4096"
PEAK_HBM_GBS = 8000.0
# Measured HBM traffic of the step kernel (rocprofv3 FETCH_SIZE / WRITE_SIZE,
# scaled by a plain copy kernel), with the hash of the device source it was
# taken on: reported only while that source is unchanged.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "kl_step_kernel_traffic.md")
CSRC = os.path.join(ROOT, "paper_2410_23668_amd", "csrc")
DEVICE_SRC = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                    if f.endswith((".hip", ".h", ".cpp")))


PEAK_BF16_FLOPS = 2.5e15   # dense bf16 matrix-core peak of MI355X


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def device_source_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in DEVICE_SRC:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """Bytes per launch from the committed counter summary, or None when it
    is missing, for another workload, or taken on other device code."""
    try:
        with open(TRAFFIC_FILE) as fh:
            text = fh.read()
        t = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    except (OSError, ValueError, IndexError):
        return None
    w = t.get("workloads", {}).get(workload)
    if not w or t.get("device_source_sha256") != device_source_sha():
        return None
    return w["fetch_bytes"] + w["write_bytes"]


def copy_probe(mib: int, reps: int = 3):
    """Plain copy kernel of known size for scaling the HBM counters: reads and
    writes mib MiB per launch (torch's elementwise negation, fp32)."""
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(reps):
        torch.neg(x, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe": {"read_bytes": 4 * n, "write_bytes": 4 * n, "launches": reps,
                                     "kernel": "torch.neg fp32 (elementwise)"}}), flush=True)


def read_stream_ceiling(gib: int = 4, reps: int = 5):
    """GB/s of kl_read_stream (the step kernel's load pattern, one pass over a
    buffer) for a few grid sizes: the practical read ceiling, for context."""
    import torch
    from paper_2410_23668_amd import binding as kb
    from paper_2410_23668_amd.device import stream_handle
    n = gib << 30
    buf = torch.zeros(n, dtype=torch.uint8, device="cuda")
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    h = stream_handle()
    rates = {}
    for wg in (256, 512, 1024, 2048, 4096):
        kb.kl_read_stream(buf.data_ptr(), n, wg, out.data_ptr(), h)   # warm-up
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            kb.kl_read_stream(buf.data_ptr(), n, wg, out.data_ptr(), h)
        e1.record()
        torch.cuda.synchronize()
        rates[wg] = n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del buf, out
    best = max(rates, key=rates.get)
    return {"bytes": n, "GBps_by_workgroups": {str(k): round(v, 1) for k, v in rates.items()},
            "best_GBps": rates[best], "best_frac_of_peak": rates[best] / PEAK_HBM_GBS,
            "step_grid_GBps": rates[256],
            "kernel": "kl_read_stream: 16-byte non-temporal loads, 16 in flight per lane, 512 "
                      "lanes per workgroup"}


PHASES = ("qkv", "attn", "oproj", "gateup", "down")


def phase_table(model, toks, pos, kv, logits, mode, cfg, B, P):
    """One traced step (kl_set_trace): per phase, the mean over layers of the
    span from the previous phase's last finishing workgroup to this phase's
    last finishing workgroup, with the phase's algorithmic bytes and the rate
    they imply.  The spans of all phases add up to the traced step."""
    import numpy as np
    import torch
    from paper_2410_23668_amd import binding as kb
    from paper_2410_23668_amd import bytemodel
    L = cfg["n_layers"]
    nwg = model.info().n_workgroups
    nph = 5 * L + 2     # embed, 5 per layer, head
    tr = torch.zeros(nph * nwg * 4, dtype=torch.int64, device="cuda")
    kb.kl_set_trace(model.state, tr.data_ptr(), nph)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    model.step(toks, pos, kv, logits, None, mode)
    e1.record()
    torch.cuda.synchronize()
    kb.kl_set_trace(model.state, None, 0)
    traced_ms = e0.elapsed_time(e1)
    a = tr.cpu().numpy().reshape(nph, nwg, 4) * 10      # 100 MHz ticks -> ns
    end = a[:, :, 0]
    last = [int(end[i][end[i] > 0].max()) for i in range(nph)]
    first = int(end[0][end[0] > 0].min())
    nb = bytemodel.phase_bytes(cfg, B, P)
    rows = {}
    for k, name in enumerate(PHASES):
        spans = [last[1 + 5 * l + k] - last[5 * l + k] for l in range(L)]
        rows[name] = float(np.mean(spans)) / 1e3
    rows["head"] = (last[nph - 1] - last[nph - 2]) / 1e3
    table = {}
    for name, us in rows.items():
        table[name] = {"us": round(us, 2), "bytes": nb[name],
                       "GBps": round(nb[name] / (us * 1e-6) / 1e9, 1),
                       "frac_of_peak": round(nb[name] / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 3)}
    layer_us = sum(rows[n] for n in PHASES)
    return {"per_layer_phase_mean": table, "layer_us": round(layer_us, 2),
            "embed_us": round((last[0] - first) / 1e3, 2),
            "traced_span_us": round((last[-1] - first) / 1e3, 1),
            "traced_step_ms": traced_ms,
            "note": "span of a phase = its last workgroup's end minus the previous phase's "
                    "(s_memrealtime stamps); bytes = the phase's algorithmic bytes"}


def time_mode(model, toks, pos, kv, logits, mode, steps, warmup):
    import torch
    for _ in range(warmup):
        model.step(toks, pos, kv, logits, None, mode)
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        starts[i].record()
        model.step(toks, pos, kv, logits, None, mode)
        ends[i].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = sorted(s.elapsed_time(e) for s, e in zip(starts, ends))   # ms
    mean = sum(per) / len(per)
    return dict(mean_ms=mean, median_ms=per[len(per) // 2], p10_ms=per[len(per) // 10],
                p90_ms=per[(9 * len(per)) // 10], wall_ms_per_step=1e3 * wall / steps)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama8b-b1-ctx4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--modes", default="looped,per_layer,per_layer_graph",
                    help="schedules to time; the first is the headline")
    ap.add_argument("--threads", type=int, default=0, help="host threads for input generation")
    ap.add_argument("--loop-tokens", type=int, default=-1,
                    help="tokens of the greedy token loop timed after the steps (its steady-state "
                         "time per output token); -1: 128 unless the model is loaded layer by "
                         "layer, 0: skip")
    ap.add_argument("--phases", action="store_true",
                    help="trace one step of the headline schedule and report per-phase times")
    ap.add_argument("--no-read-stream", action="store_true",
                    help="skip the read-stream ceiling measurement")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run the copy kernel used to scale HBM counters, then exit")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_probe_mib:
        torch.cuda.set_device(0)
        copy_probe(args.copy_probe_mib)
        return

    import synth
    from paper_2410_23668_amd import binding as kb
    from paper_2410_23668_amd import bytemodel
    from paper_2410_23668_amd.device import GpuModel, KvCache
    from synth.workloads import WORKLOADS

    wl = WORKLOADS[args.workload]
    cfg, B, P, cap = wl["model"], wl["batch"], wl["context"], wl["capacity"]
    nthr = args.threads or synth.default_threads()
    torch.cuda.set_device(0)

    t = time.perf_counter()
    # models whose weights would not fit twice in device memory (the 70B
    # shape) are generated and loaded one layer at a time
    big = bytemodel.step_bytes(cfg, 1, 0) > 40e9
    # the token loop (below) needs room for its tokens: the model's positions
    # reach that far
    n_loop = args.loop_tokens if args.loop_tokens >= 0 else (0 if big else 128)
    cap_loop = (P + n_loop + 63) // 64 * 64
    max_seq = max(cap, cap_loop)
    weights = None
    data = "synthetic (seeded N(0,0.02) weights, N(0,1) KV)"
    if big:
        # generated on the device with torch's seeded normal generator (the
        # host generator's distributions, not its values: decode cost does not
        # depend on them), loaded one layer at a time
        log(f"workload {args.workload}: generating on the device, loading layer by layer")
        data = ("synthetic, generated on the device (torch seeded normal: N(0,0.02) weights, "
                "N(1,0.01) norm gains, N(0,1) KV)")
        gen = torch.Generator(device="cuda")
        gen.manual_seed(wl["seed_weights"])

        def dev_normal(shape, mean, std):
            x = torch.empty(shape, dtype=torch.float32, device="cuda")
            x.normal_(mean, std, generator=gen)
            return x.to(torch.bfloat16).view(torch.int16)

        def dev_tensor(name, shape):
            if name.endswith("norm"):
                return dev_normal(shape, 1.0, synth.NORM_STD)
            if name in synth.BIAS_KIND:
                return dev_normal(shape, 0.0, synth.BIAS_STD)
            return dev_normal(shape, 0.0, synth.WEIGHT_STD)

        def layer(l):
            if l % 8 == 0:
                log(f"  layer {l}/{cfg['n_layers']} ({time.perf_counter() - t:.0f}s)")
            shapes = synth.layer_shapes(cfg)
            return {k: dev_tensor(k, shapes[k]) for k in synth.layer_names(cfg)}

        def globals_():
            g = {k: dev_tensor(k, v) for k, v in synth.global_shapes(cfg).items()}
            if cfg.get("tie_embeddings"):
                g["lm_head"] = g["embed"]
            return g

        model = GpuModel.from_layers(cfg, layer, globals_, B, max_seq)
    else:
        log(f"workload {args.workload}: generating weights ({nthr} threads)")
        weights = synth.model_host(cfg, wl["seed_weights"], nthr)
    tokens = synth.tokens(cfg, wl["seed_tokens"], B)
    if big:
        kv = KvCache(cfg, B, cap)
        gen.manual_seed(wl["seed_kv"])
        for l in range(cfg["n_layers"]):
            for b in range(B):
                kv.k[l, b, :, :P].copy_(dev_normal(kv.k[l, b, :, :P].shape, 0.0, 1.0))
                kv.v[l, b, :, :P].copy_(dev_normal(kv.v[l, b, :, :P].shape, 0.0, 1.0))
        K0 = V0 = None
        log(f"inputs ready in {time.perf_counter() - t:.1f}s")
    else:
        K0, V0 = synth.kv_cache_host(cfg, wl["seed_kv"], B, cap, [P] * B, nthr)
        log(f"inputs ready in {time.perf_counter() - t:.1f}s; loading model")
        model = GpuModel(cfg, weights, B, max_seq)
        kv = KvCache(cfg, B, cap, k_host=K0, v_host=V0)
    toks = torch.from_numpy(tokens).cuda()
    pos = torch.full((B,), P, dtype=torch.int32, device="cuda")
    info = model.info()

    modes = [m.strip() for m in args.modes.split(",") if m.strip()]
    res = {}
    outs = {}   # each schedule writes logits of its own
    for m in modes:
        outs[m] = torch.full((B, cfg["vocab"]), float("nan"), dtype=torch.float32, device="cuda")
        log(f"timing mode {m}: {args.warmup} warmup + {args.steps} steps")
        res[m] = time_mode(model, toks, pos, kv, outs[m], kb.MODES[m], args.steps, args.warmup)
        log(f"  {m}: mean {res[m]['mean_ms']:.3f} ms/step")
    err = model.device_error()
    if err:
        log(f"device error word {err:#x}")
        sys.exit(1)

    head = modes[0]
    step_ms = res[head]["mean_ms"]
    nbytes = bytemodel.step_bytes(cfg, B, P)
    achieved = nbytes / (step_ms * 1e-3) / 1e9      # GB/s
    out = {
        "metric": METRIC,
        "value": B / (step_ms * 1e-3),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "accum_dtype": "f32",
        "data": data,
        "config": {"workload": args.workload, "batch": B, "context": P, "mode": head},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS,
                     "traffic": measured_traffic(args.workload) if head == "looped" else None,
                     "algorithmic_bytes_per_launch": nbytes,
                     "kernel": "kl_step_kernel (one launch per step)"},
        "modes": {m: r for m, r in res.items()},
        "dispatches_per_step": {"looped": 1, "per_layer": cfg["n_layers"] + 2,
                                "per_op": 5 * cfg["n_layers"] + 2,
                                "per_layer_graph": cfg["n_layers"] + 2},
        "grid": {"workgroups": info.n_workgroups, "threads": info.threads_per_group,
                 "lds_bytes": info.lds_bytes},
    }
    if "per_layer" in res and head != "per_layer":
        out["speedup_vs_per_layer"] = res["per_layer"]["mean_ms"] / step_ms
    # the greedy token loop (sampling fused into the LM head, each token fed to
    # the next step on the device): steady-state time per output token over
    # n tokens, in a cache with room for them
    if n_loop > 0:
        log(f"token loop: {n_loop} tokens from position {P} ({head})")
        K1, V1 = synth.kv_cache_host(cfg, wl["seed_kv"], B, cap_loop, [P] * B, nthr)
        kv_loop = KvCache(cfg, B, cap_loop, k_host=K1, v_host=V1)
        del K1, V1
        lg = torch.empty((B, cfg["vocab"]), dtype=torch.float32, device="cuda")
        toks_out = torch.empty((n_loop, B), dtype=torch.int32, device="cuda")
        model.greedy(toks, pos, kv_loop, n_loop, toks_out, lg, kb.MODES[head])   # warm-up
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        model.greedy(toks, pos, kv_loop, n_loop, toks_out, lg, kb.MODES[head])
        e1.record()
        torch.cuda.synchronize()
        loop_ms = e0.elapsed_time(e1)
        if model.device_error():
            log("device error in the token loop")
            sys.exit(1)
        out["token_loop"] = {"tokens": n_loop, "mode": head, "ms_per_token": loop_ms / n_loop,
                             "tok_s": B * n_loop / (loop_ms * 1e-3),
                             "context": f"{P}..{P + n_loop - 1}",
                             "first_tokens": toks_out[:4, 0].tolist()}
        del kv_loop
    # every schedule computes the same bits (the timed launches' own outputs)
    for m in modes[1:]:
        out[f"bit_exact_{head}_vs_{m}"] = bool(torch.equal(outs[head].view(torch.int32),
                                                           outs[m].view(torch.int32)))
    if B >= info.mfma_min_batch:
        # the weight products run on the matrix cores, each activation as two
        # bf16 terms (two products per weight element)
        flops = bytemodel.step_flops(cfg, B, P)
        mflops = 2 * bytemodel.weight_macs(cfg) * 2 * B
        out["mfma"] = {"algorithmic_tflops": flops / (step_ms * 1e-3) / 1e12,
                       "utilisation": flops / (step_ms * 1e-3) / PEAK_BF16_FLOPS,
                       "issued_tflops": mflops / (step_ms * 1e-3) / 1e12,
                       "issued_utilisation": mflops / (step_ms * 1e-3) / PEAK_BF16_FLOPS,
                       "peak_tflops": PEAK_BF16_FLOPS / 1e12,
                       "note": "algorithmic = 2 flops per weight MAC and sequence plus attention; "
                               "issued = the matrix-core products actually run (hi and lo "
                               "activation terms), against the dense bf16 peak"}

    if args.phases:
        log("phase timeline of one traced step")
        out["phases"] = phase_table(model, toks, pos, kv, outs[head], kb.MODES[head], cfg, B, P)

    if not args.no_read_stream:
        log("read-stream ceiling")
        out["read_stream"] = read_stream_ceiling()

    # parity of the timed output, and the oracle's own time on the host
    if not args.no_cpu_baseline and weights is not None:
        import oracle
        # a bounded sample: one sequence of the batch (sequences are independent)
        nb = 1
        log(f"oracle (1 thread) on {nb} sequence(s) of the same inputs")
        Kr, Vr = K0[:, :nb].copy(), V0[:, :nb].copy()
        t = time.perf_counter()
        ref_logits, _ = oracle.decode_step(cfg, weights, tokens[:nb], [P] * nb, Kr, Vr,
                                           nthreads=1)
        cpu_s = time.perf_counter() - t
        got = outs[head][:nb].cpu().numpy()
        out["parity_rel_l2_logits"] = max(oracle.rel_l2(got[b], ref_logits[b]) for b in range(nb))
        out["parity_elem_logits"] = max(
            float(abs(got[b] - ref_logits[b]).max() / abs(ref_logits[b]).max()) for b in range(nb))
        out["parity_of"] = f"{head} schedule, the timed launches' logits, sequence(s) 0..{nb - 1}"
        out["cpu_baseline"] = {"value": nb / cpu_s, "unit": "tok/s", "cores": 1, "kind": "oracle",
                               "nproc": os.cpu_count(), "cpu_model": cpu_model(),
                               "sample": f"one decode step of {nb} sequence(s) of "
                                         f"{args.workload} (all layers), fp64 oracle, "
                                         f"1 thread, {cpu_s:.1f} s"}
    print(json.dumps(out), flush=True)
    # release device memory before interpreter shutdown
    model.close()
    del kv, toks, pos, outs
    torch.cuda.synchronize()


if __name__ == "__main__":
    main()
