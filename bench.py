"""Benchmark of the large-beam GDN decode hot path on one MI355X.

One *step* is one pass of the whole hot path over one batch (one request
group) of synthetic input: ``onela_init`` (bind + split S_ctx), then for every
decode step t: ``onela_resolve_ancestry`` -> ``onela_append_records`` ->
``onela_decode_step``.  The default workload is 1 GDN layer, 16 heads,
d_k = d_v = 128, bf16 inputs, a 4096-token prompt, 512 beams, 4 decode steps,
Zipf(1.1) parents.

Inputs are resident in HBM when timing starts: the bench keeps ``--batches``
independent copies of every input, workspace and output, and step i uses
batch i % batches, so a batch's data was last touched far more than the
256 MiB Infinity Cache ago.  Timed steps are replayed from HIP graphs (one
captured graph per batch) so host launch cost does not pace the GPU.

Printed: one JSON line with the whole-job throughput (beam-tokens/s), the
per-kernel roofline of the decode kernel (algorithmic bytes / average kernel
duration from HIP events on the kernels' stream), the per-beam FullState GPU
baseline, and the fp64 CPU oracle timed on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def unique_record_slots(wl, t):
    """Distinct record slots read by decode step t, per request: the current
    slab (W_t slots) plus every distinct ancestral (step, slot)."""
    spec = wl.spec
    counts = []
    for r in range(spec.R):
        uniq = spec.widths[t]
        if t > 0:
            # ancestral slots by pointer chasing
            cur = np.arange(spec.widths[t])
            for s in range(t, 0, -1):
                cur = wl.steps[s].parents[r][cur]
                uniq += len(np.unique(cur))
        counts.append(uniq)
    return counts


def decode_alg_bytes(wl, t):
    """Algorithmic HBM bytes of one decode launch at step t: split S_ctx once,
    q, o, the unique records referenced and the ancestry indices."""
    s = wl.spec
    io = 2 if s.io_dtype == "bf16" else 4
    W = s.widths[t]
    rec = s.HK * s.dk * io + s.HV * (s.dv * io + 8)  # one slot, all heads
    b = s.R * s.HV * s.dv * s.dk * 4          # S_ctx hi + lo bf16
    b += s.R * W * s.HK * s.dk * io           # q
    b += s.R * W * s.HV * s.dv * 4            # o (fp32)
    b += sum(unique_record_slots(wl, t)) * rec
    b += s.R * W * t * 4                      # h_t
    return b


def step_alg_bytes(wl):
    """Algorithmic bytes of one whole step: split (read fp32 S, write hi/lo),
    per t: resolve (parents + h_{t-1} rows + h_t), append (read + write one
    slab), decode."""
    s = wl.spec
    io = 2 if s.io_dtype == "bf16" else 4
    total = 2 * s.R * s.HV * s.dv * s.dk * 4
    for t, W in enumerate(s.widths):
        slab = s.R * W * (s.HK * s.dk * io + s.HV * (s.dv * io + 8))
        total += 2 * slab
        if t > 0:
            total += s.R * W * 4 + 2 * s.R * W * t * 4
        total += decode_alg_bytes(wl, t)
    return total


def cpu_baseline(wl, min_seconds):
    """The fp64 oracle (materialised per-beam states) timed on this host's
    cores over whole decodes of one request of the same workload."""
    from oracle import oracle as orc
    s = wl.spec
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    r = 0
    s0 = orc.prefill(wl.prompt_k.f64[r], wl.prompt_v.f64[r], wl.prompt_alpha.f64[r],
                     wl.prompt_beta.f64[r], nthreads=threads).astype(np.float32)
    args = (s0.astype(np.float64), [x.q.f64[r] for x in wl.steps],
            [x.k.f64[r] for x in wl.steps], [x.v.f64[r] for x in wl.steps],
            [x.alpha.f64[r] for x in wl.steps], [x.beta.f64[r] for x in wl.steps],
            [x.parents[r] for x in wl.steps[1:]])
    reps, t0 = 0, time.perf_counter()
    while True:
        orc.decode(*args, nthreads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or reps >= 200:
            break
    beam_tokens = reps * sum(s.widths)
    return {"value": beam_tokens / el, "unit": "beam-tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{reps} full {s.T}-step decodes of one request "
                      f"({s.HV} heads, {s.W} beams, S_ctx given), {el:.1f} s, "
                      f"fp64 materialised per-beam states"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--batches", type=int, default=16)
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--skip-fullstate", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    from paper_2609_12399_amd import onela as ab
    from paper_2609_12399_amd import runner
    from paper_2609_12399_amd import workload as Wm

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(3)
    ab.load_library()  # raises if libonela.so is missing: no fallback
    dev = "cuda:0"
    name = args.workload or Wm.HEADLINE
    log(f"[bench] workload {name}: generating")
    wl = Wm.make_workload(name)
    spec = wl.spec
    T = spec.T

    # ---- device data: one S_ctx from the prompt, NB copies of everything
    stream = torch.cuda.current_stream()
    dw0 = runner.to_device(wl, dev, with_prompt=True)
    s0 = runner.prefill_state(spec, dw0.prompt, dev, stream)
    torch.cuda.synchronize()
    NB = args.batches
    cfg = runner.config_for(spec)
    ws_bytes = ab.onela_workspace_bytes(cfg)
    batches = []
    for i in range(NB):
        steps = [runner.DeviceStep(st.q.clone(), st.k.clone(), st.v.clone(), st.alpha.clone(),
                                   st.beta.clone(),
                                   None if st.parents is None else st.parents.clone(),
                                   st.width) for st in dw0.steps]
        outs = [torch.empty((spec.R, st.width, spec.HV, spec.dv), dtype=torch.float32,
                            device=dev) for st in dw0.steps]
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        batches.append(dict(steps=steps, outs=outs, ws=ws, s0=s0.clone()))
    torch.cuda.synchronize()
    footprint = sum(x.numel() * x.element_size() for b in batches for x in
                    [b["ws"], b["s0"]] + b["outs"] +
                    [getattr(st, f) for st in b["steps"] for f in ("q", "k", "v", "alpha", "beta")])
    log(f"[bench] {NB} batches, {footprint / 2**20:.0f} MiB resident")

    def one_step(b, events=None):
        """init + T x (resolve, append, decode) on the current stream."""
        ctx = ab.onela_init(cfg, b["s0"], b["ws"], ws_bytes, None)
        for t, st in enumerate(b["steps"]):
            ab.onela_resolve_ancestry(ctx, t, st.width, st.parents, None)
            ab.onela_append_records(ctx, t, st.k, st.v, st.alpha, st.beta)
            if events is not None:
                events[t][0].record()
            ab.onela_decode_step(ctx, t, st.q, b["outs"][t])
            if events is not None:
                events[t][1].record()
        ab.onela_destroy(ctx)

    # ---- capture one graph per batch
    graphs = None
    if not args.no_graph:
        graphs = []
        for b in batches:
            one_step(b)  # eager once before capture
        torch.cuda.synchronize()
        for b in batches:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                one_step(b)
            graphs.append(g)
        torch.cuda.synchronize()

    def run_steps(n, start):
        for i in range(n):
            k = (start + i) % NB
            if graphs is not None:
                graphs[k].replay()
            else:
                one_step(batches[k])

    log(f"[bench] warmup {args.warmup}")
    run_steps(args.warmup, 0)
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps
    K = args.steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_host = time.perf_counter()
    e0.record()
    run_steps(K, args.warmup)
    e1.record()
    torch.cuda.synchronize()
    host_s = time.perf_counter() - t_host
    ms_total = e0.elapsed_time(e1)
    ms_per_step = ms_total / K
    beam_tokens_per_step = spec.R * sum(spec.widths)
    value = beam_tokens_per_step * K / (ms_total / 1e3)
    log(f"[bench] {K} steps: {ms_per_step * 1e3:.1f} us/step (host {host_s / K * 1e6:.1f} us/step)")

    # ---- decode-kernel roofline: events around every decode launch (eager)
    n_roof = max(K // 4, 2 * NB)
    dec_ms = np.zeros((n_roof, T))
    for i in range(n_roof):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(T)]
        one_step(batches[i % NB], ev)
        torch.cuda.synchronize()
        dec_ms[i] = [a.elapsed_time(b) for a, b in ev]
    dec_us = dec_ms[NB // 2:].mean(axis=0) * 1e3  # drop the first rotation
    bytes_t = [decode_alg_bytes(wl, t) for t in range(T)]
    achieved = sum(bytes_t) / (dec_us.sum() * 1e-6) / 1e9
    log(f"[bench] decode us per t: {np.round(dec_us, 2).tolist()}  "
        f"alg MB: {[round(b / 1e6, 2) for b in bytes_t]}  -> {achieved:.0f} GB/s")

    result = {
        "metric": "beam-tokens/s and decode-step latency (us) at 512 beams, H=16, d=128; HBM GB/s",
        "value": value,
        "unit": "beam-tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": name, "requests": spec.R, "qk_heads": spec.HK,
                   "v_heads": spec.HV, "d_k": spec.dk, "d_v": spec.dv, "prompt": spec.P,
                   "beams": spec.W, "decode_steps": T, "io_dtype": spec.io_dtype,
                   "parents": f"{spec.parents}{spec.zipf_s if spec.parents == 'zipf' else ''}",
                   "step": "init + per t (resolve_ancestry, append_records, decode_step)",
                   "contraction": "S_ctx.P on bf16 MFMA, hi/lo split, 3 products, fp32 accum",
                   "graph": graphs is not None, "batches": NB},
        "decode_step_us": {"per_t": [round(float(x), 3) for x in dec_us],
                           "mean": round(float(dec_us.mean()), 3)},
        "beam_tokens_per_step": beam_tokens_per_step,
        "step_alg_bytes": step_alg_bytes(wl),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "decode_kernel", "alg_bytes_per_t": bytes_t},
    }

    # ---- per-beam FullState GPU baseline
    if not args.skip_fullstate:
        base = runner.FullStateBaseline(spec, s0, dev)
        b0 = batches[0]
        dwb = runner.DeviceWorkload(spec, b0["steps"], None)
        base.run(dwb)
        torch.cuda.synchronize()
        reps = 5
        fe0, fe1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fe0.record()
        for _ in range(reps):
            base.run(dwb)
        fe1.record()
        torch.cuda.synchronize()
        fs_ms = fe0.elapsed_time(fe1) / reps
        result["fullstate_baseline"] = {
            "ms_per_step": fs_ms, "unit": "ms per T-step decode (all beams, all heads)",
            "beam_tokens_per_s": beam_tokens_per_step / (fs_ms / 1e3),
            "speedup_whole_step": fs_ms / ms_per_step,
            "speedup_decode_kernels": fs_ms / (dec_us.sum() / 1e3)}
        log(f"[bench] fullstate baseline {fs_ms:.3f} ms/step")
        del base

    if not args.skip_cpu:
        log("[bench] cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
