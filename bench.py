"""Benchmark of the large-beam GDN decode hot path on one MI355X.

One *step* is one pass of the whole hot path over one batch (one request
group) of synthetic input: ``onela_init`` (binds S_ctx, enqueues nothing), then for every
decode step t one ``onela_decode_step_fused`` (ancestry resolve, record append
and decode in one launch).  The same step through the three separate calls
(``onela_resolve_ancestry`` -> ``onela_append_records`` ->
``onela_decode_step``) is timed too and reported beside it.  The default workload is 1 GDN layer, 16 heads,
d_k = d_v = 128, bf16 inputs, a 4096-token prompt, 512 beams, 4 decode steps,
Zipf(1.1) parents.

Inputs are resident in HBM when timing starts: the bench keeps ``--batches``
independent copies of every input, workspace and output.  Steps run in groups
of G consecutive batches (G = the largest divisor of the timed step count K
not above ``--graph-group``), interleaved by decode step: every batch of the
group is initialised, then step t runs for every batch of the group before
step t + 1 runs for any, so a launch never directly follows the previous step
of its own batch, whose data is G - 1 launches (about G x 13 MB at the
headline) old.  Each group is one captured HIP graph, replayed whole: the
timed region is always K / G whole groups, so the figure does not depend on
K, and the graph-launch cost is paid once per G steps.

Printed: one JSON line with the whole-job throughput (beam-tokens/s), the
per-kernel roofline of the fused step kernel (algorithmic bytes / average
launch duration from HIP events around back-to-back launches on the kernels'
stream), the separate-call path, the per-beam FullState GPU baseline, and the
fp64 CPU oracle timed on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
# The sources the fused decode kernel is compiled from (its traffic profile is
# tied to their combined hash).
KERNEL_SRCS = [os.path.join(ROOT, "paper_2609_12399_amd", "csrc", f)
               for f in ("kernel_decode.hip", "device_common.h", "internal.h")]


def kernel_sources_sha256() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "decode_fused_h16_d128_w512_traffic.md")


def measured_traffic(workload: str, variant: str):
    """HBM bytes per fused launch per step t from the committed PMC summary
    (FETCH_SIZE and WRITE_SIZE runs, copy-calibrated), or None when the
    summary is missing, is for another workload or record variant, or was
    taken on a different kernel source than the one built now."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    want = kernel_sources_sha256()
    for line in open(TRAFFIC_PROFILE):
        if line.startswith("bench-traffic: "):
            rec = json.loads(line[len("bench-traffic: "):])
            if (rec.get("kernel_source_sha256") == want and rec.get("workload") == workload
                    and rec.get("variant", "inputs") == variant):
                return rec["bytes_per_t"]
    return None


SELECT_SRC = os.path.join(ROOT, "paper_2609_12399_amd", "csrc", "kernels_select.hip")
SELECT_PROFILE = os.path.join(ROOT, "profiles", "select_beams_r1_wprev512_v8192_w512_kernel_trace.md")


def measured_select_traffic(workload: str):
    """HBM bytes per selection call from the committed selection profile, or
    None when it is missing, for another shape, or taken on another source."""
    if not os.path.exists(SELECT_PROFILE):
        return None
    want = hashlib.sha256(open(SELECT_SRC, "rb").read()).hexdigest()
    for line in open(SELECT_PROFILE):
        if line.startswith("bench-select-traffic: "):
            rec = json.loads(line[len("bench-select-traffic: "):])
            if rec.get("select_source_sha256") == want and rec.get("workload") == workload:
                return rec["bytes_per_call"]
    return None


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
    """Algorithmic HBM bytes of one decode launch at step t: S_ctx (fp32) once,
    q, o, the unique records referenced and the ancestry indices."""
    s = wl.spec
    io = 2 if s.io_dtype == "bf16" else 4
    W = s.widths[t]
    rec = s.HK * s.dk * io + s.HV * (s.dv * io + 8)  # one slot, all heads
    b = s.R * s.HV * s.dv * s.dk * 4          # S_ctx fp32
    b += s.R * W * s.HK * s.dk * io           # q
    b += s.R * W * s.HV * s.dv * 4            # o (fp32)
    b += sum(unique_record_slots(wl, t)) * rec
    b += s.R * W * t * 4                      # h_t
    return b


def slab_bytes(wl, t):
    s = wl.spec
    io = 2 if s.io_dtype == "bf16" else 4
    return s.R * s.widths[t] * (s.HK * s.dk * io + s.HV * (s.dv * io + 8))


def unique_parents(wl, t):
    return sum(len(np.unique(wl.steps[t].parents[r])) for r in range(wl.spec.R)) if t else 0


def fused_alg_bytes(wl, t, borrow=False):
    """Algorithmic HBM bytes of one fused step launch at step t: the decode's
    bytes with the step-t records read from the caller instead of the arena,
    plus writing them into the arena (not with borrowed record slabs, which
    the later steps read in place), the parents, the parents' rows of h_{t-1}
    and the new h_t."""
    s = wl.spec
    W = s.widths[t]
    b = decode_alg_bytes(wl, t) - s.R * W * t * 4   # h_t is written, not read
    if not borrow:
        b += slab_bytes(wl, t)                      # arena write of the step-t records
    if t == 0:
        b += s.R * s.HV * s.dv * s.dk * 4           # S_ctx split (bf16 hi + lo) write
    if t > 0:
        b += s.R * W * 4                            # parents
        b += unique_parents(wl, t) * (t - 1) * 4    # parents' rows of h_{t-1}
        b += s.R * W * t * 4                        # h_t
    return b


def fused_alg_bytes_delta(wl, t):
    """Algorithmic HBM bytes of one fused step launch with transition records
    (alpha, delta, k): S_ctx, q, o, the step's inputs read from the caller,
    the key, gates and new delta written to the arena, the distinct ancestral
    records (key, gates, delta) and the ancestry indices."""
    s = wl.spec
    io = 2 if s.io_dtype == "bf16" else 4
    W = s.widths[t]
    rec = s.HK * s.dk * io + s.HV * (s.dv * io + 8)  # key + delta + (alpha, beta) per slot
    b = s.R * s.HV * s.dv * s.dk * 4                 # S_ctx
    b += s.R * W * s.HK * s.dk * io                  # q
    b += s.R * W * s.HV * s.dv * 4                   # o
    b += slab_bytes(wl, t)                           # k_t, v_t, alpha_t, beta_t read
    b += s.R * W * rec                               # k_t, delta_t, (alpha_t, beta_t) written
    b += (sum(unique_record_slots(wl, t)) - s.R * W) * rec  # ancestral records
    if t == 0:
        b += s.R * s.HV * s.dv * s.dk * 4            # S_ctx split write
    if t > 0:
        b += s.R * W * 4 + unique_parents(wl, t) * (t - 1) * 4 + s.R * W * t * 4
    return b


# Record variants: (record kind, record storage) of the library's config.
VARIANTS = {"borrow": ("inputs", "borrow"), "inputs": ("inputs", "copy"),
            "delta": ("delta", "copy")}


def kernel_alg_bytes(wl, t, variant):
    if variant == "delta":
        return fused_alg_bytes_delta(wl, t)
    return fused_alg_bytes(wl, t, borrow=variant == "borrow")


FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32


def prefill_chunked_flops(spec):
    """fp32 flops of onela_prefill_state_chunked as implemented: per chunk of
    C = 64 tokens and (request, value head), the lower ten of the sixteen
    16 x 16 tiles of K K^T, the two products with the unit lower-triangular T
    (row block a needs k < 16 (a + 1): 10/16 of the dense product), then the
    scan's X = W' S^T and K^T D' over the whole chunk."""
    C = 64
    nch = -(-spec.P // C)
    tri = 10 / 16
    per_chunk = (2 * C * C * spec.dk * tri          # K K^T
                 + 2 * C * C * spec.dk * tri        # T (diag(beta gamma) K)
                 + 2 * C * C * spec.dv * tri        # T (diag(beta) V)
                 + 2 * C * spec.dk * spec.dv        # W' S^T
                 + 2 * C * spec.dk * spec.dv)       # K^T D'
    return spec.R * spec.HV * nch * per_chunk


def step_alg_bytes(wl, fused=True, variant="borrow"):
    """Algorithmic bytes of one whole step (T decode steps; init moves none)."""
    s = wl.spec
    total = 0
    for t, W in enumerate(s.widths):
        if fused:
            total += kernel_alg_bytes(wl, t, variant)
        else:
            append = 0 if variant == "borrow" else 2 * slab_bytes(wl, t)
            total += append + decode_alg_bytes(wl, t)
            if t > 0:
                total += s.R * W * 4 + unique_parents(wl, t) * (t - 1) * 4 + s.R * W * t * 4
    return total


def cpu_model() -> str:
    """The host CPU's model name (``/proc/cpuinfo``), or "unknown"."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_threads() -> int:
    """Threads the CPU oracle runs with: the process's CPU affinity, capped by
    OMP_NUM_THREADS when the environment sets it (a shared host's share)."""
    n = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        n = min(n, int(env))
    return max(1, n)


def cpu_baseline(wl, min_seconds, gpu_outs=None):
    """The fp64 oracle (materialised per-beam states) timed on this host's
    cores over whole decodes of one request of the same workload, with all
    the threads it may use and with one thread.  With the GPU's outputs of
    that request (``gpu_outs``: list over t of [W_t][HV][dv]) it also reports
    their max normwise relative error against the oracle, which builds S_ctx
    with its own fp64 prefill."""
    from oracle import oracle as orc
    s = wl.spec
    threads = oracle_threads()
    r = 0
    t0 = time.perf_counter()
    s0 = orc.prefill(wl.prompt_k.f64[r], wl.prompt_v.f64[r], wl.prompt_alpha.f64[r],
                     wl.prompt_beta.f64[r], nthreads=threads).astype(np.float32)
    prefill_s = time.perf_counter() - t0
    args = (s0.astype(np.float64), [x.q.f64[r] for x in wl.steps],
            [x.k.f64[r] for x in wl.steps], [x.v.f64[r] for x in wl.steps],
            [x.alpha.f64[r] for x in wl.steps], [x.beta.f64[r] for x in wl.steps],
            [x.parents[r] for x in wl.steps[1:]])

    def timed(nthreads, seconds, max_reps):
        reps, t0 = 0, time.perf_counter()
        while True:
            orc.decode(*args, nthreads=nthreads)
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds or reps >= max_reps:
                return reps, el

    reps, el = timed(threads, min_seconds, 200)
    # one thread: at least one whole decode, about a third of the budget
    reps1, el1 = timed(1, min_seconds / 3, 200)
    beam_tokens = sum(s.widths)
    err = None
    if gpu_outs is not None:
        ref = orc.decode(*args, nthreads=threads)
        errs = []
        for t in range(s.T):
            got = np.asarray(gpu_outs[t], dtype=np.float64)
            num = np.max(np.abs(got - ref[t]), axis=-1)
            den = np.maximum(np.max(np.abs(ref[t]), axis=-1), 1e-30)
            errs.append(np.max(num / den))
        err = float(np.max(errs))  # a NaN anywhere propagates
    return {"value": reps * beam_tokens / el, "unit": "beam-tokens/s", "cores": threads,
            "ms_per_step": 1e3 * el / reps,
            "one_thread": {"value": reps1 * beam_tokens / el1, "unit": "beam-tokens/s",
                           "cores": 1, "ms_per_step": 1e3 * el1 / reps1,
                           "sample": f"{reps1} decodes, {el1:.1f} s"},
            "affinity_cpus": len(os.sched_getaffinity(0)),
            "omp_num_threads_env": os.environ.get("OMP_NUM_THREADS"),
            "cpu_model": cpu_model(),
            "prefill_s": prefill_s,
            "max_rel_err_gpu_vs_oracle": err,
            "kind": "oracle",
            "sample": f"{reps} full {s.T}-step decodes of one request "
                      f"({s.HV} heads, {s.W} beams, S_ctx given), {el:.1f} s on {threads} "
                      f"threads, fp64 materialised per-beam states; S_ctx prefill "
                      f"({s.P} tokens) timed separately"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--batches", type=int, default=40)
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--graph-group", type=int, default=20,
                    help="largest number of batches interleaved step by step in one graph "
                         "(the group is the largest divisor of --steps not above it)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--skip-fullstate", action="store_true")
    ap.add_argument("--variant", choices=tuple(VARIANTS), default="borrow",
                    help="record variant of the headline path: borrowed zero-copy input "
                         "records, input records copied into the arena, or the paper's "
                         "delta records (the others are timed as an A/B)")
    ap.add_argument("--skip-ab", action="store_true")
    ap.add_argument("--skip-select", action="store_true")
    ap.add_argument("--skip-loop", action="store_true",
                    help="skip the closed-loop leg (fused decode + beam selection per step)")
    ap.add_argument("--skip-prefill", action="store_true")
    ap.add_argument("--layers", type=int, default=18,
                    help="GDN layers of the multi-layer leg (the paper's model has 18)")
    ap.add_argument("--skip-layers", action="store_true",
                    help="skip the multi-layer leg (one decode step over L layers' contexts)")
    ap.add_argument("--select-vocab", type=int, default=None,
                    help="codebook size of the beam-selection measurement")
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
    cfgs = {v: runner.config_for(spec, records=rk, storage=st) for v, (rk, st) in VARIANTS.items()}
    ws_bytes = max(ab.onela_workspace_bytes(c) for c in cfgs.values())
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

    def group_steps(bs, fused, kind):
        """One whole step (init + T decode steps) of every batch in ``bs``,
        interleaved by decode step, on the current stream."""
        ctxs = [ab.onela_init(cfgs[kind], b["s0"], b["ws"], ws_bytes, None) for b in bs]
        for t in range(T):
            for ctx, b in zip(ctxs, bs):
                st = b["steps"][t]
                if fused:
                    ab.onela_decode_step_fused(ctx, t, st.width, st.parents, st.k, st.v,
                                               st.alpha, st.beta, st.q, b["outs"][t])
                else:
                    ab.onela_resolve_ancestry(ctx, t, st.width, st.parents, None)
                    ab.onela_append_records(ctx, t, st.k, st.v, st.alpha, st.beta)
                    ab.onela_decode_step(ctx, t, st.q, b["outs"][t])
        for ctx in ctxs:
            ab.onela_destroy(ctx)

    def capture(fn):
        fn()  # eager once before capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        torch.cuda.synchronize()
        return g

    def group_size(K):
        """Largest divisor of K that is at most --graph-group and the batch count."""
        cap = max(1, min(args.graph_group, NB))
        return max(g for g in range(1, cap + 1) if K % g == 0)

    G = group_size(args.steps)
    NG = NB // G  # groups of distinct batches, replayed round robin

    def timed_steps(fused, K, warmup, kind):
        """Exactly K steps as K / G whole groups (group i uses batches
        G*(i % NG) .. G*(i % NG) + G - 1); the warm-up is rounded up to whole
        groups.  Returns ms per step."""
        groups = [batches[G * g:G * g + G] for g in range(NG)]
        graphs = None
        if not args.no_graph:
            graphs = [capture(lambda bs=bs: group_steps(bs, fused, kind)) for bs in groups]

        def run(ngroups, start):
            for i in range(ngroups):
                g = (start + i) % NG
                if graphs is None:
                    group_steps(groups[g], fused, kind)
                else:
                    graphs[g].replay()

        nw = -(-warmup // G)
        run(nw, 0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run(K // G, nw)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    K = args.steps
    kind = args.variant
    log(f"[bench] fused path ({kind}): warmup {args.warmup}, {K} timed steps")
    ms_per_step = timed_steps(True, K, args.warmup, kind)
    # outputs of the headline path, before any other leg reuses the buffers
    head_outs = [o[0].cpu().numpy() for o in batches[0]["outs"]]
    beam_tokens_per_step = spec.R * sum(spec.widths)
    value = beam_tokens_per_step / (ms_per_step / 1e3)
    log(f"[bench] fused: {ms_per_step * 1e3:.1f} us/step")
    ms_sep = timed_steps(False, K, args.warmup, kind)
    log(f"[bench] separate calls: {ms_sep * 1e3:.1f} us/step")

    # ---- dominant-kernel roofline: the fused step kernel.  Per decode step t
    # one graph holds the fused launches of every batch back to back (batch b
    # at step t), bracketed by HIP events on the same stream; a batch's data
    # was last touched NB - 1 launches earlier.
    ctxs = [None] * NB
    rs = torch.cuda.Stream()  # contexts bound to the stream the graphs capture

    def capture_on_rs(fn):
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=rs):
            fn()
        torch.cuda.synchronize()
        return g

    def fused_kernel_us(kind):
        """Average fused-launch duration per decode step t: graphs of the step-t
        launches of G batches (a group of the whole-step protocol, so that
        the caches hold what they hold there) and of the first G / 2,
        replayed in turn; the difference of their event times over the
        G - G / 2 extra launches leaves out the fixed cost of a graph replay."""
        def init_all():
            for i, b in enumerate(batches):
                ctxs[i] = ab.onela_init(cfgs[kind], b["s0"], b["ws"], ws_bytes, rs)

        def fused_all(t, nb):
            for i, b in enumerate(batches[:nb]):
                st = b["steps"][t]
                ab.onela_decode_step_fused(ctxs[i], t, st.width, st.parents, st.k, st.v,
                                           st.alpha, st.beta, st.q, b["outs"][t])

        # Graphs hold kernel arguments by value, so each one is captured with
        # the host-side contexts already advanced to the step it replays;
        # replaying graphs[0..T-1] redoes the whole sequence on the device
        # (onela_init enqueues nothing).
        full, half = G, max(1, G // 2)
        graphs = {}
        for nb in (full, half):
            for t in range(T):
                with torch.cuda.stream(rs):
                    init_all()
                    for tt in range(t):
                        fused_all(tt, full)
                graphs[nb, t] = capture_on_rs(lambda t=t, nb=nb: fused_all(t, nb))
                for c in ctxs:
                    ab.onela_destroy(c)
        torch.cuda.synchronize()
        n_roof = max(4, args.steps // 20)
        ms = {nb: np.zeros((n_roof, T)) for nb in (full, half)}
        for i in range(n_roof):
            for nb in (full, half):
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(T + 1)]
                ev[0].record()
                for t in range(T):
                    graphs[nb, t].replay()
                    ev[t + 1].record()
                torch.cuda.synchronize()
                ms[nb][i] = [ev[t].elapsed_time(ev[t + 1]) for t in range(T)]
        if full > half:
            diff = (ms[full][1:] - ms[half][1:]).mean(axis=0) / (full - half)
        else:  # a group of one batch: the replay cost stays in
            diff = ms[full][1:].mean(axis=0) / full
        return diff * 1e3

    dec_us = fused_kernel_us(kind)
    bytes_t = [kernel_alg_bytes(wl, t, kind) for t in range(T)]
    achieved = sum(bytes_t) / (dec_us.sum() * 1e-6) / 1e9
    log(f"[bench] fused kernel us per t: {np.round(dec_us, 2).tolist()}  "
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
        "dtype": ("bf16 in, f32 accum" if spec.io_dtype == "bf16" else "f32"),
        "data": "synthetic",
        "config": {"workload": name, "requests": spec.R, "qk_heads": spec.HK,
                   "v_heads": spec.HV, "d_k": spec.dk, "d_v": spec.dv, "prompt": spec.P,
                   "beams": spec.W, "decode_steps": T, "io_dtype": spec.io_dtype,
                   "parents": f"{spec.parents}{spec.zipf_s if spec.parents == 'zipf' else ''}",
                   "step": "onela_init + per t onela_decode_step_fused (resolve + append "
                           "+ decode in one launch)",
                   "records": {"borrow": "step inputs (k, v, alpha, beta), borrowed "
                                         "in place (zero-copy slabs)",
                               "inputs": "step inputs (k, v, alpha, beta) copied into the "
                                         "workspace arena",
                               "delta": "(alpha, delta fp16, k) transition records"}[kind],
                   "contraction": "S_ctx.P on bf16 MFMA, hi/lo split in registers, 3 products, "
                                  "fp32 accum",
                   "variant": kind, "graph": not args.no_graph, "graph_group": G, "batches": NB,
                   "protocol": f"K / {G} whole groups of {G} batches, each group one HIP graph "
                               f"with the batches' steps interleaved by decode step"},
        "decode_step_us": {"per_t": [round(float(x), 3) for x in dec_us],
                           "mean": round(float(dec_us.mean()), 3)},
        "beam_tokens_per_step": beam_tokens_per_step,
        "step_alg_bytes": step_alg_bytes(wl, fused=True, variant=kind),
        "separate_calls": {"ms_per_step": ms_sep,
                           "beam_tokens_per_s": beam_tokens_per_step / (ms_sep / 1e3),
                           "step": "onela_init + per t (resolve_ancestry, append_records, "
                                   "decode_step)",
                           "step_alg_bytes": step_alg_bytes(wl, fused=False, variant=kind)},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": ("replay_kernel<FUSED>" if kind == "delta"
                                else "decode_kernel<FUSED>"),
                     "alg_bytes_per_t": bytes_t,
                     "us_per_t": [round(float(x), 3) for x in dec_us],
                     "timing": f"HIP events around graphs of the step-t launches of {G} "
                               f"and of {max(1, G // 2)} batches (one whole-step group and "
                               f"half of it); their difference per extra launch"},
    }

    # ---- A/B: the other record variants (borrowed or copied input records
    # with the backward query fold; the paper's (alpha, delta, k) records with
    # forward replay), same workload and protocol
    if not args.skip_ab:
        result["record_variant_ab"] = {}
        for other in VARIANTS:
            if other == kind:
                continue
            ms_o = timed_steps(True, K, args.warmup, other)
            us_o = fused_kernel_us(other)
            bytes_o = [kernel_alg_bytes(wl, t, other) for t in range(T)]
            result["record_variant_ab"][other] = {
                "ms_per_step": ms_o,
                "beam_tokens_per_s": beam_tokens_per_step / (ms_o / 1e3),
                "fused_kernel_us_per_t": [round(float(x), 3) for x in us_o],
                "alg_bytes_per_t": bytes_o,
                "achieved_GBs": sum(bytes_o) / (us_o.sum() * 1e-6) / 1e9}
            log(f"[bench] A/B {other}: {ms_o * 1e3:.1f} us/step, kernel us per t "
                f"{np.round(us_o, 2).tolist()}")

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
            "speedup_fused_kernels": fs_ms / (dec_us.sum() / 1e3)}
        log(f"[bench] fullstate baseline {fs_ms:.3f} ms/step")
        del base

    # ---- S_ctx prefill of the workload's prompt (supplementary: setup work
    # before the decode loop): the sequential kernel and the chunked one
    if not args.skip_prefill and dw0.prompt is not None:
        cfg_p = runner.config_for(spec)
        pf_bytes = ab.onela_prefill_workspace_bytes(cfg_p, spec.P)
        pf_ws = torch.empty(max(pf_bytes, 1), dtype=torch.uint8, device=dev)
        s_tmp = torch.empty_like(s0)

        def time_ms(fn, reps):
            fn()
            torch.cuda.synchronize()
            a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a0.record()
            for _ in range(reps):
                fn()
            a1.record()
            torch.cuda.synchronize()
            return a0.elapsed_time(a1) / reps

        seq_ms = time_ms(lambda: ab.onela_prefill_state(cfg_p, spec.P, *dw0.prompt, s_tmp), 3)
        chk_ms = time_ms(lambda: ab.onela_prefill_state_chunked(cfg_p, spec.P, *dw0.prompt, s_tmp,
                                                                pf_ws, pf_bytes), 10)
        flops = prefill_chunked_flops(spec)
        result["prefill"] = {
            "prompt_tokens": spec.P, "requests": spec.R,
            "sequential_ms": seq_ms, "chunked_ms": chk_ms,
            "chunked_tokens_per_s": spec.R * spec.P / (chk_ms / 1e3),
            "chunked_workspace_bytes": pf_bytes,
            "roofline": {"bound": "mfma", "achieved": flops / (chk_ms / 1e3) / 1e12,
                         "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": flops / (chk_ms / 1e3) / 1e12 / FP32_MFMA_PEAK_TFLOPS,
                         "flops": flops,
                         "count": "the fp32 products of the chunked method as computed: "
                                  "K K^T, T.(diag(beta gamma) K), T.(diag(beta) V) per "
                                  "chunk, W' S^T and K^T D' per chunk and 16-row block "
                                  "(with bf16 keys the products with T and K^T D' run as "
                                  "exact products of bf16 parts on the bf16 instruction; "
                                  "counted once, as fp32 products)"},
            "note": "onela_prefill_state (token by token) vs onela_prefill_state_chunked "
                    "(64-token chunks); setup work, not part of `value`"}
        log(f"[bench] prefill {spec.P} tokens: sequential {seq_ms:.2f} ms, chunked {chk_ms:.3f} ms")
        del pf_ws, s_tmp

    # ---- global top-W beam selection (supplementary: not part of `value`):
    # the next step's parents from W_prev x V candidate scores per request
    if not args.skip_select:
        wp = spec.widths[-1]
        vocab = args.select_vocab or Wm.SELECT_CODEBOOK
        logp_np, beam_np = Wm.make_select_inputs(spec.R, wp, vocab, seed=spec.seed + 1)
        logp_d = torch.from_numpy(logp_np).to(dev)
        beam_d = torch.from_numpy(beam_np).to(dev)
        ss = torch.cuda.Stream()
        sel = runner.BeamSelector(spec.R, wp, vocab, wp, dev, stream=ss)
        sel(logp_d, beam_d)
        torch.cuda.synchronize()
        reps_g = 20
        gsel = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gsel, stream=ss):
            for _ in range(reps_g):
                sel(logp_d, beam_d)
        torch.cuda.synchronize()
        gsel.replay()
        torch.cuda.synchronize()
        se0, se1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(ss):
            se0.record()
            for _ in range(5):
                gsel.replay()
            se1.record()
        torch.cuda.synchronize()
        sel_us = se0.elapsed_time(se1) * 1e3 / (5 * reps_g)
        sel_bytes = spec.R * wp * (vocab + 1) * 4 + spec.R * wp * 12
        # reference: torch.topk over precomputed candidate scores (no fused
        # beam-score add, no defined order among ties)
        flat = (beam_d[:, :, None] + logp_d).reshape(spec.R, -1)
        torch.topk(flat, wp, dim=1)
        torch.cuda.synchronize()
        te0, te1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        te0.record()
        for _ in range(20):
            torch.topk(flat, wp, dim=1)
        te1.record()
        torch.cuda.synchronize()
        topk_us = te0.elapsed_time(te1) * 1e3 / 20
        result["beam_selection"] = {
            "workload": f"R{spec.R}_wprev{wp}_v{vocab}_w{wp}",
            "us_per_call": sel_us, "alg_bytes": sel_bytes,
            "achieved_GBs": sel_bytes / (sel_us * 1e-6) / 1e9,
            "frac_of_hbm_peak": sel_bytes / (sel_us * 1e-6) / 8.0e12,
            "torch_topk_us": topk_us,
            "traffic_bytes_per_call": measured_select_traffic(f"R{spec.R}_wprev{wp}_v{vocab}_w{wp}"),
            "traffic_source": os.path.relpath(SELECT_PROFILE, ROOT),
            "note": "onela_select_beams (fused beam-score add, total order); torch.topk is "
                    "timed on precomputed scores as a reference only"}
        log(f"[bench] beam selection {sel_us:.1f} us/call ({wp}x{vocab} -> {wp}), "
            f"torch.topk {topk_us:.1f} us")
        del sel, gsel, logp_d, beam_d, flat

    # ---- closed decode loop (supplementary, not part of `value`): after every
    # fused decode step the global top-W selection over the step's beams x the
    # codebook, whose parents the next step takes and whose candidate scores
    # are the next selection's beam scores (Sec. 2.1, Fig. 1; Sec. 3.3).  The
    # log-probabilities are seeded synthetic inputs (the model producing them
    # is not part of the path).  Batches interleaved by step as above.
    if not args.skip_loop:
        vocab = args.select_vocab or Wm.SELECT_CODEBOOK
        GL = max(1, min(8, NB // 2))
        nlb = 2 * GL
        lb = []
        for i in range(nlb):
            b = batches[i]
            L = dict(b=b, logp=[], par=[None], tok=[], sc=[], ws=None, ws_bytes=0)
            for t in range(T):
                wt = spec.widths[t]
                wn = spec.widths[t + 1] if t + 1 < T else spec.widths[t]
                logp_np, _ = Wm.make_select_inputs(spec.R, wt, vocab, seed=spec.seed + 31 * t + i,
                                                   with_beam=False)
                L["logp"].append(torch.from_numpy(logp_np).to(dev))
                L["par"].append(torch.zeros((spec.R, wn), dtype=torch.int32, device=dev))
                L["tok"].append(torch.empty((spec.R, wn), dtype=torch.int32, device=dev))
                L["sc"].append(torch.empty((spec.R, wn), dtype=torch.float32, device=dev))
                L["ws_bytes"] = max(L["ws_bytes"],
                                    ab.onela_select_workspace_bytes(spec.R, wt, vocab, wn))
            L["ws"] = torch.zeros(max(L["ws_bytes"], 1), dtype=torch.uint8, device=dev)
            lb.append(L)
        torch.cuda.synchronize()

        def loop_group(ls):
            ctxs = [ab.onela_init(cfgs[kind], L["b"]["s0"], L["b"]["ws"], ws_bytes, None)
                    for L in ls]
            for t in range(T):
                wt = spec.widths[t]
                wn = spec.widths[t + 1] if t + 1 < T else wt
                for ctx, L in zip(ctxs, ls):
                    st = L["b"]["steps"][t]
                    ab.onela_decode_step_fused(ctx, t, wt, L["par"][t], st.k, st.v, st.alpha,
                                               st.beta, st.q, L["b"]["outs"][t])
                for L in ls:
                    ab.onela_select_beams(spec.R, wt, vocab, wn, L["logp"][t],
                                          L["sc"][t - 1] if t > 0 else None, L["par"][t + 1],
                                          L["tok"][t], L["sc"][t], L["ws"], L["ws_bytes"])
            for ctx in ctxs:
                ab.onela_destroy(ctx)

        lgroups = [lb[GL * g:GL * g + GL] for g in range(2)]
        lgraphs = [capture(lambda ls=ls: loop_group(ls)) for ls in lgroups]
        for gr in lgraphs:
            gr.replay()
        torch.cuda.synchronize()
        nrep = 10
        le0, le1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        le0.record()
        for i in range(nrep):
            lgraphs[i % 2].replay()
        le1.record()
        torch.cuda.synchronize()
        loop_ms = le0.elapsed_time(le1) / (nrep * GL)
        # the same graphs without the selections, for the split
        result["closed_loop"] = {
            "ms_per_search": loop_ms,
            "us_per_step": loop_ms * 1e3 / T,
            "beam_tokens_per_s": beam_tokens_per_step / (loop_ms / 1e3),
            "decode_only_ms_per_search": ms_per_step,
            "selection_share": max(0.0, 1.0 - ms_per_step / loop_ms),
            "codebook": vocab,
            "step": f"per decode step t: onela_decode_step_fused, then onela_select_beams "
                    f"over W_t x {vocab} candidates -> W_(t+1) (parents of step t + 1, "
                    f"scores = next beam scores); {T} steps per search",
            "protocol": f"{nrep} graph replays of {GL} batches interleaved by step"}
        log(f"[bench] closed loop: {loop_ms * 1e3:.1f} us per {T}-step search "
            f"({loop_ms * 1e3 / T:.1f} us per decode + select)")
        del lb, lgraphs

    # ---- a model with L GDN layers (supplementary, not part of `value`): L
    # contexts, each with its own S_ctx, record slabs and workspace, advanced
    # through the T decode steps; every step launches the fused kernel of each
    # layer in turn (the layers of one token step are independent here: the
    # model's other layers, which would feed one GDN layer's q, k, v from the
    # previous one's output, are outside the path).  One graph per search.
    if not args.skip_layers and args.layers > 0:
        L = min(args.layers, NB)
        lay = batches[:L]
        lgraph = capture(lambda: group_steps(lay, True, kind))
        lgraph.replay()
        torch.cuda.synchronize()
        nrep = 10
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(nrep):
            lgraph.replay()
        e1.record()
        torch.cuda.synchronize()
        search_us = e0.elapsed_time(e1) * 1e3 / nrep
        result["layers"] = {
            "layers": L, "decode_steps": T,
            "us_per_search": search_us,
            "us_per_token_step_all_layers": search_us / T,
            "us_per_layer_launch": search_us / (T * L),
            "beam_tokens_per_s": beam_tokens_per_step / (search_us * 1e-6),
            "note": f"{L} GDN layers per token step, each its own context; T steps x L "
                    f"fused launches (onela_init per layer) in one HIP graph, {nrep} replays"}
        log(f"[bench] {L} layers: {search_us:.1f} us per {T}-step search "
            f"({search_us / (T * L):.2f} us per layer launch)")
        del lgraph

    # ---- practical HBM ceiling: a plain device copy (torch copy_, 16-byte
    # vector blit) of the same size as the dominant kernel's traffic, and of
    # a size far beyond the caches, buffers rotated so data comes from HBM
    ceil = {}
    for label, nbytes in (("same_size", int(np.mean(bytes_t))), ("large", 256 << 20)):
        half = (nbytes // 2) // 16 * 16
        nbuf = max(2, int(np.ceil(1.5 * (512 << 20) / max(2 * half, 1))))
        src = [torch.empty(half, dtype=torch.uint8, device=dev) for _ in range(nbuf)]
        dst = [torch.empty(half, dtype=torch.uint8, device=dev) for _ in range(nbuf)]
        for i in range(nbuf):
            dst[i].copy_(src[i])
        torch.cuda.synchronize()
        reps = 4 * nbuf
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for i in range(reps):
            dst[i % nbuf].copy_(src[(i + 1) % nbuf])
        c1.record()
        torch.cuda.synchronize()
        us = c0.elapsed_time(c1) * 1e3 / reps
        ceil[label] = {"bytes": 2 * half, "us_per_copy": us, "GB/s": 2 * half / us / 1e3}
        del src, dst
    result["copy_ceiling"] = ceil
    result["roofline"]["frac_of_copy_ceiling_same_size"] = achieved / ceil["same_size"]["GB/s"]
    traffic = measured_traffic(name, kind)
    if traffic is not None:
        result["roofline"]["traffic"] = float(np.mean(traffic))
        result["roofline"]["traffic_per_t"] = traffic
        result["roofline"]["traffic_source"] = os.path.relpath(TRAFFIC_PROFILE, ROOT)
    log(f"[bench] copy ceiling: {ceil['same_size']['GB/s']:.0f} GB/s at "
        f"{ceil['same_size']['bytes'] / 1e6:.1f} MB, {ceil['large']['GB/s']:.0f} GB/s at 256 MiB")

    if not args.skip_cpu:
        log("[bench] cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, head_outs)

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
