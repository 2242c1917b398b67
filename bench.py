"""Benchmark of the paged mixed-bitwidth MoE layer on one MI355X.

A step is one pass of the whole hot path over one batch: route (top-K and
token permutation), paged gate/up GEMM + SwiGLU, paged down GEMM, combine.
Inputs are seeded synthetic tensors already resident in HBM.

Default workload: the Mixtral-shaped decode layer (8 experts, top-2,
H=4096, F=14336, 64 tokens bf16, 128-row pages with 50% 16-bit / 25% int8 /
25% int4, group 128, pool order shuffled). The metric is weight-read HBM
GB/s: bytes of every page (codes plus scale/zero) of the experts with routed
tokens, per step, divided by the step time.

One JSON line is printed on stdout. ``--gpus`` above 1 is refused: this build
runs on one GPU.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "paged mixed-bit MoE layer: weight-read HBM GB/s (decode), MFMA % (prefill)"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_PEAK_BF16 = 2.5166e15     # dense bf16 MFMA, flop/s (256 CU x 2.4 GHz x 4096)
# sources of the decode kernels the traffic counters describe
KERNEL_SRC = [os.path.join(ROOT, "paper_2607_16184_amd", "csrc", f) for f in ("pw_decode.hip", "pw_device.hpp")]


def log(msg):
    sys.stderr.write("[bench] %s\n" % msg)
    sys.stderr.flush()


def kernel_hash():
    h = hashlib.sha256()
    for path in KERNEL_SRC:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def describe(cfg):
    mix = "iid{16,8,4}" if cfg.mix is None else "%d/%d/%d%% 16-bit/int8/int4" % tuple(round(100 * m) for m in cfg.mix)
    experts = ("%d experts" % cfg.E if not cfg.n_shared
               else "%d routed + %d shared (gated) experts" % (cfg.E_routed, cfg.n_shared))
    return ("%s: %s top-%d, H=%d, F=%d, %d tokens %s, %d-row pages %s, G=%d, shuffled pool"
            % (cfg.name, experts, cfg.K, cfg.H, cfg.F, cfg.T, "bf16" if cfg.act else "fp16", cfg.R, mix, cfg.G))


def page_bytes_active(cfg, bits, counts):
    from paper_2607_16184_amd import pw
    per = {}
    for p in range(3):
        tot = 0
        for e in range(cfg.E):
            if counts[e] == 0:
                continue
            for b in bits[p][e]:
                tot += pw.pw_page_bytes(cfg, p, int(b))
        per[p] = tot
    return per


def build_layer(cfg, w16=None, bits=None):
    import numpy as np
    from paper_2607_16184_amd import synth
    from paper_2607_16184_amd.layer import PagedLayer
    t0 = time.time()
    if w16 is None:
        w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    if bits is None:
        bits = synth.bitmap(cfg)
    L = PagedLayer(cfg, PagedLayer.pool_bytes_for(cfg, bits, slack=0.0))
    L.load_pages(w16, bits, synth.pool_order(cfg))
    log("%s: weights generated and paged in %.1f s" % (cfg.name, time.time() - t0))
    return L, w16, bits


def time_steps(L, cfg, x, logits, steps, warmup):
    """Warm up; time `steps` eager steps with per-kernel HIP-event profiling,
    with the routed experts in one chain (each GEMM launch alone: the
    per-kernel durations), then `steps` eager steps with the layers' default
    two chains; then capture one step (route + paged GEMMs + combine) in a
    HIP graph and time exactly `steps` replays of it, which is the step time
    reported (and the same with one chain, for comparison). Every
    replay's output is checked bit-exact against the eager step. L may be a
    list of layers holding the same pages in separate pools: step i then runs
    on layer i mod len(L), so that no step finds another's weights in a cache."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import pw
    from paper_2607_16184_amd.layer import PagedLayer
    Ls = L if isinstance(L, (list, tuple)) else [L]
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, cfg.K + cfg.n_shared)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.int16, device="cuda")
    gate = None
    if cfg.n_shared:
        from paper_2607_16184_amd import synth
        gate = torch.from_numpy(synth.shared_gate(cfg)).cuda()
        for Li in Ls:
            Li.set_shared_experts(cfg.n_shared)

    def step(i):
        Li = Ls[i % len(Ls)]
        if cfg.n_shared:
            routing = Li.route_shared(logits, cfg.K, cfg.n_shared, gate=gate, out=rbuf)
        else:
            routing = Li.route(logits, cfg.K, out=rbuf)
        Li.forward(x, routing, y=y)

    for i in range(max(warmup, len(Ls))):
        step(i)
    torch.cuda.synchronize()
    y_eager = y.clone()

    def profiled(chains):
        """`steps` eager steps with the layers' launch profiling on; per-phase
        milliseconds and counts summed over the layers, wall and event ms."""
        for Li in Ls:
            pw.pw_layer_set_chains(Li.handle, chains)
            pw.pw_profile_read(Li.handle, reset=True)
            pw.pw_profile_enable(Li.handle, True)
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record()
        for i in range(steps):
            step(i)
        ev1.record()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        ms, cnt = [0.0] * pw.PW_NPHASE, [0] * pw.PW_NPHASE
        for Li in Ls:
            pw.pw_profile_enable(Li.handle, False)
            m, c = pw.pw_profile_read(Li.handle, reset=True)
            for k in range(pw.PW_NPHASE):
                ms[k] += m[k]
                cnt[k] += c[k]
        if not torch.equal(y, y_eager):
            raise RuntimeError("the %d-chain step differs from the first eager step" % chains)
        return ms, cnt, (t1 - t0) * 1e3 / steps, ev0.elapsed_time(ev1) / steps

    # per-kernel durations with the experts in one chain (each GEMM launch
    # alone on the GPU); then the eager step with the layers' default two
    # chains
    ms1, cnt1, _, _ = profiled(1)
    _, _, wall_ms, eager_ms = profiled(2)
    # per step (a layer with shared experts launches each GEMM phase twice)
    per_kernel = {name: (ms1[i] / steps if cnt1[i] else None)
                  for i, name in enumerate(("gateup", "down", "combine", "requant"))}
    counts = (rbuf[2][1:] - rbuf[2][:-1]).cpu().numpy()
    out = {"wall_ms": wall_ms, "eager_ms": eager_ms,
           "kernel_ms": per_kernel, "counts": counts, "graph": False, "layers": len(Ls)}
    out["event_ms"] = out["eager_ms"]

    def graph_steps(chains):
        """Capture one step per layer with `chains` expert chains, check
        replays bit-exact, time exactly `steps` replays: (ms per step, the
        per-step p10/p50/p90)."""
        for Li in Ls:
            pw.pw_layer_set_chains(Li.handle, chains)
        graphs = []
        side = torch.cuda.Stream()
        for i in range(len(Ls)):
            g = torch.cuda.CUDAGraph()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                step(i)                              # the capture stream's own warm-up
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                step(i)
            graphs.append(g)
        for i in range(max(warmup, 2) * len(graphs)):
            y.zero_()
            graphs[i % len(graphs)].replay()
            torch.cuda.synchronize()
            if not torch.equal(y, y_eager):
                raise RuntimeError("graph replay differs from the eager step")
        # an untimed run of back-to-back replays first, at least `steps` of
        # them and about 50 ms (by the eager step time): the first such run
        # of a process measures a few per cent slow
        for i in range(max(steps, int(50.0 / max(eager_ms, 1e-3)) + 1)):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        # the timed run: events before the first and after the last replay only
        # (an event after every replay costs about 1.5 % per step)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(steps):
            graphs[i % len(graphs)].replay()
        e1.record()
        torch.cuda.synchronize()
        if not torch.equal(y, y_eager):
            raise RuntimeError("graph replay differs from the eager step")
        ms = e0.elapsed_time(e1) / steps
        # then as many replays with an event after each, for the spread
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        evs[0].record()
        for i in range(steps):
            graphs[i % len(graphs)].replay()
            evs[i + 1].record()
        torch.cuda.synchronize()
        per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(steps))
        return ms, [round(float(np.percentile(per, q)), 4) for q in (10, 50, 90)]

    try:
        # the step as reported (the layers' default two chains), then the
        # same step with one chain, for comparison
        out["event_ms"], out["step_ms_p10_p50_p90"] = graph_steps(2)
        out["event_ms_one_chain"], _ = graph_steps(1)
        out["graph"] = True
    except Exception as exc:                          # report eager timing instead
        log("graph timing unavailable (%s); reporting eager steps" % exc)
    finally:
        for Li in Ls:
            pw.pw_layer_set_chains(Li.handle, 2)
    return out


def traffic_for(kernel, workload, algo_bytes):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.json" % (kernel, workload))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sha256_16") != kernel_hash():
        return None
    return rec.get("bytes_per_launch")


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _median3(fn):
    ts = []
    for _ in range(3):
        t = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t)
    return sorted(ts)[1]


def _oracle_step_s(O, x16, ids, w, T, budget_s):
    """Seconds of one whole oracle step: the median of 3 full steps when one
    fits a quarter of the budget, else a growing sample of tokens scaled to
    T. Returns (seconds, tokens timed, description)."""
    t = time.perf_counter()
    O.forward(x16, ids, w, tokens=[0])
    one = time.perf_counter() - t
    if one * T <= budget_s / 4:
        return _median3(lambda: O.forward(x16, ids, w)), T, "median of 3 full steps"
    done, spent, chunk = 1, one, 1
    while done < T and spent < budget_s:
        toks = list(range(done, min(T, done + chunk)))
        t = time.perf_counter()
        O.forward(x16, ids, w, tokens=toks)
        spent += time.perf_counter() - t
        done += len(toks)
        chunk = min(chunk * 2, 8)
    if done == T:
        return spent, done, "all %d tokens once, in growing chunks" % T
    return spent * T / done, done, "%d of %d tokens, scaled to %d" % (done, T, T)


def cpu_baseline(cfg, w16, bits, logits_np, x16, weight_bytes, budget_s=12.0):
    """The oracle (plain C, fp64 FFN, OpenMP over output rows), timed on this
    host: the benchmark's decode step with every thread (median of 3 steps)
    and on one thread (a sample of tokens, scaled), routing alone, and the
    other workloads' steps, each bounded, with what was sampled stated."""
    import numpy as np
    import oracle
    from paper_2607_16184_amd import synth
    threads = oracle.threads()
    t0 = time.time()
    O = oracle.OracleLayer(cfg.E, cfg.H, cfg.F, cfg.R, cfg.G, cfg.act, cfg.sdt, w16, bits)
    log("oracle layer built in %.1f s" % (time.time() - t0))
    route_s = _median3(lambda: oracle.route(logits_np, cfg.K))
    ids, w = oracle.route(logits_np, cfg.K)
    step_s, done, how = _oracle_step_s(O, x16, ids, w, cfg.T, budget_s)
    # one thread: a sample of tokens, scaled to the step
    oracle.set_threads(1)
    try:
        st_s, st_done, st_how = _oracle_step_s(O, x16, ids, w, cfg.T, budget_s / 2)
    finally:
        oracle.set_threads(threads)
    out = {"value": weight_bytes / step_s / 1e9, "unit": "GB/s", "cores": threads,
           "kind": "oracle", "cpu_model": cpu_model(),
           "sample": "oracle step (routing + fp64 forward of every routed slot, OpenMP over %d threads) "
                     "of the %s layer: %s, %.3f s per step" % (threads, cfg.name, how, step_s),
           "step_s": round(step_s, 4), "routing_ms": round(route_s * 1e3, 4),
           "single_thread": {"value": weight_bytes / st_s / 1e9, "unit": "GB/s", "step_s": round(st_s, 3),
                             "sample": st_how}}
    configs = {}
    # tiny layer: whole steps, every thread and one thread
    c1 = synth.CONFIGS["tiny"]
    w1 = [synth.expert_weights(c1, p) for p in range(3)]
    O1 = oracle.OracleLayer(c1.E, c1.H, c1.F, c1.R, c1.G, c1.act, c1.sdt, w1, synth.bitmap(c1))
    lg1, x1 = synth.logits(c1), synth.activations(c1)
    ids1, w1r = oracle.route(lg1, c1.K)
    mt = _median3(lambda: O1.forward(x1, ids1, w1r))
    oracle.set_threads(1)
    try:
        s1 = _median3(lambda: O1.forward(x1, ids1, w1r))
    finally:
        oracle.set_threads(threads)
    configs["tiny"] = {"step_ms": round(mt * 1e3, 3), "step_ms_single_thread": round(s1 * 1e3, 3),
                       "routing_ms": round(_median3(lambda: oracle.route(lg1, c1.K)) * 1e3, 4),
                       "sample": "median of 3 full steps"}
    # prefill: its routing over all 4096 tokens; the forward of a 64-token
    # slice (per-token cost depends on the shapes and the bitwidth mix only,
    # which the decode layer's pages share), one run, scaled to 4096 tokens
    c3 = synth.CONFIGS["mixtral_prefill"]
    lg3, x3 = synth.logits(c3), synth.activations(c3)
    t = time.perf_counter()
    ids3, w3 = oracle.route(lg3, c3.K)
    r3 = time.perf_counter() - t
    t = time.perf_counter()
    O.forward(x3, ids3, w3, tokens=list(range(64)))
    f3 = (time.perf_counter() - t) * c3.T / 64
    configs["mixtral_prefill"] = {"step_s_scaled": round(f3, 2), "routing_ms": round(r3 * 1e3, 3),
                                  "gflops_per_s": round(6.0 * c3.S * c3.H * c3.F / f3 / 1e9, 2),
                                  "sample": "one run of a 64-token slice scaled to 4096 tokens (labelled "
                                            "scaled), on the decode layer's pages (same shapes and mix)"}
    # fine-grained layer: whole steps
    c4 = synth.CONFIGS["finegrained"]
    w4 = [synth.expert_weights(c4, p) for p in range(3)]
    b4 = synth.bitmap(c4)
    O4 = oracle.OracleLayer(c4.E, c4.H, c4.F, c4.R, c4.G, c4.act, c4.sdt, w4, b4)
    lg4, x4 = synth.logits(c4), synth.activations(c4)
    ids4, w4r = oracle.route(lg4, c4.K)
    s4, _, how4 = _oracle_step_s(O4, x4, ids4, w4r, c4.T, budget_s)
    configs["finegrained"] = {"step_s": round(s4, 3), "routing_ms": round(_median3(lambda: oracle.route(lg4, c4.K)) * 1e3, 4),
                              "gflops_per_s": round(6.0 * c4.S * c4.H * c4.F / s4 / 1e9, 2), "sample": how4}
    del O4, w4
    # runtime downshift: the requant of the 256 plan pages (16 -> int4)
    c5 = synth.CONFIGS["downshift"]
    plan = [blk for ch in synth.downshift_plan(c5, bits) for blk in ch]
    rows = [w16[p][e, rb * cfg.R:(rb + 1) * cfg.R] for (e, p, rb) in plan]
    rq = _median3(lambda: [oracle.quantize_page16(r, cfg.act, cfg.G, 4, cfg.sdt) for r in rows])
    moved = sum(oracle.page_bytes(cfg.R, cfg.kdim(p), cfg.G, 16) + oracle.page_bytes(cfg.R, cfg.kdim(p), cfg.G, 4)
                for (_, p, _) in plan)
    configs["downshift_requant"] = {"pages": len(plan), "requant_s": round(rq, 3),
                                    "GBps": round(moved / rq / 1e9, 3),
                                    "sample": "median of 3 runs of the oracle quantizer over the 256 pages "
                                              "(single-threaded per page), on the decode layer's weights"}
    out["configs"] = configs
    return out


def leg_layer(name, steps, warmup, pools=1):
    """Time another workload's full step; GB/s of active pages and MFMA share.
    pools > 1: that many copies of the layer in separate pools, stepped in turn
    (for weight sets that a 256 MB last-level cache could otherwise serve)."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import synth
    cfg = synth.CONFIGS[name]
    L, w16, bits = build_layer(cfg)
    Ls = [L]
    for _ in range(pools - 1):
        Ls.append(build_layer(cfg, w16=w16, bits=bits)[0])
    del w16
    logits = torch.from_numpy(synth.logits(cfg)).cuda()
    x = torch.from_numpy(synth.activations(cfg).view(np.int16)).cuda()
    r = time_steps(Ls, cfg, x, logits, steps, warmup)
    per = page_bytes_active(cfg, bits, r["counts"])
    wb = per[0] + per[1] + per[2]
    km = r["kernel_ms"]
    gemm_ms = km["gateup"] + km["down"]
    flops = 6.0 * cfg.S * cfg.H * cfg.F
    for Li in Ls:
        Li.close()
    return {"workload": describe(cfg), "steps": steps, "ms_per_step": round(r["event_ms"], 4),
            "pools_rotated": pools,
            "eager_ms_per_step": round(r["eager_ms"], 4),
            "step_timing": "hip_graph_replay" if r["graph"] else "eager",
            "step_ms_p10_p50_p90": r.get("step_ms_p10_p50_p90"),
            "weight_GBps_per_step": round(wb / (r["event_ms"] * 1e-3) / 1e9, 1),
            "gateup_ms": round(km["gateup"], 4), "down_ms": round(km["down"], 4),
            "combine_ms": round(km["combine"], 4),
            "ms_per_step_one_chain": round(r["event_ms_one_chain"], 4) if r.get("event_ms_one_chain") else None,
            "mfma_frac_gemm": round(flops / (gemm_ms * 1e-3) / MFMA_PEAK_BF16, 4),
            "mfma_frac_step": round(flops / (r["event_ms"] * 1e-3) / MFMA_PEAK_BF16, 4),
            "tflops_gemm": round(flops / (gemm_ms * 1e-3) / 1e12, 1)}


def leg_downshift(steps_before=8, steps_after=8):
    """Decode steps of the Mixtral-shaped layer while 8 chunks of 32 16-bit pages
    are requantized to int4 on a side stream and committed at step boundaries."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import pw, synth
    from paper_2607_16184_amd.layer import PagedLayer
    cfg = synth.CONFIGS["downshift"]
    t0 = time.time()
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    bits = synth.bitmap(cfg)
    plan = synth.downshift_plan(cfg, bits)
    # requant alone: the plan's pages in a pool of their own, idle GPU
    pages = [pg for chunk in plan for pg in chunk]
    # warm-up: one requant in a layer of its own (the first launches load the kernels)
    e0, p0, rb0 = pages[0]
    Lw = PagedLayer(cfg, pw.pw_page_bytes(cfg, p0, 16) + pw.pw_page_bytes(cfg, p0, 4) + (1 << 20))
    Lw.load_pages(w16, bits, [pages[0]])
    pw.pw_profile_enable(Lw.handle, True)
    Lw.requant([pages[0]], 4)
    Lw.commit()
    Lw.reclaim()
    torch.cuda.synchronize()
    Lw.close()
    del Lw
    need = sum(pw.pw_page_bytes(cfg, p, 16) + pw.pw_page_bytes(cfg, p, 4) for (_, p, _) in pages)
    alone_moved = need

    def alone(chunks, head_start):
        """Requant of the plan's pages on an idle GPU, one call per chunk:
        (kernel ms summed over the launches, call ms per chunk, launches).
        head_start: a bounded spin (torch.cuda._sleep) occupies the stream
        before each call, so the call's launches are queued before the GPU
        reaches them and the kernel events hold no host submission time."""
        Li = PagedLayer(cfg, int(need * 1.05) + (1 << 20))
        Li.load_pages(w16, bits, pages)
        torch.cuda.synchronize()
        evi = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in chunks]
        pw.pw_profile_read(Li.handle, reset=True)
        pw.pw_profile_enable(Li.handle, True)
        for k, chunk in enumerate(chunks):
            if head_start:
                torch.cuda._sleep(2_000_000)
            evi[k][0].record()
            Li.requant(chunk, 4)
            evi[k][1].record()
            Li.commit()
            Li.reclaim()
        torch.cuda.synchronize()
        pw.pw_profile_enable(Li.handle, False)
        ms, cnt = pw.pw_profile_read(Li.handle, reset=True)
        Li.close()
        return ms[pw.PW_PH_REQUANT], [a.elapsed_time(b) for a, b in evi], cnt[pw.PW_PH_REQUANT]

    # the whole plan in one call (launches of up to 448 pages per bitwidth
    # pair), then the plan's chunks one call each (one launch per chunk);
    # the call time of the one call is also taken without the head start
    alone_kernel_ms, gpu_call_ms, alone_launches = alone([pages], True)
    chunk_kernel_ms, chunk_ms, _ = alone(plan, True)
    _, alone_ms, _ = alone([pages], False)
    log("requant alone: one call %.3f ms with host submission, %.3f ms queued ahead (%d launches, kernels "
        "%.4f ms); per chunk call ms: %s" % (alone_ms[0], gpu_call_ms[0], alone_launches, alone_kernel_ms,
                                           " ".join("%.3f" % m for m in chunk_ms)))
    L = PagedLayer(cfg, PagedLayer.pool_bytes_for(cfg, bits, slack=0.1))
    L.load_pages(w16, bits, synth.pool_order(cfg))
    del w16
    log("downshift layer ready in %.1f s" % (time.time() - t0))
    nsteps = steps_before + len(plan) + steps_after
    ins = []
    for s in range(nsteps):
        lg, x16 = synth.step_inputs(cfg, s)
        ins.append((torch.from_numpy(lg).cuda(), torch.from_numpy(x16.view(np.int16)).cuda()))
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, cfg.K)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.int16, device="cuda")
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nsteps)]
    for s in range(2):   # warm-up
        L.forward(ins[s][1], L.route(ins[s][0], cfg.K, out=rbuf), y=y)
    torch.cuda.synchronize()
    free0 = L.stats()[1]
    pw.pw_profile_read(L.handle, reset=True)
    pw.pw_profile_enable(L.handle, True)
    moved = 0
    for s in range(nsteps):
        k = s - steps_before
        if 0 <= k < len(plan):
            side.wait_stream(main)
            L.requant(plan[k], 4, stream=side)
            for (e, p, rb) in plan[k]:
                moved += pw.pw_page_bytes(cfg, p, 16) + pw.pw_page_bytes(cfg, p, 4)
        ev[s][0].record()
        L.forward(ins[s][1], L.route(ins[s][0], cfg.K, out=rbuf), y=y)
        ev[s][1].record()
        if 0 <= k < len(plan):
            L.commit()
        L.reclaim()
    torch.cuda.synchronize()
    L.reclaim()
    pw.pw_profile_enable(L.handle, False)
    ms, cnt = pw.pw_profile_read(L.handle, reset=True)
    step_ms = [a.elapsed_time(b) for a, b in ev]
    before = float(np.median(step_ms[:steps_before]))
    during = float(np.median(step_ms[steps_before:steps_before + len(plan)]))
    after = float(np.median(step_ms[steps_before + len(plan):]))
    freed = L.stats()[1] - free0
    post = [b.copy() for b in bits]
    for chunk in plan:
        for (e, p, rb) in chunk:
            post[p][e, rb] = 4
    post_bytes = sum(pw.pw_page_bytes(cfg, p, int(b)) for p in range(3) for b in post[p].ravel())
    L.close()
    rq_ms = ms[pw.PW_PH_REQUANT]
    return {"workload": "mixtral_decode layer, 64-token steps; 8 chunks of 32 16-bit pages -> int4 "
                        "on a side stream, committed at step boundaries",
            "step_ms_before": round(before, 4), "step_ms_during": round(during, 4),
            "step_ms_after": round(after, 4), "decode_slowdown": round(during / before - 1.0, 4),
            "requant_alone_GBps": round(alone_moved / (alone_kernel_ms * 1e-3) / 1e9, 1),
            "requant_alone_kernel_ms": round(alone_kernel_ms, 4),
            "requant_alone_launches": alone_launches,
            "requant_alone_call_ms": round(alone_ms[0], 4),
            "requant_alone_call_ms_queued_ahead": round(gpu_call_ms[0], 4),
            "requant_alone_chunked_GBps": round(alone_moved / (chunk_kernel_ms * 1e-3) / 1e9, 1),
            "requant_alone_chunked_kernel_ms_all_chunks": round(chunk_kernel_ms, 4),
            "requant_alone_chunked_call_ms_all_chunks": round(sum(chunk_ms), 4),
            "requant_during_decode_GBps": round(moved / (rq_ms * 1e-3) / 1e9, 1) if rq_ms else None,
            "requant_ms_per_launch_during_decode": round(rq_ms / max(cnt[pw.PW_PH_REQUANT], 1), 4),
            "bytes_freed": int(freed), "post_switch_weight_GBps": round(post_bytes / (after * 1e-3) / 1e9, 1)}


def leg_offload(steps_before=6, steps_after=6):
    """Sec. 3.1 offload order on the Mixtral-shaped layer: the 256 16-bit pages
    of the downshift plan are copied to pinned host memory, lowered to int4,
    and later reloaded chunk by chunk on a side stream while decode steps run;
    each chunk is committed at the first step boundary after its transfer
    completed. Copies cross PCIe: these rates are host-link figures."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import pw, synth
    from paper_2607_16184_amd.layer import PagedLayer
    cfg = synth.CONFIGS["downshift"]
    t0 = time.time()
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    bits = synth.bitmap(cfg)
    plan = synth.downshift_plan(cfg, bits)
    pages = [pg for chunk in plan for pg in chunk]
    L = PagedLayer(cfg, PagedLayer.pool_bytes_for(cfg, bits, slack=0.1))
    L.load_pages(w16, bits, synth.pool_order(cfg))
    del w16
    b16 = [pw.pw_page_bytes(cfg, p, 16) for (_, p, _) in pages]
    L.set_host_pool(sum((b + 255) // 256 * 256 for b in b16))
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    # warm-up transfer (first use of the copy engines), then its slot is dropped
    L.offload([pages[0]], stream=side)
    torch.cuda.synchronize()
    L.drop_host_copy(*pages[0])
    L.reclaim()
    log("offload layer ready in %.1f s" % (time.time() - t0))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    side.wait_stream(main)
    e0.record(side)
    L.offload(pages, stream=side)
    e1.record(side)
    L.requant(pages, 4, stream=side)
    L.commit()
    torch.cuda.synchronize()
    L.reclaim()
    d2h_ms = e0.elapsed_time(e1)
    nin = 16
    ins = []
    for s in range(nin):
        lg, x16 = synth.step_inputs(cfg, s)
        ins.append((torch.from_numpy(lg).cuda(), torch.from_numpy(x16.view(np.int16)).cuda()))
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, cfg.K)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.int16, device="cuda")
    for s in range(2):
        L.forward(ins[s][1], L.route(ins[s][0], cfg.K, out=rbuf), y=y)
    torch.cuda.synchronize()
    ev = []
    rev = []
    k, inflight, last = 0, None, None
    during = []
    s = 0
    # bounded: every chunk's reload is issued once the previous one committed
    while s < 2000 and (last is None or k < len(plan) or inflight is not None or s < last + 1 + steps_after):
        if s >= steps_before and inflight is None and k < len(plan):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(side)
            L.reload(plan[k], stream=side)
            b.record(side)
            rev.append((a, b))
            inflight = b
            k += 1
        ev.append((torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)))
        ev[s][0].record()
        xi = ins[s % nin]
        L.forward(xi[1], L.route(xi[0], cfg.K, out=rbuf), y=y)
        ev[s][1].record()
        if s > 0:
            ev[s - 1][1].synchronize()   # a serving loop: the host runs one step ahead
        if inflight is not None:
            during.append(s)
            if inflight.query():
                L.commit()
                inflight = None
                last = s
        L.reclaim()
        s += 1
    torch.cuda.synchronize()
    if inflight is not None:
        L.commit()
        torch.cuda.synchronize()
    L.reclaim()
    done = all(L.entry(*pg).bits == 16 for pg in pages)
    step_ms = [a.elapsed_time(b) for a, b in ev]
    before = float(np.median(step_ms[:steps_before]))
    dur = float(np.median([step_ms[i] for i in during])) if during else None
    after = float(np.median(step_ms[last + 1:])) if last is not None and last + 1 < len(step_ms) else None
    h2d_ms = sum(a.elapsed_time(b) for a, b in rev)
    L.close()
    return {"workload": "mixtral_decode layer, 64-token steps; 256 16-bit pages (8 chunks of 32) offloaded "
                        "to pinned host memory, lowered to int4, then reloaded chunk by chunk during decode",
            "bytes": int(sum(b16)), "d2h_GBps": round(sum(b16) / (d2h_ms * 1e-3) / 1e9, 1),
            "h2d_GBps": round(sum(b16) / (h2d_ms * 1e-3) / 1e9, 1),
            "reload_chunks": len(rev), "reload_all_back_to_16_bits": bool(done),
            "steps_with_reload_in_flight": len(during),
            "step_ms_before_plan_pages_int4": round(before, 4),
            "step_ms_during_reload": round(dur, 4) if dur is not None else None,
            "step_ms_after_plan_pages_16bit": round(after, 4) if after is not None else None,
            "decode_slowdown": round(dur / before - 1.0, 4) if dur is not None else None}


def leg_planner():
    """Alg. 1 on the Mixtral-shaped decode layer: per-expert routing statistics
    on the GPU each step, one planner step over the whole table under a
    128 MiB KV-pressure target (synthetic sensitivities and heads: the
    calibration tables need trained weights), and the plan requantized on a
    side stream and committed."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import pw, synth
    from paper_2607_16184_amd.layer import PagedLayer
    cfg = synth.CONFIGS["mixtral_decode"]
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    bits = synth.bitmap(cfg)
    L = PagedLayer(cfg, PagedLayer.pool_bytes_for(cfg, bits, slack=0.1))
    L.load_pages(w16, bits, synth.pool_order(cfg))
    del w16
    rng = np.random.default_rng(2000 + 9)
    sens = np.sort(rng.gamma(1.0, 1.0, (L.n_entries, 3)), 1)
    pcfg = pw.planner_config(bucket_frac=[0.25, 0.25, 0.5], mult=[8.0, 2.0, 1.0],
                             floors=[[16, 8, 8], [8, 8, 4], [8, 4, 4], [4, 4, 4]], alpha=0.5,
                             rho_min=-0.5, rho_max=0.5, eps=1e-9, head_w=rng.normal(0, 0.01, (2, 2, 3)),
                             head_a=rng.normal(0, 0.2, (2, 2)), head_c=rng.uniform(0.3, 1.0, (2, 2)))
    planner = L.planner(sens, pcfg)
    lg, x16 = synth.step_inputs(cfg, 0)
    logits = torch.from_numpy(lg).cuda()
    x = torch.from_numpy(x16.view(np.int16)).cuda()
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, cfg.K)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.int16, device="cuda")
    routing = L.route(logits, cfg.K, out=rbuf)
    stats = torch.zeros((cfg.E, 5), dtype=torch.float64, device="cuda")
    stats_dn = torch.zeros((cfg.E, 5), dtype=torch.float64, device="cuda")
    for _ in range(3):
        L.forward(x, routing, y=y)
        L.routing_stats(x, routing, out=stats)
        L.routing_stats(L.hidden_rows(cfg.T, cfg.K), routing, rows_by_position=True, out=stats_dn)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    n = 20
    ev[0].record()
    for _ in range(n):
        L.routing_stats(x, routing, out=stats)
    ev[1].record()
    for _ in range(n):
        L.routing_stats(L.hidden_rows(cfg.T, cfg.K), routing, rows_by_position=True, out=stats_dn)
    ev[2].record()
    for _ in range(n):
        L.forward(x, routing, y=y)
    ev[3].record()
    torch.cuda.synchronize()
    st_x_ms = ev[0].elapsed_time(ev[1]) / n
    st_h_ms = ev[1].elapsed_time(ev[2]) / n
    before = ev[2].elapsed_time(ev[3]) / n
    planner.add_request(stats, stats_dn, 1.0)
    kvb, thr = 2 << 20, 63
    t0 = time.perf_counter()
    reps = 5
    for _ in range(reps):
        r = planner.step(L, free_blocks=0, free_threshold=thr, kv_block_bytes=kvb)
    host_ms = (time.perf_counter() - t0) * 1e3 / reps
    plan = planner.plan()
    free0 = L.stats()[1]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    pw.pw_profile_read(L.handle, reset=True)
    pw.pw_profile_enable(L.handle, True)
    delta = planner.apply(L, stream=side)
    L.commit()
    torch.cuda.synchronize()
    pw.pw_profile_enable(L.handle, False)
    rq_ms = pw.pw_profile_read(L.handle, reset=True)[0][pw.PW_PH_REQUANT]
    L.reclaim()
    freed = L.stats()[1] - free0
    ev[0].record()
    for _ in range(n):
        L.forward(x, routing, y=y)
    ev[1].record()
    torch.cuda.synchronize()
    after = ev[0].elapsed_time(ev[1]) / n
    planner.close()
    L.close()
    return {"workload": "mixtral_decode layer (2688 table entries, 2048 pages); 64-token step statistics; "
                        "one planner step, 4 bitwidth-floor stages, KV target 64 blocks of 2 MiB",
            "stats_gate_up_input_ms": round(st_x_ms, 4), "stats_down_input_ms": round(st_h_ms, 4),
            "plan_step_host_ms": round(host_ms, 3), "target_bytes": int(r.target), "plan_bytes": int(r.bytes),
            "plan_stage": int(r.stage), "plan_units": len(plan), "bytes_freed": int(freed),
            "requant_ms": round(rq_ms, 4), "eager_step_ms_before": round(before, 4),
            "eager_step_ms_after": round(after, 4)}


def leg_apl(steps=20):
    """Nested bit-plane pages on the Mixtral-shaped decode layer: the quantized
    pages of the 50/25/25 % mix (8-bit and 4-bit) are bit-plane pages with
    per-row LUTs (16-bit pages stay plain). Reports the quantization time, the
    decode step (streaming kernel, every page at its committed bitwidth) and
    the 8 -> 4 downshift of all 8-bit pages, which runs no kernel: the commit
    republishes the entries and reclaim frees the page tails."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import pw, synth
    from paper_2607_16184_amd.layer import PagedLayer
    cfg = synth.CONFIGS["mixtral_decode"]
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    bits = synth.bitmap(cfg)
    R = cfg.R
    sizes = {p: {16: pw.pw_page_bytes(cfg, p, 16),
                 8: R * (cfg.F if p == 2 else cfg.H) + 544 * R,
                 4: R * (cfg.F if p == 2 else cfg.H) // 2 + 32 * R} for p in range(3)}
    need = sum(sizes[p][int(b)] for p in range(3) for b in np.asarray(bits[p]).ravel())
    L = PagedLayer(cfg, int(need * 1.05) + (1 << 20))
    order = synth.pool_order(cfg)
    L.load_pages(w16, bits, [pg for pg in order if bits[pg[1]][pg[0], pg[2]] == 16])
    qp = [(e, p, rb, int(bits[p][e, rb])) for (e, p, rb) in order if bits[p][e, rb] != 16]
    torch.cuda.synchronize()
    t0 = time.time()
    L.load_pages_apl(w16, qp)
    quant_s = time.time() - t0
    del w16
    lg, x16 = synth.step_inputs(cfg, 0)
    logits = torch.from_numpy(lg).cuda()
    x = torch.from_numpy(x16.view(np.int16)).cuda()
    rbuf = PagedLayer.routing_buffers(cfg.T, cfg.E, cfg.K)
    y = torch.empty((cfg.T, cfg.H), dtype=torch.int16, device="cuda")

    def timed():
        for _ in range(3):
            L.forward(x, L.route(logits, cfg.K, out=rbuf), y=y)
        torch.cuda.synchronize()
        pw.pw_profile_read(L.handle, reset=True)
        pw.pw_profile_enable(L.handle, True)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            L.forward(x, L.route(logits, cfg.K, out=rbuf), y=y)
        b.record()
        torch.cuda.synchronize()
        pw.pw_profile_enable(L.handle, False)
        ms, cnt = pw.pw_profile_read(L.handle, reset=True)
        return a.elapsed_time(b) / steps, ms[pw.PW_PH_GATEUP] / max(cnt[pw.PW_PH_GATEUP], 1), \
            ms[pw.PW_PH_DOWN] / max(cnt[pw.PW_PH_DOWN], 1)

    cur = [b.copy() for b in bits]
    wbytes = sum(sizes[p][int(b)] for p in range(3) for b in np.asarray(cur[p]).ravel())
    step0, gu0, dn0 = timed()
    eight = [(e, p, rb) for (e, p, rb, b) in qp if b == 8]
    free0 = L.stats()[1]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    t0 = time.perf_counter()
    delta = L.requant(eight, 4, stream=side)
    L.commit()
    torch.cuda.synchronize()
    L.reclaim()
    drop_ms = (time.perf_counter() - t0) * 1e3
    freed = L.stats()[1] - free0
    for (e, p, rb) in eight:
        cur[p][e, rb] = 4
    wbytes1 = sum(sizes[p][int(b)] for p in range(3) for b in np.asarray(cur[p]).ravel())
    step1, gu1, dn1 = timed()
    L.close()
    return {"workload": "mixtral_decode layer, 64-token steps; 8-bit and 4-bit pages as nested bit-planes "
                        "with per-row LUTs (streaming kernel); then every 8-bit page dropped to 4 bits",
            "quantize_s": round(quant_s, 2), "pages_bitplane": len(qp),
            "eager_step_ms": round(step0, 4), "gateup_ms": round(gu0, 4), "down_ms": round(dn0, 4),
            "weight_GBps": round(wbytes / (step0 * 1e-3) / 1e9, 1),
            "downshift_pages": len(eight), "downshift_bytes_freed": int(freed), "downshift_delta": int(delta),
            "downshift_host_ms": round(drop_ms, 3),
            "eager_step_ms_after": round(step1, 4), "gateup_ms_after": round(gu1, 4), "down_ms_after": round(dn1, 4),
            "weight_GBps_after": round(wbytes1 / (step1 * 1e-3) / 1e9, 1)}


def leg_bitwidths(steps=30, warmup=5):
    """The decode layer with every page at one bitwidth (16, 8, 4) beside the
    50/25/25 % mix: per-format rates of the paged GEMMs, counted over the pages
    of the experts the step routes to."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import synth
    cfg = synth.CONFIGS["mixtral_decode"]
    w16 = [synth.expert_weights(cfg, p) for p in range(3)]
    mixed = synth.bitmap(cfg)
    logits = torch.from_numpy(synth.logits(cfg)).cuda()
    x = torch.from_numpy(synth.activations(cfg).view(np.int16)).cuda()
    res = {"workload": "mixtral_decode layer, 64-token steps, every page at one bitwidth vs the mix"}
    for name, b in (("mix", None), ("all16", 16), ("all8", 8), ("all4", 4)):
        bits = mixed if b is None else [np.full_like(bp, b) for bp in mixed]
        L = build_layer(cfg, w16=w16, bits=bits)[0]
        r = time_steps(L, cfg, x, logits, steps, warmup)
        L.close()
        per = page_bytes_active(cfg, bits, r["counts"])
        km = r["kernel_ms"]
        res[name] = {"step_ms": round(r["event_ms"], 4), "gateup_ms": round(km["gateup"], 4),
                     "gateup_page_GBps": round((per[0] + per[1]) / (km["gateup"] * 1e-3) / 1e9, 1),
                     "down_ms": round(km["down"], 4),
                     "down_page_GBps": round(per[2] / (km["down"] * 1e-3) / 1e9, 1)}
    return res


def leg_ceilings(reps=5):
    """What the device delivers: a plain streaming read of 4 GiB (16-byte
    nontemporal loads, 8 workgroups per CU) and back-to-back independent
    32x32x16 bf16 MFMAs from two waves per SIMD, each timed with HIP events
    on the stream it runs on (median of `reps` launches)."""
    import numpy as np
    import torch
    from paper_2607_16184_amd import pw
    st = torch.cuda.current_stream()
    nbytes, nblk_r = 4 << 30, 2048
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    out = torch.zeros(2 * nblk_r, dtype=torch.int32, device="cuda")
    iters, nblk_m = 4096, 1024
    outm = torch.zeros(nblk_m, dtype=torch.float32, device="cuda")

    def timed(fn):
        fn()
        ms = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            fn()
            b.record(st)
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        return float(np.median(ms))

    ms_r = timed(lambda: pw.pw_probe_read(buf.data_ptr(), nbytes, nblk_r, out.data_ptr(), st.cuda_stream))
    if int(out[nblk_r:].sum().item()) != nblk_r:
        raise RuntimeError("read probe: not every workgroup completed")
    ms_m = timed(lambda: pw.pw_probe_mfma(iters, nblk_m, outm.data_ptr(), st.cuda_stream))
    flops = float(nblk_m) * 8 * iters * 4 * 32768
    del buf
    return {"stream_read_GBps": round(nbytes / (ms_r * 1e-3) / 1e9, 1), "stream_read_bytes": nbytes,
            "mfma_bf16_TFLOPs": round(flops / (ms_m * 1e-3) / 1e12, 1),
            "of_published_peaks": {"hbm": round(nbytes / (ms_r * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                   "mfma_bf16": round(flops / (ms_m * 1e-3) / MFMA_PEAK_BF16, 4)}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral_decode")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extras", default="ceilings,bitwidths,prefill,finegrained,shared,downshift,offload,planner,apl",
                    help="comma list of extra legs on the same JSON line ('' for none)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed steps, run one device copy of this many MiB "
                         "(a known-size kernel for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        sys.stderr.write("bench.py runs on one GPU only: the paged MoE hot path here is a "
                         "single-GPU build (no collectives); --gpus %d is not supported.\n" % args.gpus)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_16184_amd import synth

    if not torch.cuda.is_available():
        sys.stderr.write("bench.py needs a GPU\n")
        sys.exit(1)
    cfg = synth.CONFIGS[args.workload]
    L, w16, bits = build_layer(cfg)
    logits_np = synth.logits(cfg)
    x16 = synth.activations(cfg)
    logits = torch.from_numpy(logits_np).cuda()
    x = torch.from_numpy(x16.view(np.int16)).cuda()
    r = time_steps(L, cfg, x, logits, args.steps, args.warmup)
    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    per = page_bytes_active(cfg, bits, r["counts"])
    wbytes = per[0] + per[1] + per[2]
    ms = r["event_ms"]
    value = wbytes / (ms * 1e-3) / 1e9
    S = cfg.T * cfg.K
    # dominant kernel: the gate/up GEMM. Algorithmic bytes per launch: its pages
    # (codes + scale/zero) of active experts, the activations read and the
    # SwiGLU output written.
    gu_ms = r["kernel_ms"]["gateup"]
    gu_bytes = per[0] + per[1] + cfg.T * cfg.H * 2 + S * cfg.F * 2
    achieved = gu_bytes / (gu_ms * 1e-3) / 1e9
    dn_ms = r["kernel_ms"]["down"]
    dn_bytes = per[2] + S * cfg.F * 2 + S * cfg.H * 4
    flops = 6.0 * S * cfg.H * cfg.F
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.act else "f16",
        "data": "synthetic",
        "config": {"workload": describe(cfg), "tokens": cfg.T, "experts": cfg.E, "top_k": cfg.K,
                   "hidden": cfg.H, "ffn": cfg.F, "page_rows": cfg.R, "group": cfg.G,
                   "weight_bytes_per_step": int(wbytes)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic_for("gateup", cfg.name, gu_bytes),
                     "kernel": "k_gateup (paged gate/up GEMM + SwiGLU)",
                     "algorithmic_bytes_per_launch": int(gu_bytes), "avg_launch_ms": round(gu_ms, 4),
                     "launched": "alone: one launch over all routed experts per step, in eager profiled "
                                 "steps (the timed graph step runs the experts as two concurrent chains "
                                 "of gate/up then down)"},
        "kernels": {
            "gateup_ms": round(gu_ms, 4), "down_ms": round(dn_ms, 4),
            "combine_ms": round(r["kernel_ms"]["combine"], 4),
            "down_GBps": round(dn_bytes / (dn_ms * 1e-3) / 1e9, 1),
            "gemm_weight_GBps": round((per[0] + per[1] + per[2]) / ((gu_ms + dn_ms) * 1e-3) / 1e9, 1),
            "kernel_timing": "gateup_ms, down_ms, combine_ms: HIP events around each launch, launched "
                             "alone (the routed experts in one chain), eager profiled steps",
            "step_ms_one_chain": round(r["event_ms_one_chain"], 4) if r.get("event_ms_one_chain") else None,
            "mfma_frac": round(flops / ((gu_ms + dn_ms) * 1e-3) / MFMA_PEAK_BF16, 5),
            "wall_ms_per_step_eager": round(r["wall_ms"], 4),
            "eager_ms_per_step": round(r["eager_ms"], 4),
            "step_timing": "hip_graph_replay" if r["graph"] else "eager",
            "step_ms_p10_p50_p90": r.get("step_ms_p10_p50_p90"),
        },
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, w16, bits, logits_np, x16, wbytes)
    L.close()
    del L, w16
    extras = {}
    for leg in [e for e in args.extras.split(",") if e]:
        t0 = time.time()
        if leg == "ceilings":
            extras["ceilings"] = leg_ceilings()
        elif leg == "bitwidths":
            extras["bitwidths"] = leg_bitwidths()
        elif leg == "prefill":
            extras["prefill"] = leg_layer("mixtral_prefill", steps=20, warmup=2)
        elif leg == "finegrained":
            # 0.57 GB of weights: three pools in turn, so no step reads the
            # previous step's weights from the 256 MB last-level cache
            extras["finegrained"] = leg_layer("finegrained", steps=51, warmup=3, pools=3)
        elif leg == "shared":
            # Qwen-shaped layer with 60 routed + 4 shared experts: routed
            # experts on the decode kernels, shared ones on the tiled kernel;
            # 0.57 GB of weights, so three pools in turn as above
            extras["shared"] = leg_layer("qwen_shared", steps=51, warmup=3, pools=3)
        elif leg == "downshift":
            extras["downshift"] = leg_downshift()
        elif leg == "offload":
            extras["offload"] = leg_offload()
        elif leg == "planner":
            extras["planner"] = leg_planner()
        elif leg == "apl":
            extras["apl"] = leg_apl()
        log("leg %s done in %.1f s" % (leg, time.time() - t0))
    if extras:
        out["extras"] = extras
    print(json.dumps(out))


if __name__ == "__main__":
    main()
