#!/usr/bin/env python3
"""Throughput of the data-parallel optimizer update on one MI355X.

One step = the whole hot path over one batch of synthetic input: aggregate
the R ranks' BF16 gradients, global-norm clip, AdamW on the FP32 master and
moments, BF16 re-emit.  The timed workload is the largest one whose states
fit in HBM: one Qwen2.5-72B decoder layer (877,674,496 parameters, R = 8)
with its states in HBM (device mode), where the norm pass stores the mean
gradient and the fused update reads it back (50 B per parameter).  The JSON
line also carries:
  roofline      -- the dominant kernel, the fused update reading the stored
                   mean gradient (30 B per parameter), against 8 TB/s: its
                   duration from HIP events the library records around each
                   launch on its stream, over a second pass of the same
                   number of steps (the headline pass runs without those
                   events); traffic from the committed counter record;
  norm_roofline -- the same for the norm pass that stores the mean gradient;
  copy_ceiling  -- device copies of 2 GiB measured in the same run: the
                   library's 16-byte-per-lane copy kernel, the runtime's
                   hipMemcpyAsync and torch's copy_;
  qwen3_8b_layer -- one Qwen3-8B layer (192,946,176 parameters, R = 4) in
                   device mode (42 B per parameter), with its own roofline and
                   the update's access pattern with trivial arithmetic;
  torch_eager   -- for comparison, the headline step written with PyTorch ops
                   (FP32 mean gradient, clip_grad_norm_, fused AdamW, BF16
                   cast) on the same GPU;
  streamed      -- one Qwen3-14B layer (330,311,680 parameters, R = 4) in
                   pinned host memory, streamed in 32M-element chunks, against
                   the link bound from the faster of the engine's two copy
                   paths per direction, measured in the same run (runtime
                   copies; the library's device-to-host copy kernel), with
                   the BF16 parameters rounded on the host, the staged mode
                   on pageable memory, parameter delivery, a chunk sweep
                   beside the step-time model and the model's chunk;
  host_route    -- the paper's own datapath for the same Qwen3-14B layer:
                   gradients in HBM, states in pageable host memory, the mean
                   gradient copied down (FP32 or BF16) and AdamW on this
                   host's cores, with the host AdamW's core scaling;
  full_model    -- the full Qwen3-14B model (14,768,291,840 parameters,
                   R = 2, 266 GB of pageable host state): the staged streamed
                   step against the same link bound, and the host-update
                   route (inputs generated before the timed steps);
  cpu_baseline  -- the CPU oracle on the headline layer, on this host's cores.
Inputs are generated before the timed region and stay resident; the same
gradient buffers are reused by every timed step.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "AdamW-step params/s + HBM GB/s (% peak); streamed GB/s vs pinned host link"
HBM_PEAK_GBS = 8000.0
KERNEL_SRC = os.path.join(ROOT, "paper_2609_34162_amd", "csrc", "sdp_kernels.hip")
# HBM counter records (rocprofv3 FETCH_SIZE / WRITE_SIZE, calibrated against a
# plain copy); each is valid only for the kernel source it was taken on
TRAFFIC_FILES = {
    1: os.path.join(ROOT, "profiles", "traffic_qwen3_8b_layer_device.json"),
    4: os.path.join(ROOT, "profiles", "traffic_qwen2.5_72b_layer_device.json"),
}


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def measured_traffic(cid, kernel):
    """HBM bytes per launch of `kernel` ("update" or "norm") from the committed
    counter record of workload `cid`, if it was taken on the current kernel
    source (else None)."""
    try:
        rec = json.load(open(TRAFFIC_FILES[cid]))
    except (OSError, ValueError, KeyError):
        return None
    if rec.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return rec.get("kernels", {}).get(kernel, {}).get("hbm_bytes_per_launch")


def events_ms(torch, stream, fn, reps):
    """GPU time of `reps` calls of fn() on `stream`, from torch events."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


def copy_ceiling(torch, sdp, ctx, stream):
    """Device-to-device copies of 2 GiB, ten each after two: the library's
    16-byte-per-lane copy kernel, the runtime's hipMemcpyAsync and torch's
    copy_.  GB/s counts bytes read plus bytes written."""
    nbytes = 2 << 30
    dev = torch.device("cuda:0")
    a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    b = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    a.fill_(1)
    sh = stream.cuda_stream
    ways = {
        "library_copy_kernel": lambda: sdp.sdp_probe_copy(ctx, b.data_ptr(), a.data_ptr(), nbytes, sh),
        "hip_memcpy_async": lambda: sdp.sdp_probe_memcpy(ctx, b.data_ptr(), a.data_ptr(), nbytes, sh),
        "torch_copy": lambda: b.copy_(a),
    }
    out = {}
    with torch.cuda.stream(stream):
        for name, fn in ways.items():
            events_ms(torch, stream, fn, 2)
            best = max(2 * nbytes * 10 / (events_ms(torch, stream, fn, 10) * 1e-3) / 1e9 for _ in range(3))
            out[name] = best
    del a, b
    torch.cuda.empty_cache()
    return out


def device_leg(args, torch, np, synth, sdp, cid, steps, warmup, pattern):
    """Times `steps` device-mode steps of workload `cid` after `warmup` ones,
    then the same number again with the library's per-launch events."""
    w = synth.workload(cid)
    N, R = w.numel, w.ranks
    log(f"device leg: {w.name} N={N} R={R}; generating inputs")
    dev = torch.device("cuda:0")
    master = synth.master(w, 0)
    p = torch.from_numpy(master).to(dev)
    m = torch.zeros(N, dtype=torch.float32, device=dev)
    v = torch.zeros(N, dtype=torch.float32, device=dev)
    pb = torch.zeros(N, dtype=torch.int16, device=dev)
    host_grads = []
    g = []
    for r in range(R):
        hg = synth.grad_bf16(w, 0, 1, r)
        host_grads.append(hg)
        g.append(torch.from_numpy(hg.view(np.int16)).to(dev))
    ctx = sdp.sdp_ctx_create(0, 0, R, 0)
    segs = sdp.segments_from_tensors([(p, m, v, pb, g)])
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    def step(t):
        sdp.sdp_agg_adam_step(ctx, segs, sdp.make_params(**w.hparams(t)), w.chunk, sh)

    log(f"device leg: {warmup} warmup + {steps} timed steps, then {steps} steps with per-launch events")
    torch.cuda.synchronize()
    for t in range(1, warmup + 1):
        step(t)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(warmup + 1, warmup + steps + 1):
        step(t)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # Kernel durations: the same number of steps again, with the library's
    # HIP events around each launch on its stream.  Those event records cost
    # about 20 us per step on the GPU, so the timed steps above run without them.
    sdp.sdp_ctx_set_timing(ctx, True)
    t0 = time.perf_counter()
    for t in range(warmup + steps + 1, warmup + 2 * steps + 1):
        step(t)
    torch.cuda.synchronize()
    elapsed_events = time.perf_counter() - t0
    kt = sdp.sdp_ctx_get_timing(ctx)
    sdp.sdp_ctx_set_timing(ctx, False)
    norm, clip, bad = sdp.sdp_ctx_last_norm(ctx)
    assert not bad and clip < 1.0, (norm, clip)  # these workloads clip every step

    step_bytes, _ = sdp.sdp_bytes_per_elem(False, R, 0)
    stored = R > 4                                   # the library's default policy
    upd_bytes_per_elem = (4 if stored else 2 * R) + 12 + 14
    norm_bytes_per_elem = 2 * R + (4 if stored else 0)
    upd_s = kt.update_ms / kt.update_launches / 1e3
    norm_s = kt.norm_ms / kt.norm_launches / 1e3
    res = dict(
        workload=w.name, N=N, R=R, chunk=w.chunk, steps=steps, warmup=warmup, elapsed=elapsed,
        ms_per_step=elapsed / steps * 1e3, params_per_s=N * steps / elapsed,
        ms_per_step_with_events=elapsed_events / steps * 1e3,
        step_bytes_per_elem=step_bytes, step_hbm_gbs=step_bytes * N * steps / elapsed / 1e9,
        stored_gbar=stored,
        update_ms=upd_s * 1e3, norm_ms=norm_s * 1e3,
        finalize_ms=kt.finalize_ms / max(kt.finalize_launches, 1),
        update_bytes_per_elem=upd_bytes_per_elem, norm_bytes_per_elem=norm_bytes_per_elem,
        update_gbs=upd_bytes_per_elem * N / upd_s / 1e9, update_bytes=upd_bytes_per_elem * N,
        norm_gbs=norm_bytes_per_elem * N / norm_s / 1e9, norm_bytes=norm_bytes_per_elem * N,
        grad_norm=norm, clip=clip,
    )
    if stored:
        # the g_bar-storing norm pass's own access pattern with trivial
        # arithmetic (into the context's workspace; the states are not
        # touched): its traffic-mix ceiling
        reps = 10
        with torch.cuda.stream(stream):
            events_ms(torch, stream, lambda: sdp.sdp_probe_norm_pattern(ctx, segs, sh), 2)
            ms = events_ms(torch, stream, lambda: sdp.sdp_probe_norm_pattern(ctx, segs, sh), reps)
        res["norm_pattern_gbs"] = norm_bytes_per_elem * N * reps / (ms * 1e-3) / 1e9
        # the same steps without the stored mean gradient (the update reads
        # the R gradients again: 58 instead of 50 B per element), same data
        ctx2 = sdp.sdp_ctx_create(0, 0, R, sdp.SDP_FLAG_DEVICE_GBAR_NEVER)
        for t in range(1, warmup + 1):
            sdp.sdp_agg_adam_step(ctx2, segs, sdp.make_params(**w.hparams(t)), w.chunk, sh)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(warmup + 1, warmup + steps + 1):
            sdp.sdp_agg_adam_step(ctx2, segs, sdp.make_params(**w.hparams(t)), w.chunk, sh)
        torch.cuda.synchronize()
        el2 = time.perf_counter() - t0
        sdp.sdp_ctx_destroy(ctx2)
        nb, _ = sdp.sdp_bytes_per_elem(False, R, sdp.SDP_FLAG_DEVICE_GBAR_NEVER)
        res["unstored_gbar"] = dict(ms_per_step=el2 / steps * 1e3, params_per_s=N * steps / el2,
                                    step_bytes_per_elem=nb, step_hbm_gbs=nb * N * steps / el2 / 1e9)
    if pattern:
        # the update's own access pattern with trivial arithmetic (overwrites
        # the states, whose results were read above): its traffic-mix ceiling
        reps = 10
        with torch.cuda.stream(stream):
            events_ms(torch, stream, lambda: sdp.sdp_probe_update_pattern(ctx, segs, sh), 2)
            ms = events_ms(torch, stream, lambda: sdp.sdp_probe_update_pattern(ctx, segs, sh), reps)
        res["pattern_gbs"] = upd_bytes_per_elem * N * reps / (ms * 1e-3) / 1e9
    res["ctx"] = ctx
    res["_keep"] = (p, m, v, pb, g)
    return res, master, host_grads, w


def release(torch, sdp, res):
    sdp.sdp_ctx_destroy(res.pop("ctx"))
    res.pop("_keep")
    torch.cuda.empty_cache()


def roofline(res, kernel, cid, kind):
    """The roofline object of one kernel of a device leg."""
    ach = res[f"{kernel}_gbs"]
    return {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
            "traffic": measured_traffic(cid, kernel), "kernel": kind,
            "algorithmic_bytes_per_launch": res[f"{kernel}_bytes"],
            "bytes_per_param": res[f"{kernel}_bytes_per_elem"], "launch_ms": res[f"{kernel}_ms"]}


def torch_leg(torch, np, w, master, host_grads, steps, warmup):
    """For comparison only: the same step as a PyTorch user would write it on
    the same GPU, in FP32 arithmetic -- mean of the rank gradients,
    clip_grad_norm_, torch.optim.AdamW(fused=True), cast to BF16.  The
    library never runs this; it shows what the fused kernels replace."""
    N, R = w.numel, w.ranks
    dev = torch.device("cuda:0")
    hp = w.hparams(1)
    p = torch.from_numpy(master).to(dev)
    g = [torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16) for x in host_grads]
    pb = torch.empty(N, dtype=torch.bfloat16, device=dev)
    try:
        opt = torch.optim.AdamW([p], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                                weight_decay=hp["weight_decay"], fused=True)
    except (RuntimeError, ValueError) as e:
        log(f"torch leg: fused AdamW unavailable ({e})")
        return None

    def step():
        acc = g[0].float()
        for x in g[1:]:
            acc.add_(x.float())
        acc.div_(R)
        p.grad = acc
        torch.nn.utils.clip_grad_norm_([p], hp["max_grad_norm"])
        opt.step()
        pb.copy_(p)

    log(f"torch leg: {warmup} warmup + {steps} timed steps of the same update in PyTorch ops")
    for _ in range(warmup):
        step()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del p, g, pb, opt
    torch.cuda.empty_cache()
    return dict(ms_per_step=ms, params_per_s=N / (ms * 1e-3),
                ops="fp32 mean of the R bf16 gradients, clip_grad_norm_, AdamW(fused=True), bf16 cast")


def brief(res, cid, pattern=False):
    """The device-leg figures reported for a workload beside the headline."""
    out = {k: res[k] for k in ("workload", "N", "R", "chunk", "steps", "warmup", "ms_per_step", "params_per_s",
                               "step_bytes_per_elem", "step_hbm_gbs", "stored_gbar", "update_ms", "update_gbs",
                               "norm_ms", "norm_gbs", "finalize_ms")}
    out["step_hbm_frac"] = res["step_hbm_gbs"] / HBM_PEAK_GBS
    out["roofline"] = roofline(res, "update", cid, "fused aggregate+clip+AdamW+BF16 update")
    out["norm_roofline"] = roofline(res, "norm", cid, "norm partials")
    if pattern:
        out["update_pattern_gbs"] = res["pattern_gbs"]
        out["update_frac_of_pattern"] = res["update_gbs"] / res["pattern_gbs"]
    return out


def cpu_leg(args, np, synth, oracle, master, host_grads, w):
    log("cpu leg: oracle on the same layer")
    st = oracle.State([master])
    grads = [host_grads]
    steps = 0
    t0 = time.perf_counter()
    while True:
        rc, _ = oracle.step(st, grads, oracle.hparams(**w.hparams(steps + 1)))
        assert rc == oracle.ORC_OK
        steps += 1
        el = time.perf_counter() - t0
        if el >= args.cpu_seconds or steps >= 20:
            break
    cores = oracle.num_threads()
    # one thread on the 1024 x 1024 workload, for scale
    t = synth.workload(0)
    tm = synth.master(t, 0)
    tg = [[synth.grad_bf16(t, 0, 1, r) for r in range(t.ranks)]]
    ts = oracle.State([tm])
    oracle.set_num_threads(1)
    try:
        t1 = time.perf_counter()
        for k in range(t.steps):
            oracle.step(ts, tg, oracle.hparams(**t.hparams(k + 1)))
        one = t.numel * t.steps / (time.perf_counter() - t1)
    finally:
        oracle.set_num_threads(cores)
    return dict(value=w.numel * steps / el, unit="params/s", cores=cores, kind="oracle",
                sample=f"{steps} full oracle steps of the {w.name} workload "
                       f"({w.numel} params, R={w.ranks}), {el:.1f} s",
                one_thread=dict(workload=t.name, params_per_s=one, steps=t.steps),
                host=host_cpus())


def host_cpus():
    """The host's CPUs as this process sees them: model, logical CPUs, the
    CPUs this process may run on, sockets and NUMA nodes (from /proc and
    /sys; nothing is bound)."""
    out = {"logical_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0))}
    try:
        sockets, model = set(), None
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k = k.strip()
                if k == "model name" and model is None:
                    model = v.strip()
                elif k == "physical id":
                    sockets.add(v.strip())
        out["model"] = model
        out["sockets"] = len(sockets) or None
    except OSError:
        pass
    try:
        out["numa_nodes"] = len([d for d in os.listdir("/sys/devices/system/node") if d.startswith("node")])
    except OSError:
        pass
    return out


SWEEP_CHUNKS = [1 << 20, 1 << 21, 1 << 22, 1 << 23, 1 << 24, 1 << 25]  # 4-128 MiB per FP32 state array


def dep_latency_us(torch, n=64, reps=3):
    """Latency of an event dependency between two GPU streams, as the streamed
    engine's h2d_done and slot_free events order its copy and compute
    streams: n rounds of a 1 MiB host-to-device copy on one stream and a
    one-element kernel on the other, each waiting on the other's event,
    against each chain alone.  Every chain is queued behind a spin kernel on
    its first stream, so the GPU-side times leave the host's enqueue cost
    out.  Best of `reps`."""
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    src = torch.empty(1 << 20, dtype=torch.uint8).pin_memory()
    dst = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    x = torch.zeros(1, device="cuda")
    spin = 50_000_000  # GPU clock cycles, about 20 ms: longer than enqueueing a chain

    def timed(first, body):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(first):
            torch.cuda._sleep(spin)
        e0.record(first)
        body()
        e1.record(first)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3  # us

    def copies():
        with torch.cuda.stream(s1):
            for _ in range(n):
                dst.copy_(src, non_blocking=True)

    def kernels():
        with torch.cuda.stream(s2):
            for _ in range(n):
                x.add_(1.0)

    def ping_pong():
        a = [torch.cuda.Event() for _ in range(n)]
        b = [torch.cuda.Event() for _ in range(n)]
        for i in range(n):
            with torch.cuda.stream(s1):
                dst.copy_(src, non_blocking=True)
            a[i].record(s1)
            s2.wait_event(a[i])
            with torch.cuda.stream(s2):
                x.add_(1.0)
            b[i].record(s2)
            s1.wait_event(b[i])

    t_c = min(timed(s1, copies) for _ in range(reps))
    t_k = min(timed(s2, kernels) for _ in range(reps))
    t_pp = min(timed(s1, ping_pong) for _ in range(reps))
    return max(0.0, (t_pp - t_c - t_k) / (2 * n))


def measure_rates(args, torch, np, sdp, ctx, link, dres):
    """The step-time model's inputs, each measured on this machine: link rates
    (passed in), the per-command copy cost, the kernels' HBM rates and the
    launch cost from the device leg, the norm read-back round trip, the host
    threads' copy bandwidth, the host AdamW lane's rate and per-call cost,
    the host memory a DMA byte takes from that lane, and the latency of an
    event between two GPU streams."""
    big, small = 256 << 20, 1 << 20
    ha, hb = sdp.HostBuffer(big), sdp.HostBuffer(big)
    da = torch.empty(big, dtype=torch.uint8, device="cuda")
    db = torch.empty(big, dtype=torch.uint8, device="cuda")
    per = {}
    for cb in (small, 64 << 20):
        gbs = max(sdp.sdp_probe_link(ctx, ha.ptr, hb.ptr, da.data_ptr(), db.data_ptr(), big, cb, 2)[0]
                  for _ in range(3))
        per[cb] = (big / (gbs * 1e9), big // cb)
    copy_cmd_us = max(0.0, (per[small][0] - per[64 << 20][0]) / (per[small][1] - per[64 << 20][1]) * 1e6)
    del da, db
    ha.close()
    hb.close()
    sdp.sdp_ctx_last_norm(ctx)
    t0 = time.perf_counter()
    for _ in range(200):
        sdp.sdp_ctx_last_norm(ctx)
    sync_us = (time.perf_counter() - t0) / 200 * 1e6
    src = np.ones(1 << 28, np.float32)
    dst = np.empty_like(src)
    sdp.sdp_probe_host_copy(ctx, dst.ctypes.data, src.ctypes.data, src.nbytes, 1)
    host_gbs = max(sdp.sdp_probe_host_copy(ctx, dst.ctypes.data, src.ctypes.data, src.nbytes, 2) for _ in range(3))
    del src, dst
    # the host AdamW lane alone: time(n) = hand-off + bytes / rate, from calls
    # of 1M and 16M elements (FP32 mean gradient: 30 B per element); the
    # intercept is the fixed cost of one hand-off to the host threads
    # (waking them, and the last task's tail)
    hp3 = sdp.make_params(step=3)
    st = [np.full(1 << 26, 1e-2, np.float32) for _ in range(4)]
    pb = np.zeros(1 << 26, np.uint16)

    def lane(n):
        sdp.sdp_host_adamw(ctx, st[0].ctypes.data, st[1].ctypes.data, st[2].ctypes.data, pb.ctypes.data,
                           st[3].ctypes.data, sdp.SDP_GBAR_F32, n, 1.0, hp3)

    def per_call_us(n, reps):
        lane(n)
        best = float("inf")
        for _ in range(3):
            t0 = time.perf_counter()
            for _ in range(reps):
                lane(n)
            best = min(best, (time.perf_counter() - t0) / reps * 1e6)
        return best

    n1, n2 = 1 << 20, 1 << 24
    t1, t2 = per_call_us(n1, 40), per_call_us(n2, 6)
    host_adam_gbs = 30 * (n2 - n1) / ((t2 - t1) * 1e3)
    host_task_us = max(0.0, t1 - 30 * n1 / (host_adam_gbs * 1e3))
    # the same lane while a device-to-host copy streams into pinned memory as
    # in the host-update route -- 128 MiB copies into two pinned buffers used
    # in turn, the route's stage buffers at 32M-element chunks: how much host
    # memory bandwidth each DMA byte takes from it
    piece = 128 << 20
    n_copies = 48
    src_d = torch.empty(piece, dtype=torch.uint8, device="cuda")
    dst_h = [torch.empty(piece, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(side):
        e0.record(side)
        for k in range(n_copies):
            dst_h[k % 2].copy_(src_d, non_blocking=True)
        e1.record(side)
    time.sleep(0.005)  # the copies are running
    # timed as the lane alone was (best of three rounds), and per call less
    # the hand-off, so that the two rates compare like with like
    lane_dma_us = float("inf")
    for _ in range(3):
        t0 = time.perf_counter()
        for _ in range(6):
            lane(n2)
        lane_dma_us = min(lane_dma_us, (time.perf_counter() - t0) / 6 * 1e6)
    busy = not e1.query()  # the copies outlasted the lane's timing
    torch.cuda.synchronize()
    d2h_gbs_meas = n_copies * piece / (e0.elapsed_time(e1) * 1e-3) / 1e9
    host_adam_dma_gbs = 30 * n2 / (max(lane_dma_us - host_task_us, 1.0) * 1e3)
    del src_d, dst_h, st, pb
    # the model gives a host task min(its own rate, host_gbs - cost * DMA
    # rate): a lane slowed below its own rate fixes the cost; a lane that
    # kept its own rate bounds it from above, and the largest cost that keeps
    # it there is taken.  A DMA byte costs at least the byte itself.
    dma_host_cost = 1.0
    if busy and d2h_gbs_meas > 0:
        dma_host_cost = max(1.0, (host_gbs - min(host_adam_dma_gbs, host_adam_gbs)) / d2h_gbs_meas)
    else:
        log("the host lane outlasted the device-to-host copies: DMA cost per byte taken as 1")
    kern_ms = dres["update_ms"] + dres["norm_ms"] + dres["finalize_ms"]
    launch_us = max(0.0, (dres["ms_per_step"] - kern_ms) / 3 * 1e3)
    if hasattr(torch.cuda, "_sleep"):
        dep_us = dep_latency_us(torch)
    else:  # the probe needs the spin kernel to keep host enqueue time out
        log("no torch.cuda._sleep: cross-stream event latency not measured, taken as 0")
        dep_us = 0.0
    vals = dict(h2d_gbs=link[0], d2h_gbs=link[1], both_gbs=link[2], copy_cmd_us=copy_cmd_us,
                norm_gbs=dres["norm_gbs"], update_gbs=dres["update_gbs"], launch_us=launch_us, sync_us=sync_us,
                host_gbs=host_gbs, host_task_us=host_task_us, host_adam_gbs=host_adam_gbs, dep_us=dep_us,
                dma_host_cost=dma_host_cost)
    log(f"host lane beside a {d2h_gbs_meas:.1f} GB/s device-to-host copy: {host_adam_dma_gbs:.1f} GB/s "
        f"(alone {host_adam_gbs:.1f} GB/s)")
    log("model rates: " + ", ".join(f"{k} {v:.1f}" for k, v in vals.items()))
    return sdp.make_rates(**vals), vals


def chunk_sweep(sdp, schedule, numels, R, rates, run_at, passes=1, rates_after=None):
    """Measured step time at each chunk size beside the model's prediction,
    and the chunk each would pick.  run_at(c) returns the times of single
    steps at chunk c; a chunk's figure is their median.  With passes > 1 the
    chunk sizes are measured that many times, in alternating order, so that
    every chunk size sees the same spread of conditions on the host.
    rates_after(), if given, supplies the model's rates once all the
    measurements are in (rates measured during the sweep itself)."""
    meas = {c: [] for c in SWEEP_CHUNKS}
    for k in range(passes):
        for c in (SWEEP_CHUNKS if k % 2 == 0 else SWEEP_CHUNKS[::-1]):
            meas[c].extend(run_at(c))
    if rates_after is not None:
        rates = rates_after()
    rows = []
    for c in SWEEP_CHUNKS:
        pr = sdp.sdp_predict_step(schedule, numels, R, c, 0, rates)
        v = sorted(meas[c])
        ms = v[len(v) // 2]
        rows.append(dict(chunk_elems=c, measured_ms=ms, predicted_ms=pr.predicted_ms, bound_ms=pr.bound_ms,
                         steps=len(v)))
        log(f"  chunk {c >> 20:3d}M: measured {ms:.2f} ms, predicted {pr.predicted_ms:.2f} ms, "
            f"bound {pr.bound_ms:.2f} ms")
    best_pred, _ = sdp.sdp_tune_chunk(schedule, numels, R, 0, rates, SWEEP_CHUNKS)
    best_meas = min(rows, key=lambda r: r["measured_ms"])
    at_pick = next(r["measured_ms"] for r in rows if r["chunk_elems"] == best_pred)
    for r in rows:
        r["rel_error"] = (r["predicted_ms"] - r["measured_ms"]) / r["measured_ms"]
    err = [abs(r["rel_error"]) for r in rows]
    mid = [abs(r["rel_error"]) for r in rows if (1 << 22) <= r["chunk_elems"] <= (1 << 25)]
    out = dict(rows=rows, model_pick=best_pred, measured_best=best_meas["chunk_elems"],
               measured_at_model_pick_ms=at_pick, measured_best_ms=best_meas["measured_ms"],
               mean_abs_rel_error=sum(err) / len(err), max_abs_rel_error=max(err),
               max_abs_rel_error_4m_to_32m=max(mid))
    if rates_after is not None:
        out["model_rates"] = {f: getattr(rates, f) for f, _ in rates._fields_}
    return out


LINK_COPY_BYTES = (32 << 20, 64 << 20, 128 << 20)  # the update pass's copies at 8M, 16M, 32M-element chunks


def measure_link(torch, np, sdp, ctx, pinned, runs=4):
    """Pinned link bandwidth on both of the engine's device-to-host paths, at
    the copy sizes of the engine's update pass: runtime copies both ways
    (sdp_probe_link), and runtime copies in with the library's copy kernel
    out (sdp_probe_link_kernel).  The bound takes, per direction and for both
    at once, the fastest figure of either path at any of these sizes over
    `runs` runs: the largest rate, so the tightest bound that is still a
    bound for whichever path the engine takes."""
    probe_bytes = 1 << 30
    ha, hb = pinned(np.uint8, probe_bytes), pinned(np.uint8, probe_bytes)
    ha[:] = 1
    da = torch.empty(probe_bytes, dtype=torch.uint8, device="cuda")
    db = torch.empty(probe_bytes, dtype=torch.uint8, device="cuda")
    args = (ctx, ha.ctypes.data, hb.ctypes.data, da.data_ptr(), db.data_ptr(), probe_bytes)
    sdp.sdp_probe_link(*args, LINK_COPY_BYTES[-1], 2)  # first copies on fresh streams do not overlap
    sdp.sdp_probe_link_kernel(*args, LINK_COPY_BYTES[-1], 2)
    table = []
    for cb in LINK_COPY_BYTES:
        rt = [sdp.sdp_probe_link(*args, cb, 2) for _ in range(runs)]
        kn = [sdp.sdp_probe_link_kernel(*args, cb, 2) for _ in range(runs)]
        table.append(dict(copy_bytes=cb, runtime=[max(r[k] for r in rt) for k in range(3)],
                          copy_kernel=[max(r[k] for r in kn) for k in range(3)]))
    del da, db
    best = [max(max(row["runtime"][k], row["copy_kernel"][k]) for row in table) for k in range(3)]
    return best, table


def link_bound_ms(N, R, link, d2h_per_param=14):
    """The streamed step's resource lower bound (ms): the norm pass's 2R B per
    parameter in, then the update pass's 12 B in and 14 B (12 with the BF16
    parameters rounded on the host) out, each direction at its own rate and
    both together at the bidirectional rate."""
    h2d, d2h, both = (x * 1e9 for x in link)
    return 1e3 * (2 * R * N / h2d + max(12 * N / h2d, d2h_per_param * N / d2h, (12 + d2h_per_param) * N / both))


def stream_leg(args, torch, np, synth, sdp, dres):
    w = synth.workload(2)
    N, R, C = w.numel, w.ranks, w.chunk
    log(f"streamed leg: {w.name} N={N} R={R} chunk={C}; pinning {N * (14 + 2 * R) / 1e9:.2f} GB")
    bufs = []

    def pinned(dtype, count):
        hb = sdp.HostBuffer(count * np.dtype(dtype).itemsize)
        bufs.append(hb)
        return hb.view(dtype, count)

    p = pinned(np.float32, N)
    synth.master(w, 0, out=p)
    m = pinned(np.float32, N)
    m[:] = 0
    v = pinned(np.float32, N)
    v[:] = 0
    pb = pinned(np.uint16, N)
    pb[:] = 0
    g = []
    for r in range(R):
        x = pinned(np.uint16, N)
        synth.grad_bf16(w, 0, 1, r, out=x)
        g.append(x)
    segs = sdp.Segments([(p.ctypes.data, m.ctypes.data, v.ctypes.data, pb.ctypes.data,
                          [x.ctypes.data for x in g], N)])
    ctx = sdp.sdp_ctx_create(0, C, R, 0)
    link, link_table = measure_link(torch, np, sdp, ctx, pinned)
    log(f"streamed leg: link h2d {link[0]:.1f} d2h {link[1]:.1f} both {link[2]:.1f} GB/s (best of both paths)")
    def timed(c, sg):
        sdp.sdp_stream_step(c, sg, sdp.make_params(**w.hparams(1)), C)  # warmup
        t0 = time.perf_counter()
        for t in range(2, args.stream_steps + 2):
            sdp.sdp_stream_step(c, sg, sdp.make_params(**w.hparams(t)), C)
        return (time.perf_counter() - t0) / args.stream_steps

    el = timed(ctx, segs)
    rates, rate_vals = measure_rates(args, torch, np, sdp, ctx, link, dres)
    h2d_b, d2h_b = sdp.sdp_bytes_per_elem(True, R, 0)
    t_link = link_bound_ms(N, R, link) / 1e3
    sdp.sdp_ctx_destroy(ctx)
    out = dict(workload=w.name, params=N, ranks=R, chunk_elems=C, ms_per_step=el * 1e3,
               params_per_s=N / el, h2d_gbs=h2d_b * N / el / 1e9, d2h_gbs=d2h_b * N / el / 1e9,
               link_gbs={"h2d": link[0], "d2h": link[1], "bidir": link[2]}, link_probe=link_table,
               t_link_ms=t_link * 1e3, frac_of_link_bound=t_link / el, model_rates=rate_vals,
               predicted_ms=sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, C, 0, rates).predicted_ms)
    # the same step with the BF16 parameters rounded on the host from the
    # returned master: 12 B per element back instead of 14
    log("streamed leg: BF16 parameters rounded on the host")
    hctx = sdp.sdp_ctx_create(0, C, R, sdp.SDP_FLAG_STREAM_HOST_CAST)
    hel = timed(hctx, segs)
    sdp.sdp_ctx_destroy(hctx)
    t_link_hc = link_bound_ms(N, R, link, d2h_per_param=12) / 1e3
    out["host_cast"] = dict(ms_per_step=hel * 1e3, params_per_s=N / hel, d2h_bytes_per_param=12,
                            t_link_ms=t_link_hc * 1e3, frac_of_link_bound=t_link_hc / hel,
                            predicted_ms=sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, C,
                                                              sdp.SDP_FLAG_STREAM_HOST_CAST, rates).predicted_ms)
    if not args.no_extra:
        log("streamed leg: chunk sweep")

        def run_at(c):
            cctx = sdp.sdp_ctx_create(0, c, R, 0)
            try:
                sdp.sdp_stream_step(cctx, segs, sdp.make_params(**w.hparams(1)), c)
                times = []
                for t in (2, 3, 4):
                    t0 = time.perf_counter()
                    sdp.sdp_stream_step(cctx, segs, sdp.make_params(**w.hparams(t)), c)
                    times.append((time.perf_counter() - t0) * 1e3)
                return times
            finally:
                sdp.sdp_ctx_destroy(cctx)
        out["chunk_sweep"] = chunk_sweep(sdp, sdp.SDP_SCHED_STREAMED, [N], R, rates, run_at)
        # the step at the chunk the library's own tuning picks (sdp_tune_chunk)
        sw = out["chunk_sweep"]
        out["tuned"] = dict(chunk_elems=sw["model_pick"], ms_per_step=sw["measured_at_model_pick_ms"],
                            params_per_s=N / (sw["measured_at_model_pick_ms"] / 1e3),
                            frac_of_link_bound=t_link * 1e3 / sw["measured_at_model_pick_ms"])
        # the same step with the states in pageable memory, through the staged mode
        log("streamed leg: staged mode on pageable copies of the same state")
        # the staged context pins its bounce buffers before the pageable state exists
        sctx = sdp.sdp_ctx_create(0, C, R, sdp.SDP_FLAG_STREAM_STAGED)
        pg = [np.array(x) for x in (p, m, v, pb)] + [np.array(x) for x in g]
        sseg = sdp.Segments([(pg[0].ctypes.data, pg[1].ctypes.data, pg[2].ctypes.data, pg[3].ctypes.data,
                              [x.ctypes.data for x in pg[4:]], N)])
        sel = timed(sctx, sseg)
        sdp.sdp_ctx_destroy(sctx)
        out["staged_pageable"] = dict(ms_per_step=sel * 1e3, params_per_s=N / sel, frac_of_link_bound=t_link / sel)
        # parameter delivery of the updated master as BF16 into a device window
        log("streamed leg: parameter delivery")
        window = torch.empty(N, dtype=torch.int16, device="cuda")
        dctx = sdp.sdp_ctx_create(0, C, R, 0)
        deliv = {}
        for mname, mode in (("host_cast", sdp.SDP_DELIVER_HOST_CAST), ("device_cast", sdp.SDP_DELIVER_DEVICE_CAST)):
            for sname, src in (("pinned", p), ("pageable", pg[0])):
                sdp.sdp_deliver_params(dctx, src.ctypes.data, window.data_ptr(), N, C, mode)
                t0 = time.perf_counter()
                for _ in range(3):
                    sdp.sdp_deliver_params(dctx, src.ctypes.data, window.data_ptr(), N, C, mode)
                el_d = (time.perf_counter() - t0) / 3
                link_bytes = (2 if mode == sdp.SDP_DELIVER_HOST_CAST else 4) * N
                deliv[f"{mname}_{sname}"] = dict(ms=el_d * 1e3, params_per_s=N / el_d, bf16_gbs=2 * N / el_d / 1e9,
                                                 link_gbs=link_bytes / el_d / 1e9)
                # the same deliveries back to back with the gate on the GPU:
                # the host enqueues the next one while the copies still run
                consumer = torch.cuda.current_stream()
                sdp.sdp_deliver_params_async(dctx, src.ctypes.data, window.data_ptr(), N, C, mode,
                                             consumer_stream=consumer.cuda_stream)
                consumer.synchronize()
                t0 = time.perf_counter()
                for _ in range(3):
                    sdp.sdp_deliver_params_async(dctx, src.ctypes.data, window.data_ptr(), N, C, mode,
                                                 consumer_stream=consumer.cuda_stream)
                consumer.synchronize()
                el_g = (time.perf_counter() - t0) / 3
                deliv[f"{mname}_{sname}"]["gated"] = dict(ms=el_g * 1e3, bf16_gbs=2 * N / el_g / 1e9,
                                                          link_gbs=link_bytes / el_g / 1e9)
        sdp.sdp_ctx_destroy(dctx)
        out["delivery"] = deliv
        del pg, window
    for hbuf in bufs:
        hbuf.close()
    return out, rates


def host_route_leg(args, torch, np, synth, sdp, rates):
    """The paper's own datapath on one GPU: the rank gradients in HBM, the
    states in pageable host memory, the GPU's norm pass and mean gradient,
    chunked copies to the host, and AdamW on this host's cores."""
    w = synth.workload(2)
    N, R, C = w.numel, w.ranks, w.chunk
    log(f"host route leg: {w.name} N={N} R={R} chunk={C}")
    p = synth.master(w, 0)
    m = np.zeros(N, np.float32)
    v = np.zeros(N, np.float32)
    pb = np.zeros(N, np.uint16)
    g = []
    tmp = np.empty(N, np.uint16)
    for r in range(R):
        synth.grad_bf16(w, 0, 1, r, out=tmp)
        g.append(torch.from_numpy(tmp.view(np.int16)).to("cuda"))
    torch.cuda.synchronize()
    del tmp
    segs = sdp.Segments([(p.ctypes.data, m.ctypes.data, v.ctypes.data, pb.ctypes.data,
                          [x.data_ptr() for x in g], N)])
    ctx = sdp.sdp_ctx_create(0, C, R, 0)
    threads = sdp.sdp_ctx_host_threads(ctx)
    # host memory ceiling of the same threads: a copy of 1 GiB
    src = np.ones(1 << 28, np.float32)
    dst = np.empty_like(src)
    sdp.sdp_probe_host_copy(ctx, dst.ctypes.data, src.ctypes.data, src.nbytes, 1)
    host_copy = max(sdp.sdp_probe_host_copy(ctx, dst.ctypes.data, src.ctypes.data, src.nbytes, 2) for _ in range(3))
    del src, dst
    # D2H alone, pinned, with the route's copy size
    ha, hb = sdp.HostBuffer(4 * C), sdp.HostBuffer(4 * C)
    da = torch.empty(4 * C, dtype=torch.uint8, device="cuda")
    db = torch.empty(4 * C, dtype=torch.uint8, device="cuda")
    d2h = max(sdp.sdp_probe_link(ctx, ha.ptr, hb.ptr, da.data_ptr(), db.data_ptr(), 4 * C, 4 * C, 4)[1]
              for _ in range(3))
    del da, db
    ha.close()
    hb.close()
    log(f"host route leg: {threads} host threads, host copy {host_copy:.1f} GB/s, d2h {d2h:.1f} GB/s")
    out = dict(workload=w.name, params=N, ranks=R, chunk_elems=C, host_threads=threads,
               host_copy_gbs=host_copy, d2h_gbs_probe=d2h, states="pageable host memory",
               grads="device memory")
    for name, fmt, gsz in (("f32", sdp.SDP_GBAR_F32, 4), ("bf16", sdp.SDP_GBAR_BF16, 2)):
        sdp.sdp_host_update_step(ctx, segs, sdp.make_params(**w.hparams(1)), C, fmt)  # warmup
        # Each step timed on its own (the library's timers reset per step);
        # every figure below is the median over the steps: a step is 30 ms of
        # host work, and one slowed by other load on the host's memory would
        # move a mean by several percent.
        per = []
        for t in range(2, max(args.stream_steps, 5) + 2):
            sdp.sdp_ctx_set_timing(ctx, 1)
            t0 = time.perf_counter()
            sdp.sdp_host_update_step(ctx, segs, sdp.make_params(**w.hparams(t)), C, fmt)
            el_t = time.perf_counter() - t0
            kt = sdp.sdp_ctx_get_timing(ctx)
            per.append(dict(el=el_t, adam_ms=kt.host_adam_ms, wait_ms=kt.host_wait_ms,
                            issue_us=kt.host_issue_ms * 1e3 / max(kt.host_issues, 1),
                            gpu_norm_ms=kt.norm_ms + kt.finalize_ms, gbar_ms=kt.gbar_ms))
        sdp.sdp_ctx_set_timing(ctx, 0)

        def med(key):
            v = sorted(x[key] for x in per)
            return v[len(v) // 2]

        el = med("el")
        # the calling thread's time to enqueue one piece (kernel and copy),
        # timed by the library around those calls: the model's per-piece
        # host cost of this schedule
        issue_us = med("issue_us")
        host_bytes = (26 + gsz) * N  # p, m, v read and written, g_bar read, BF16 params written
        adam_s = med("adam_ms") / 1e3
        route_rates = None
        if rates is not None:
            # The host lane as it runs in this route, beside the route's own
            # device-to-host copies: its bytes over the host threads' busy
            # time, from the library's timers.  That rate already carries
            # what those copies take from host memory, so the model's DMA
            # cost per byte is the byte itself.  (The lane timed beside
            # torch's device-to-host copies runs slower than it does here;
            # that probe's cost stays in the streamed schedules' rates.)
            # For the same reason host memory must not cap the lane below
            # that rate while the copies run: the ceiling is raised to at
            # least the lane's rate plus the copies'.
            route_rates = type(rates).from_buffer_copy(rates)
            route_rates.host_issue_us = issue_us
            route_rates.host_adam_gbs = host_bytes / adam_s / 1e9
            route_rates.dma_host_cost = 1.0
            route_rates.host_gbs = max(route_rates.host_gbs, route_rates.host_adam_gbs + route_rates.d2h_gbs)
        # host memory carries the host lane's bytes and the copies' bytes
        bound = max((host_bytes + gsz * N) / (host_copy * 1e9), gsz * N / (d2h * 1e9))
        out[name] = dict(ms_per_step=el * 1e3, params_per_s=N / el, d2h_bytes_per_param=gsz, host_issue_us=issue_us,
                         steps=len(per), statistic="median of single steps",
                         gpu_norm_ms=med("gpu_norm_ms"), gbar_kernel_ms=med("gbar_ms"),
                         host_adam_ms=adam_s * 1e3, host_wait_ms=med("wait_ms"),
                         host_adam_gbs=host_bytes / adam_s / 1e9, host_adam_params_per_s=N / adam_s,
                         bound_ms=bound * 1e3, frac_of_bound=bound / el)
        sched = sdp.SDP_SCHED_HOST_ROUTE_BF16 if fmt == sdp.SDP_GBAR_BF16 else sdp.SDP_SCHED_HOST_ROUTE_F32
        if route_rates is not None:
            out[name]["predicted_ms"] = sdp.sdp_predict_step(sched, [N], R, C, 0, route_rates).predicted_ms
            out[name]["model_rates"] = {f: getattr(route_rates, f) for f, _ in route_rates._fields_}
        log(f"host route leg {name}: {el * 1e3:.1f} ms/step, host AdamW {adam_s * 1e3:.1f} ms "
            f"({host_bytes / adam_s / 1e9:.1f} GB/s), waits {med('wait_ms'):.1f} ms")
        if rates is not None and not args.no_extra:
            log(f"host route leg {name}: chunk sweep")

            # Single steps, each timed by the library as well.  The host
            # lane's busy time per step is bytes / rate + pieces x a cost per
            # piece (waking the host threads, the last task's tail); both are
            # fitted, by least squares over the per-chunk medians, to the
            # lane's own busy times in the sweep's steps (not to the step
            # times), and the per-piece issue cost is their median.  The
            # model's host inputs and the measured steps thus see the same
            # conditions on the host, whose memory other load slows from
            # time to time by up to 10%.
            lane, issue = {}, []

            def run_at(c, fmt=fmt):
                sdp.sdp_host_update_step(ctx, segs, sdp.make_params(**w.hparams(1)), c, fmt)
                times = []
                for t in range(2, 7):
                    sdp.sdp_ctx_set_timing(ctx, 1)
                    t0 = time.perf_counter()
                    sdp.sdp_host_update_step(ctx, segs, sdp.make_params(**w.hparams(t)), c, fmt)
                    times.append((time.perf_counter() - t0) * 1e3)
                    kt = sdp.sdp_ctx_get_timing(ctx)
                    lane.setdefault(c, []).append((kt.host_issues + 1, kt.host_adam_ms))  # pieces, busy ms
                    issue.append(kt.host_issue_ms * 1e3 / max(kt.host_issues, 1))
                sdp.sdp_ctx_set_timing(ctx, 0)
                return times

            def rates_after():
                pts = []
                for c, v in lane.items():
                    v = sorted(v, key=lambda x: x[1])
                    pts.append((float(v[len(v) // 2][0]), v[len(v) // 2][1]))
                xm = sum(x for x, _ in pts) / len(pts)
                ym = sum(y for _, y in pts) / len(pts)
                slope = (sum((x - xm) * (y - ym) for x, y in pts) / max(sum((x - xm) ** 2 for x, _ in pts), 1e-12))
                slope = max(slope, 0.0)
                base_ms = ym - slope * xm
                r = type(route_rates).from_buffer_copy(route_rates)
                r.host_adam_gbs = host_bytes / (base_ms * 1e-3) / 1e9
                r.host_task_us = slope * 1e3
                r.host_issue_us = sorted(issue)[len(issue) // 2]
                r.host_gbs = max(r.host_gbs, r.host_adam_gbs + r.d2h_gbs)
                return r
            out[name]["chunk_sweep"] = chunk_sweep(sdp, sched, [N], R, route_rates, run_at, passes=2,
                                                   rates_after=rates_after)
            # the step at C, predicted with the rates the sweep measured
            swr = out[name]["chunk_sweep"]["model_rates"]
            r = type(route_rates).from_buffer_copy(route_rates)
            for f_, v_ in swr.items():
                setattr(r, f_, v_)
            out[name]["predicted_ms"] = sdp.sdp_predict_step(sched, [N], R, C, 0, r).predicted_ms
    # core scaling of the host AdamW alone on the same layer (the paper's
    # CPU Adam scaling microbenchmark)
    gb = np.full(N, 1e-3, np.float32)
    hp = sdp.make_params(**w.hparams(3))
    scaling = []
    for t in (1, 2, 4, 8, 12, 16):
        if t > max(threads, 16):
            break
        sdp.sdp_ctx_set_host_threads(ctx, t)
        call = lambda: sdp.sdp_host_adamw(ctx, p.ctypes.data, m.ctypes.data, v.ctypes.data,  # noqa: E731
                                          pb.ctypes.data, gb.ctypes.data, sdp.SDP_GBAR_F32, N, 1.0, hp)
        call()
        reps = 2 if t < 4 else 4
        t0 = time.perf_counter()
        for _ in range(reps):
            call()
        el = (time.perf_counter() - t0) / reps
        scaling.append(dict(threads=t, params_per_s=N / el, gbs=30 * N / el / 1e9))
        log(f"host AdamW {t:2d} threads: {N / el / 1e9:.2f} G params/s, {30 * N / el / 1e9:.1f} GB/s")
    out["adamw_core_scaling"] = scaling
    sdp.sdp_ctx_destroy(ctx)
    del g
    return out


def mem_available_gib():
    with open("/proc/meminfo") as f:
        for line in f:
            if line.startswith("MemAvailable:"):
                return int(line.split()[1]) / (1 << 20)
    return 0.0


def full_model_leg(args, torch, np, synth, sdp, link):
    """The full Qwen3-14B model (42 segments, R = 2, 32M-element chunks) with
    every state in pageable host memory: the staged streamed step against the
    same link bound as the layer, and the host-update route with the BF16
    mean gradient (its gradients copied to HBM first).  Inputs are generated
    before the timed steps; one untimed step comes first in each mode."""
    w = synth.workload(3)
    sizes = [s.numel for s in w.segments]
    N, R, C = w.numel, w.ranks, w.chunk
    need = N * (14 + 2 * R) / (1 << 30) + 8
    avail = mem_available_gib()
    if avail < need:
        log(f"full model leg skipped: needs {need:.0f} GiB of host memory, {avail:.0f} GiB available")
        return dict(workload=w.name, skipped=f"needs {need:.0f} GiB of host memory, {avail:.0f} GiB available")
    log(f"full model leg: {w.name} N={N} R={R} chunk={C}, {len(sizes)} segments; {avail:.0f} GiB available")
    # the staged context pins its bounce buffers before the host state exists
    ctx = sdp.sdp_ctx_create(0, C, R, sdp.SDP_FLAG_STREAM_STAGED)
    t0 = time.perf_counter()
    p, m, v, pb, g = [], [], [], [], []
    for s, n in enumerate(sizes):
        p.append(synth.master(w, s))
        m.append(np.zeros(n, np.float32))
        v.append(np.zeros(n, np.float32))
        pb.append(np.zeros(n, np.uint16))
        g.append([synth.grad_bf16(w, s, 1, r) for r in range(R)])
        if s % 7 == 6:
            log(f"full model leg: {s + 1}/{len(sizes)} segments generated, {time.perf_counter() - t0:.0f} s")
    gen_s = time.perf_counter() - t0
    log(f"full model leg: inputs generated in {gen_s:.0f} s")
    segs = sdp.Segments([(p[s].ctypes.data, m[s].ctypes.data, v[s].ctypes.data, pb[s].ctypes.data,
                          [x.ctypes.data for x in g[s]], sizes[s]) for s in range(len(sizes))])
    out = dict(workload=w.name, params=N, ranks=R, chunk_elems=C, segments=len(sizes),
               states="pageable host memory", input_generation_s=gen_s)
    try:
        sdp.sdp_stream_step(ctx, segs, sdp.make_params(**w.hparams(1)), C)
        times = []
        for t in range(2, args.full_steps + 2):
            ts = time.perf_counter()
            sdp.sdp_stream_step(ctx, segs, sdp.make_params(**w.hparams(t)), C)
            times.append(time.perf_counter() - ts)
            log(f"full model leg: staged streamed step {times[-1]:.2f} s")
        el = sum(times) / len(times)
        t_link = link_bound_ms(N, R, link) / 1e3
        h2d_b, d2h_b = sdp.sdp_bytes_per_elem(True, R, 0)
        out["staged_streamed"] = dict(ms_per_step=el * 1e3, steps=len(times), params_per_s=N / el,
                                      h2d_gbs=h2d_b * N / el / 1e9, d2h_gbs=d2h_b * N / el / 1e9,
                                      t_link_ms=t_link * 1e3, frac_of_link_bound=t_link / el,
                                      link_gbs={"h2d": link[0], "d2h": link[1], "bidir": link[2]})
    finally:
        sdp.sdp_ctx_destroy(ctx)
    # the host-update route on the same state, gradients moved to HBM
    dg = [[torch.from_numpy(x.view(np.int16)).to("cuda") for x in gs] for gs in g]
    torch.cuda.synchronize()
    rctx = sdp.sdp_ctx_create(0, C, R, 0)
    try:
        rsegs = sdp.Segments([(p[s].ctypes.data, m[s].ctypes.data, v[s].ctypes.data, pb[s].ctypes.data,
                               [x.data_ptr() for x in dg[s]], sizes[s]) for s in range(len(sizes))])
        sdp.sdp_host_update_step(rctx, rsegs, sdp.make_params(**w.hparams(1)), C, sdp.SDP_GBAR_BF16)
        times = []
        for t in range(2, args.full_steps + 2):
            ts = time.perf_counter()
            sdp.sdp_host_update_step(rctx, rsegs, sdp.make_params(**w.hparams(t)), C, sdp.SDP_GBAR_BF16)
            times.append(time.perf_counter() - ts)
        el = sum(times) / len(times)
        out["host_route_bf16"] = dict(ms_per_step=el * 1e3, steps=len(times), params_per_s=N / el,
                                      grads="device memory", d2h_bytes_per_param=2)
        log(f"full model leg: host route {el:.2f} s per step")
    finally:
        sdp.sdp_ctx_destroy(rctx)
    del dg, p, m, v, pb, g
    torch.cuda.empty_cache()
    return out


def clock_trace(torch, np, synth, sdp, cid=4, idle_s=2.0, n_steps=40):
    """Device-mode steps of workload `cid` right after an idle GPU, each timed
    by events on the stream, beside the GPU's current core and memory clock
    levels, read from the driver's sysfs DPM files every 2 ms by a thread.
    Shows the warm-up ramp and what the clocks do during it."""
    import glob
    import threading
    files = {}
    for k in ("pp_dpm_sclk", "pp_dpm_mclk"):
        fs = sorted(glob.glob(f"/sys/class/drm/card*/device/{k}"))
        if fs:
            files[k] = fs[0]

    def level(path):
        try:
            for line in open(path):
                if line.strip().endswith("*"):
                    return float(line.split(":")[1].strip().rstrip("*").strip().lower().rstrip("mhz"))
        except (OSError, ValueError):
            return None
        return None

    w = synth.workload(cid)
    N, R = w.numel, w.ranks
    dev = torch.device("cuda:0")
    p = torch.from_numpy(synth.master(w, 0)).to(dev)
    m = torch.zeros(N, dtype=torch.float32, device=dev)
    v = torch.zeros(N, dtype=torch.float32, device=dev)
    pb = torch.zeros(N, dtype=torch.int16, device=dev)
    g = [torch.from_numpy(synth.grad_bf16(w, 0, 1, r).view(np.int16)).to(dev) for r in range(R)]
    ctx = sdp.sdp_ctx_create(0, 0, R, 0)
    segs = sdp.segments_from_tensors([(p, m, v, pb, g)])
    s = torch.cuda.current_stream()
    for t in range(1, 11):  # compiled, resident, then idle
        sdp.sdp_agg_adam_step(ctx, segs, sdp.make_params(**w.hparams(t)), w.chunk, s.cuda_stream)
    torch.cuda.synchronize()
    samples, stop = [], [False]
    t_base = time.perf_counter()

    def sampler():
        while not stop[0]:
            samples.append((time.perf_counter() - t_base, {k: level(f) for k, f in files.items()}))
            time.sleep(0.002)

    th = threading.Thread(target=sampler)
    th.start()
    time.sleep(idle_s)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_steps + 1)]
    t_start = time.perf_counter() - t_base
    evs[0].record(s)
    for k in range(n_steps):
        sdp.sdp_agg_adam_step(ctx, segs, sdp.make_params(**w.hparams(11 + k)), w.chunk, s.cuda_stream)
        evs[k + 1].record(s)
    torch.cuda.synchronize()
    time.sleep(0.02)
    stop[0] = True
    th.join()
    sdp.sdp_ctx_destroy(ctx)
    ends = [evs[0].elapsed_time(evs[k + 1]) for k in range(n_steps)]
    rows = []
    for k in range(n_steps):
        a = t_start + (ends[k - 1] if k else 0.0) / 1e3
        b = t_start + ends[k] / 1e3
        inside = [d for t, d in samples if a <= t <= b] or [min(samples, key=lambda x: abs(x[0] - b))[1]]
        row = {"step": k + 1, "ms": ends[k] - (ends[k - 1] if k else 0.0)}
        for key in files:
            vals = sorted(x[key] for x in inside if x[key] is not None)
            row[key.replace("pp_dpm_", "") + "_mhz"] = vals[len(vals) // 2] if vals else None
        rows.append(row)
    idle = [d for t, d in samples if t < t_start]
    return {"clock_trace": {"workload": w.name, "params": N, "ranks": R, "idle_s": idle_s,
                            "dpm_files": files, "samples": len(samples),
                            "idle_levels": idle[-1] if idle else None, "steps": rows}}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-stream", action="store_true", help="skip the streamed-mode and host-route legs")
    ap.add_argument("--no-full-model", action="store_true", help="skip the full Qwen3-14B model leg")
    ap.add_argument("--stream-steps", type=int, default=3)
    ap.add_argument("--full-steps", type=int, default=2, help="timed steps of each full-model mode")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the chunk sweeps, the staged layer run and parameter delivery")
    ap.add_argument("--clock-trace", action="store_true",
                    help="only trace the device steps of the Qwen2.5-72B layer after an idle GPU, "
                         "beside the GPU's clock levels, and print that as JSON")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the update runs on one MI355X with the R rank gradients "
              "as separate buffers, and no multi-GPU figure is produced (--gpus must be 1).",
              file=sys.stderr, flush=True)
        sys.exit(2)

    import numpy as np
    import torch
    import oracle
    import synth
    from paper_2609_34162_amd import sdp

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.clock_trace:
        print(json.dumps(clock_trace(torch, np, synth, sdp)), flush=True)
        return
    # the headline: the Qwen2.5-72B layer in HBM
    head, master, host_grads, w = device_leg(args, torch, np, synth, sdp, 4, args.steps, args.warmup, True)
    ceiling = copy_ceiling(torch, sdp, head["ctx"], torch.cuda.current_stream())
    log("copy ceiling: " + ", ".join(f"{k} {v:.0f} GB/s" for k, v in ceiling.items()))
    release(torch, sdp, head)
    tref = torch_leg(torch, np, w, master, host_grads, 10, 3)
    if tref is not None:
        tref["library_speedup"] = tref["ms_per_step"] / head["ms_per_step"]
    cpu = None if args.no_cpu else cpu_leg(args, np, synth, oracle, master, host_grads, w)
    del master, host_grads
    # the Qwen3-8B layer in HBM; its steps are 1.3 ms, so after the idle GPU of
    # the CPU leg five warm-up steps would leave the timed ones inside the
    # clocks' 30 ms transition: it warms up for 40
    q8, _, _, _ = device_leg(args, torch, np, synth, sdp, 1, args.steps, max(args.warmup, 40), True)
    release(torch, sdp, q8)
    streamed, rates = (None, None) if args.no_stream else stream_leg(args, torch, np, synth, sdp, q8)
    route = None if args.no_stream else host_route_leg(args, torch, np, synth, sdp, rates)
    full = None
    if not args.no_full_model:
        link = ([streamed["link_gbs"][k] for k in ("h2d", "d2h", "bidir")] if streamed else None)
        if link is None:
            full = dict(skipped="needs the streamed leg's link measurement")
        else:
            full = full_model_leg(args, torch, np, synth, sdp, link)

    out = {
        "metric": METRIC,
        "value": head["params_per_s"],
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": head["workload"], "params": head["N"], "ranks": head["R"],
                   "mode": "device", "chunk_elems": head["chunk"],
                   "states": "fp32 master/exp_avg/exp_avg_sq, bf16 grads and params; mean gradient stored",
                   "parallelism": "single GPU; R rank gradients as separate buffers"},
        "step_bytes_per_param": head["step_bytes_per_elem"],
        "step_hbm_gbs": head["step_hbm_gbs"],
        "step_hbm_frac": head["step_hbm_gbs"] / HBM_PEAK_GBS,
        "kernel_ms": {"fused_update": head["update_ms"], "norm_partials": head["norm_ms"],
                      "norm_finalize": head["finalize_ms"],
                      "timing": f"HIP events around each launch over {args.steps} further steps "
                                f"({head['ms_per_step_with_events']:.4f} ms per step with the events)"},
        "roofline": roofline(head, "update", 4, "fused update from the stored mean gradient (clip+AdamW+BF16)"),
        "norm_roofline": roofline(head, "norm", 4, "norm partials storing the mean gradient"),
        "norm_pattern_gbs": head.get("norm_pattern_gbs"),
        "norm_frac_of_pattern": (head["norm_gbs"] / head["norm_pattern_gbs"]) if head.get("norm_pattern_gbs") else None,
        "unstored_gbar": head.get("unstored_gbar"),
        "update_pattern_gbs": head["pattern_gbs"],
        "update_frac_of_pattern": head["update_gbs"] / head["pattern_gbs"],
        "copy_ceiling_gbs": ceiling,
        "step_frac_of_copy_ceiling": head["step_hbm_gbs"] / max(ceiling.values()),
        "grad_norm_last_step": head["grad_norm"],
        "qwen3_8b_layer": brief(q8, 1, pattern=True),
        "streamed": streamed,
        "host_route": route,
        "full_model": full,
        "torch_eager": tref,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
