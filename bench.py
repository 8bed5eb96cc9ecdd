"""Benchmark of XPipe's one-stage training step on one MI355X.

One step = one mini-batch of the stage: T forward micro-batches on the
cached forward prediction, T backward micro-batches (each recomputing its
forward) on the cached backward prediction, and the Adam update fused with
emitting the next mini-batch's two predictions.  Inputs are seeded synthetic
tensors already resident in HBM.

Prints ONE JSON line: stage samples/s (value), the predict / Adam HBM rates
of the 1e8-parameter sweep, the roofline of the dominant kernel, and the CPU
oracle timed on a bounded sample.

usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--dtype bf16|f32]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f64": 78.6, "f32": 157.3}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="inception_v3_stage")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--sweep-n", type=int, default=100_000_000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-legs", action="store_true", help="skip the other stage configurations")
    ap.add_argument("--traffic-run", action="store_true",
                    help="a few stage steps plus a 256 MiB calibration copy, for rocprofv3 --pmc "
                         "FETCH_SIZE / WRITE_SIZE runs")
    ap.add_argument("--traffic-summarize", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn the two counter_collection.csv files into profiles/traffic.json")
    return ap.parse_args()


TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic.json")
CALIB_BYTES = 256 << 20


def source_hash():
    """Hash of the kernel sources: stored HBM-traffic figures apply only to the
    kernels they were measured on."""
    import hashlib
    h = hashlib.sha1()
    d = os.path.join(ROOT, "paper_1911_04610_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h", ".cpp")):
            with open(os.path.join(d, f), "rb") as fh:
                h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def kernel_key(name):
    """Common key for rocprofv3's demangled kernel names and the library's
    launch names: no namespace or arguments, storage types as bf16 / f32, and
    without the template arguments only the compiler's name shows (the GEMM's
    gather mode, named by the library only when not 0; the weight gradient's
    grid flag, named only when set; the row kernels' rows per trip; the
    pools' channels per thread)."""
    import re
    n = name.split("(")[0].replace("void ", "").replace("xp::", "")
    n = n.replace("unsigned short", "bf16").replace(" ", "")
    n = n.replace("<float", "<f32").replace(",float", ",f32")
    m = re.match(r"^k_conv_gemm<((?:[^,>]+,){7}[^,>]+),(\d)>$", n)
    if m:
        gm = int(m.group(2))
        n = "k_conv_gemm<" + m.group(1) + ("" if gm == 0 else "," + ("strided", "strided_dgrad")[gm - 1]) + ">"
    m = re.match(r"^k_wgrad_t<((?:\d+,){4}\d+),(true|false)>$", n)
    if m:
        n = "k_wgrad_t<" + m.group(1) + (",grid>" if m.group(2) == "true" else ">")
    return re.sub(r"^(k_bn_apply_v|k_bn_bwd_v|k_maxpool3s2_fwd|k_maxpool3s2_bwd)<(bf16|f32),\d+>$",
                  r"\1<\2>", n)


def traffic_run(args):
    import torch
    # eager launches: the counters are taken per dispatch (same kernels and
    # arguments as the recorded passes)
    w, ms, wall, classes, fin = time_stage(args, timing_pass=False, graphs=False)
    a = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"traffic_run": w.name, "steps": args.steps, "ms_per_step": ms}))


def traffic_summarize(fetch_csv, write_csv):
    import csv
    from collections import defaultdict

    def load(path, counter):
        per = defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]) * 1024.0)  # KiB -> B
        return per

    fe, wr = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")
    copy = [k for k in fe if "copy" in k.lower()]
    calib_name = max(copy, key=lambda k: max(fe[k]))
    f_fac = max(fe[calib_name]) / CALIB_BYTES
    w_fac = max(wr[calib_name]) / CALIB_BYTES
    kernels = {}
    for k in fe:
        if not k.startswith("void xp::") and not k.startswith("xp::"):
            continue
        f = sum(fe[k]) / len(fe[k]) / f_fac
        wv = sum(wr.get(k, [0.0])) / max(len(wr.get(k, [])), 1) / w_fac
        key = kernel_key(k)
        kernels[key] = {"fetch_bytes": round(f), "write_bytes": round(wv),
                        "traffic_bytes": round(f + wv), "dispatches": len(fe[k])}
    out = {"source_hash": source_hash(), "unit": "bytes per launch (HBM, calibrated)",
           "calibration": {"kernel": kernel_key(calib_name), "bytes_each_way": CALIB_BYTES,
                           "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4)},
           "kernels": kernels}
    with open(TRAFFIC_JSON, "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
    print(json.dumps({"written": TRAFFIC_JSON, "kernels": len(kernels),
                      "fetch_factor": f_fac, "write_factor": w_fac}))


def stored_traffic(kernel):
    """Calibrated HBM bytes per launch of `kernel` from profiles/traffic.json,
    or None when absent or taken on other kernel sources."""
    try:
        with open(TRAFFIC_JSON) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != source_hash():
        return None
    k = t.get("kernels", {}).get(kernel_key(kernel))
    return None if k is None else k["traffic_bytes"]


def time_stage(args, timing_pass=True, graphs=True, workload=None, dtype=None, s_fwd=None,
               steps=None, warmup=None, fwd_stream=True):
    import dataclasses
    import torch
    import paper_1911_04610_amd as xp
    import workloads as wl
    w = wl.WORKLOADS[workload or args.workload]()
    if s_fwd is not None:
        w = dataclasses.replace(w, s_fwd=s_fwd)
    dtype = dtype or args.dtype
    steps = args.steps if steps is None else steps
    warmup = args.warmup if warmup is None else warmup
    dt = xp.BF16 if dtype == "bf16" else xp.F32
    tdt = torch.bfloat16 if dt == xp.BF16 else torch.float32
    inp = wl.stage_inputs(w, act_dtype=dtype if dtype == "bf16" else "f32",
                          moment_init="paper")
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dt)
    st.set_graphs(graphs)
    st.set_flat(st.W, inp.params)
    st.set_flat(st.m, inp.m)
    st.set_flat(st.v, inp.v)

    def dev(a):
        return torch.from_numpy(a).cuda().to(tdt)

    # three distinct mini-batches resident in HBM, reused round-robin
    xs = [[dev(x) for x in row] for row in inp.xs]
    labels = None if inp.labels is None else [[torch.from_numpy(l).cuda() for l in row]
                                              for row in inp.labels]
    dys = None if inp.dys is None else [[dev(d) for d in row] for row in inp.dys]
    n, H, W_, C = st.out_shape
    y = torch.empty((n, H, W_, C), dtype=tdt, device="cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    need_dx = w.rank > 0
    dx = torch.empty((w.micro_batch,) + tuple(w.in_shape), dtype=tdt, device="cuda") if need_dx else None
    hp = xp.Hyper()
    state = {"t": 0}
    st.xpipe_predict_weights(xp.FWD, w.s_fwd, hp, 0)
    st.xpipe_predict_weights(xp.BWD, w.s_bwd, hp, 0)
    stream = torch.cuda.current_stream()
    # the forwards on a stream of the stage's own, beside the backwards
    fs = st.xpipe_stage_set_fwd_stream(True) if fwd_stream else None

    def step(j):
        # steady-state order of a pipeline stage: the forward of one
        # micro-batch, then the backward of one (here the same micro-batch, as
        # on the last stage), T times; then the update with the next predictions
        J = len(xs)
        for i in range(w.T):
            st.xpipe_stage_fwd(xs[j % J][i], y, None if labels is None else labels[j % J][i],
                               loss if w.has_loss else None)
            st.xpipe_stage_bwd(xs[j % J][i], None if dys is None else dys[j % J][i],
                               None if labels is None else labels[j % J][i], dx)
        st.xpipe_adam_step(hp, state["t"], w.s_fwd, w.s_bwd, emit_pred=True)
        state["t"] += 1

    for j in range(warmup):
        step(j)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    if fs is not None:
        fs.wait_stream(stream)
    for j in range(steps):
        step(j)
    if fs is not None:
        stream.wait_stream(fs)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / steps
    if fs is not None:
        st.xpipe_stage_set_fwd_stream(False)
    if not timing_pass:
        return w, ms, wall, {}, True
    # the two passes apart (recorded graphs, all lanes): T forwards, then T
    # backwards (each with its recomputed forward), microseconds per micro-batch
    def pass_us(fn, reps=10):
        fn()  # records the pass's graphs (dropped when the forward stream was unset)
        torch.cuda.synchronize()
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record(stream)
        for _ in range(reps):
            fn()
        a1.record(stream)
        torch.cuda.synchronize()
        return a0.elapsed_time(a1) / reps / w.T * 1e3
    passes = {
        "fwd_us": round(pass_us(lambda: [st.xpipe_stage_fwd(xs[0][i], y, None if labels is None else labels[0][i],
                                                            loss if w.has_loss else None) for i in range(w.T)]), 1),
        "bwd_with_recompute_us": round(pass_us(lambda: [st.xpipe_stage_bwd(xs[0][i], None if dys is None else dys[0][i],
                                                                           None if labels is None else labels[0][i], dx)
                                                        for i in range(w.T)]), 1)}
    time_stage.passes = passes
    # per-kernel durations with HIP events around every launch, over the same
    # number of steps: the timed step's launches (with the forward stream set,
    # the chained forwards), all on the stage's stream
    if fs is not None:
        st.xpipe_stage_set_fwd_stream(True)
    st.set_timing(True)
    for j in range(steps):
        step(j)
    torch.cuda.synchronize()
    classes = st.timing()
    st.set_timing(False)
    torch.cuda.synchronize()
    fin = bool(torch.isfinite(st.W).all().item()) and (not w.has_loss or bool(torch.isfinite(loss).all().item()))
    return w, ms, wall, classes, fin


def time_interleaved(args, minibatches=6):
    """One GPU's part of the interleaved pipeline schedule (xpipe_schedule +
    xpipe_stage_run) on the same stage: the workload's rank of its pipeline,
    each micro-batch its own input buffer, bellwether predictions cached across
    updates.  Returns samples/s over the run (after one untimed run that also
    records the passes)."""
    import torch
    import paper_1911_04610_amd as xp
    import workloads as wl
    w = wl.WORKLOADS[args.workload]()
    dt = xp.BF16 if args.dtype == "bf16" else xp.F32
    tdt = torch.bfloat16 if dt == xp.BF16 else torch.float32
    inp = wl.stage_inputs(w, act_dtype=args.dtype if args.dtype == "bf16" else "f32", moment_init="paper")
    st = xp.Stage(w.layers, w.micro_batch, w.T, w.in_shape, dt)
    st.set_flat(st.W, inp.params)
    st.set_flat(st.m, inp.m)
    st.set_flat(st.v, inp.v)
    J = len(inp.xs)
    n = w.T * minibatches
    dev = lambda a: torch.from_numpy(a).cuda().to(tdt)
    xs = [dev(inp.xs[(k // w.T) % J][k % w.T]) for k in range(n)]
    labels = None if inp.labels is None else [torch.from_numpy(inp.labels[(k // w.T) % J][k % w.T]).cuda()
                                              for k in range(n)]
    dys = None if inp.dys is None else [dev(inp.dys[(k // w.T) % J][k % w.T]) for k in range(n)]
    nb, H, W_, C = st.out_shape
    ys = [torch.empty((nb, H, W_, C), dtype=tdt, device="cuda") for _ in range(n)]
    dxs = [torch.empty_like(x) for x in xs] if w.rank > 0 else None
    loss = torch.zeros(n, dtype=torch.float32, device="cuda") if w.has_loss else None
    events = xp.xpipe_schedule(w.size, w.T, w.rank, minibatches)
    hp = xp.Hyper()
    run = lambda t: st.xpipe_stage_run(events, xs, ys, hp, t, dy=dys, labels=labels, loss=loss, dx=dxs)
    # forwards on a stream of the stage's own, beside the backwards
    stream = torch.cuda.current_stream()
    fs = st.xpipe_stage_set_fwd_stream(True)
    run(0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    fs.wait_stream(stream)
    run(minibatches)
    stream.wait_stream(fs)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    return {"size": w.size, "rank": w.rank, "T": w.T, "minibatches": minibatches,
            "samples_per_s": round(n * w.micro_batch / (ms / 1e3), 2),
            "ms_per_minibatch": round(ms / minibatches, 4),
            "note": "interleaved one-forward-one-backward order of this rank, forwards on their "
                    "own stream; a prediction per bellwether and direction, updates kept separate "
                    "from predictions"}


def time_partitioned(args, net, stages=4, steps=10, warmup=3):
    """A whole network split into `stages` stages by the paper's partition rule
    (xpipe_partition), each stage trained on its own as its GPU would (T
    forward/backward pairs, the forwards on the stage's forward stream and the
    backwards with recomputation, Adam fused with the next predictions; bf16).  Reports each stage's step time and the pipeline's
    steady-state throughput bound, the slowest stage's (synthetic inputs and
    upstream gradients of each stage's shapes).  VGG-16: CIFAR-10 images
    (32 x 32), micro-batch 32, T = 4 (mini-batch 128).  ResNet-101 and
    Inception-V3: Tiny ImageNet images scaled to 224 x 224, 200 classes,
    micro-batch 100 (the paper's 4-GPU setting), T = 4."""
    import numpy as np
    import torch
    import paper_1911_04610_amd as xp
    import workloads as wl
    if net == "vgg16":
        layers, in_shape, mb, T = wl.vgg16_layers(), (32, 32, 3), 32, 4
        model = "vgg16 (32x32 inputs, 13 conv + linear)"
    elif net == "resnet101":
        layers, in_shape, mb, T = wl.resnet101_layers(), (224, 224, 3), 100, 4
        model = "resnet101 (224x224 inputs, 200 classes, 104 conv + linear)"
    else:
        layers, in_shape, mb, T = wl.inception_v3_layers(), (224, 224, 3), 100, 4
        model = "inception_v3 (224x224 inputs, 200 classes, 94 conv + linear, no auxiliary head)"
    first = xp.xpipe_partition(layers, stages)
    parts = wl.split_layers(layers, first)
    rng = np.random.default_rng(wl.PAPER_SEED + 7)
    res = []
    hp = xp.Hyper()
    for k, p in enumerate(parts):
        st = xp.Stage(p, mb, T, in_shape, xp.BF16)
        st.set_flat(st.W, wl.init_params(p, rng))
        n, H, W_, C = st.out_shape
        last = k == len(parts) - 1
        x = torch.randn((mb,) + tuple(in_shape), device="cuda").to(torch.bfloat16)
        y = torch.empty((n, H, W_, C), dtype=torch.bfloat16, device="cuda")
        dy = None if last else (1e-2 * torch.randn((n, H, W_, C), device="cuda")).to(torch.bfloat16)
        lab = torch.from_numpy(rng.integers(0, C if last else 10, mb).astype(np.int32)).cuda() if last else None
        loss = torch.zeros(1, dtype=torch.float32, device="cuda") if last else None
        dx = torch.empty_like(x) if k > 0 else None
        st.xpipe_predict_weights(xp.FWD, 1, hp, 0)
        st.xpipe_predict_weights(xp.BWD, 1, hp, 0)
        state = {"t": 0}
        stream = torch.cuda.current_stream()
        fs = st.xpipe_stage_set_fwd_stream(True)  # forwards beside the backwards

        def step():
            for _ in range(T):
                st.xpipe_stage_fwd(x, y, lab, loss)
                st.xpipe_stage_bwd(x, dy, lab, dx)
            st.xpipe_adam_step(hp, state["t"], 1, 1, emit_pred=True)
            state["t"] += 1

        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fs.wait_stream(stream)
        for _ in range(steps):
            step()
        stream.wait_stream(fs)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        res.append({"layers": [first[k], first[k + 1]], "in_shape": list(in_shape),
                    "params": int(st.P), "ms_per_step": round(ms, 4),
                    "samples_per_s": round(mb * T / (ms / 1e3), 1)})
        in_shape = (H, W_, C)
        del st, x, y, dy, dx
        torch.cuda.empty_cache()
    slow = max(r["ms_per_step"] for r in res)
    return {"model": model, "stages": stages, "micro_batch": mb, "T": T,
            "dtype": "bf16", "per_stage": res,
            "pipeline_samples_per_s_bound": round(mb * T / (slow / 1e3), 1),
            "note": "each stage timed alone on this GPU as its pipeline GPU would run it; the "
                    "pipeline's steady-state rate is bounded by its slowest stage"}


def event_offset_us(reps=300):
    """Per-launch offset of a start/stop event pair around one kernel: the
    bracketed time of a ~10 us kernel minus its period when launched back to
    back (then the kernel's own duration, as it is longer than the launch
    floor).  Subtracted from the per-kernel event averages so they measure
    what the kernel-trace profiler reports."""
    import torch
    t = torch.zeros(1 << 23, device="cuda")
    s = torch.cuda.current_stream()
    for _ in range(20):
        t.add_(1)
    torch.cuda.synchronize()
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(reps)]
    for a, b in pairs:
        a.record(s)
        t.add_(1)
        b.record(s)
    torch.cuda.synchronize()
    bracket = sum(a.elapsed_time(b) for a, b in pairs) / reps * 1e3
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(reps):
        t.add_(1)
    b.record(s)
    torch.cuda.synchronize()
    period = a.elapsed_time(b) / reps * 1e3
    return max(0.0, bracket - period), bracket, period


def time_sweep(n, steps):
    """Prediction and Adam over n flat fp32 parameters at t = 100."""
    import numpy as np
    import torch
    import paper_1911_04610_amd as xp
    import workloads as wl
    s = wl.flat_state(n)
    W, m, v, G = (torch.from_numpy(a).cuda() for a in (s.W, s.m, s.v, s.G))
    out = torch.empty_like(W)
    pf, pb = torch.empty_like(W), torch.empty_like(W)
    hp = xp.Hyper()
    res = {}

    def timed(fn, reps):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    # at least 50 calls (>= 12 ms for the shortest pass) per timed window
    reps = max(50, steps)
    for sv in (0, 1, 2, 3, 7):
        ms = timed(lambda: xp.xpipe_predict_flat(W, m, v, out, None, sv, hp, 100), reps)
        res[f"predict_s{sv}"] = {"ms": ms, "GB_s": 16.0 * n / ms / 1e6}
    ms = timed(lambda: xp.xpipe_adam_flat(W, m, v, G, hp, 100, False), reps)
    res["adam"] = {"ms": ms, "GB_s": 28.0 * n / ms / 1e6}
    ms = timed(lambda: xp.xpipe_adam_flat(W, m, v, G, hp, 100, True, pf, 2, pb, 1), reps)
    res["adam_zero_grad_2pred"] = {"ms": ms, "GB_s": 40.0 * n / ms / 1e6}
    # the other update rules with Adam-moment prediction, fused the same way:
    # momentum SGD 36 B/param (W, buf, m, v, G in; W, buf, m, v out) + zero + 2 predictions
    # = 48; RMSProp adds the squared average (44 + 12 = 56)
    buf, sq = (torch.from_numpy(a).cuda() for a in wl.rule_state(n))
    s_extra = torch.empty_like(W)
    rule = xp.Rule(rule=xp.RULE_MOMENTUM_SGD, lr=1e-2, momentum=0.9, weight_decay=5e-4)
    ms = timed(lambda: xp.xpipe_rule_flat(W, buf, None, m, v, G, rule, hp, 100, True, pf, 2, pb, 1), reps)
    res["momentum_sgd_zero_grad_2pred"] = {"ms": ms, "GB_s": 48.0 * n / ms / 1e6}
    rule = xp.Rule(rule=xp.RULE_RMSPROP, lr=1e-4, momentum=0.9, alpha=0.99, eps=1e-8)
    ms = timed(lambda: xp.xpipe_rule_flat(W, buf, sq, m, v, G, rule, hp, 100, True, pf, 2, pb, 1), reps)
    res["rmsprop_zero_grad_2pred"] = {"ms": ms, "GB_s": 56.0 * n / ms / 1e6}
    # the attainable rate of each pass's access pattern on this GPU: a bare
    # stream with the same numbers of 16-byte reads and writes per element
    ceil = {}
    for key, (nr, nw) in {"predict": (3, 1), "adam": (4, 3), "adam_zero_grad_2pred": (4, 6)}.items():
        srcs = [W, m, v, G][:nr]
        dsts = [out, pf, pb, buf, sq, s_extra][:nw]
        ms = timed(lambda: xp.xpipe_probe_stream(srcs, dsts), reps)
        ceil[key] = {"reads": nr, "writes": nw, "ms": ms, "GB_s": 4.0 * (nr + nw) * n / ms / 1e6}
    res["stream_ceiling"] = ceil
    for k in list(res):
        base = "predict" if k.startswith("predict_s") else k
        if base in ceil:
            res[k]["frac_of_stream_ceiling"] = round(res[k]["GB_s"] / ceil[base]["GB_s"], 4)
    del W, m, v, G, out, pf, pb, buf, sq, s_extra
    torch.cuda.empty_cache()
    return res


def measured_peaks():
    """Attainable peaks on this GPU from the library's probes: a 1 GiB 16-byte
    copy (read + write bytes) and back-to-back bf16 MFMAs on registers."""
    import torch
    import paper_1911_04610_amd as xp

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    n = 1 << 30
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ms = timed(lambda: xp.xpipe_probe_copy(src, dst))
    copy_gbs = 2.0 * n / (ms / 1e3) / 1e9
    del src, dst
    waves, iters = 256 * 4 * 2, 4096
    out = torch.empty(waves, dtype=torch.float32, device="cuda")
    ms = timed(lambda: xp.xpipe_probe_mfma(out, iters))
    tflops = waves * iters * 8 * 32768.0 / (ms / 1e3) / 1e12
    return {"hbm_copy_GB_s": round(copy_gbs, 1), "mfma_bf16_TFLOP_s": round(tflops, 1),
            "copy_bytes": 2 * n, "mfma": "v_mfma_f32_32x32x16_bf16, %d waves x %d x 8" % (waves, iters)}


def graph_costs():
    """What the launch lanes cost inside a recorded graph: microseconds per
    diamond (one launch, `width` branches of `len` launches on other streams,
    joined back) against the same launches as one chain, for empty launches
    and for launches of about 28 us (256 workgroups, 2000 dependent FMAs per
    thread)."""
    import torch
    import paper_1911_04610_amd as xp
    scratch = torch.zeros(2048, dtype=torch.float32, device="cuda")
    res = []
    for spin in (0, 2000):
        for width, length in ((1, 1), (2, 1), (3, 1), (2, 3)):
            par, ser = xp.xpipe_probe_graph(scratch, width, length, 40, spin)
            res.append({"spin": spin, "width": width, "len": length, "launches": 1 + width * length,
                        "branches_us": round(par, 2), "chain_us": round(ser, 2)})
    return res


def vendor_reference(off_us, reps=50):
    """The stage's convolution shapes (32 x 35 x 35 NHWC, bf16) against the
    vendor libraries, per launch, with HIP events over back-to-back launches.
    Forward: this library's implicit GEMM (forward of a one-convolution
    stage: one k_conv_gemm launch), MIOpen's convolution through torch
    (channels-last), and hipBLASLt's plain GEMM of the same M x K x N through
    torch.mm (no im2col: the library GEMM reads a ready K-major operand, which
    the convolution does not have).  Weight gradient: this library's
    k_wgrad_t plus its split reduction (per-launch events in the one-
    convolution stage's backward, event offset removed) against MIOpen's
    backward-weights convolution.  Context for the MFMA fraction of these
    skinny shapes, not a dependency: the stage itself never calls the vendor
    libraries."""
    import numpy as np
    import torch
    import paper_1911_04610_amd as xp
    import workloads as wl

    def timed(fn):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e3

    torch.backends.cudnn.benchmark = True  # MIOpen picks its fastest algorithm per shape
    out = []
    nb, H, W = 32, 35, 35
    for cin, cout, k in ((64, 96, 3), (96, 96, 3), (48, 64, 5), (256, 176, 1)):
        b = wl._Builder()
        b.conv(-1, cin, cout, k)
        st = xp.Stage(b.layers, nb, 1, (H, W, cin), xp.BF16, stream=torch.cuda.current_stream())
        rng = np.random.default_rng(wl.PAPER_SEED + 9)
        st.set_flat(st.W, wl.init_params(b.layers, rng))
        hp = xp.Hyper()
        st.xpipe_predict_weights(xp.FWD, 0, hp, 0)
        st.set_graphs(False)
        x = torch.randn(nb, H, W, cin, device="cuda").to(torch.bfloat16)
        y = torch.empty(nb, H, W, cout, device="cuda", dtype=torch.bfloat16)
        ours = timed(lambda: st.xpipe_stage_fwd(x, y))
        st.set_timing(True)
        st.xpipe_stage_fwd(x, y)
        torch.cuda.synchronize()
        launched = sorted(st.timing())
        st.set_timing(False)
        xc = x.permute(0, 3, 1, 2)  # NCHW view of the NHWC data: channels-last
        wt = torch.randn(cout, cin, k, k, device="cuda").to(torch.bfloat16).to(memory_format=torch.channels_last)
        miopen = timed(lambda: torch.nn.functional.conv2d(xc, wt, padding=k // 2))
        M, K = nb * H * W, k * k * cin
        A = torch.randn(M, K, device="cuda").to(torch.bfloat16)
        B = torch.randn(K, cout, device="cuda").to(torch.bfloat16)
        blas = timed(lambda: A @ B)
        fl = 2.0 * M * cout * K
        # weight gradient: the backward of the one-convolution stage (no input
        # gradient); only its weight-gradient launches are counted
        st.xpipe_predict_weights(xp.BWD, 0, hp, 0)
        dy = torch.randn(nb, H, W, cout, device="cuda").to(torch.bfloat16)
        for _ in range(3):
            st.xpipe_stage_bwd(x, dy)
        torch.cuda.synchronize()
        st.set_timing(True)
        for _ in range(reps):
            st.xpipe_stage_bwd(x, dy)
        torch.cuda.synchronize()
        tm = st.timing()
        st.set_timing(False)
        wl_names = sorted(n for n in tm if n.startswith(("k_wgrad", "k_split_reduce")))
        ours_wg = sum(tm[n][0] * 1e3 - off_us * tm[n][1] for n in wl_names) / reps
        dyc = dy.permute(0, 3, 1, 2)
        miopen_wg = timed(lambda: torch.ops.aten.convolution_backward(
            dyc, xc, wt, None, [1, 1], [k // 2, k // 2], [1, 1], False, [0, 0], 1, [False, True, False]))
        out.append({"shape": f"conv {k}x{k} {cin}->{cout}, 32x35x35 NHWC bf16 (M={M}, N={cout}, K={K})",
                    "ours_us": round(ours, 2), "ours_launches": launched, "miopen_conv_us": round(miopen, 2),
                    "hipblaslt_gemm_us": round(blas, 2),
                    "ours_TFLOP_s": round(fl / ours / 1e6, 1),
                    "miopen_TFLOP_s": round(fl / miopen / 1e6, 1),
                    "hipblaslt_TFLOP_s": round(fl / blas / 1e6, 1),
                    "wgrad_ours_us": round(ours_wg, 2), "wgrad_ours_launches": wl_names,
                    "wgrad_miopen_us": round(miopen_wg, 2),
                    "wgrad_ours_TFLOP_s": round(fl / ours_wg / 1e6, 1),
                    "wgrad_miopen_TFLOP_s": round(fl / miopen_wg / 1e6, 1)})
        del st
    return out


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, dtype, sweep_n=10_000_000):
    """The oracle as it stands, on the host: one whole step of the same stage
    (both predictions, T forwards, T backwards with recomputation and the Adam
    update: the oracle's mini-batch driver, one mini-batch) with the BLAS
    thread pool at its default size, the first micro-batch's forward alone on
    one thread, and the oracle's prediction and Adam passes over sweep_n flat
    parameters (the 1e8-parameter sweep's distributions, a tenth of its size)
    on one thread and on all."""
    import numpy as np
    import oracle
    import workloads as wl
    from threadpoolctl import threadpool_info, threadpool_limits
    info = threadpool_info()
    threads = max((i.get("num_threads", 0) for i in info), default=0) or os.cpu_count()
    storage = "bf16" if dtype == "bf16" else "f32"
    inp = wl.stage_inputs(w, act_dtype=storage, moment_init="paper")
    st = oracle.Stage(w.layers, storage)
    t0 = time.perf_counter()
    oracle.train_stage(st, inp.params, inp.m, inp.v, inp.xs, w.s_fwd, w.s_bwd, oracle.Hyper(),
                       labels=inp.labels, dys=inp.dys, need_dx=w.rank > 0, minibatches=1, t0=1)
    sec = time.perf_counter() - t0
    samples = w.T * w.micro_batch
    with threadpool_limits(limits=1):
        t1 = time.perf_counter()
        st.forward(inp.params, inp.xs[0][0], None if inp.labels is None else inp.labels[0][0],
                   samples)
        fwd1 = time.perf_counter() - t1
    fs = wl.flat_state(sweep_n)
    W, m, v, G = (a.astype(np.float64) for a in (fs.W, fs.m, fs.v, fs.G))
    hp = oracle.Hyper()

    def sweep():
        t1 = time.perf_counter()
        oracle.predict(W, m, v, 100, 2, hp.lr, hp.beta1, hp.beta2, hp.eps)
        tp = time.perf_counter() - t1
        t1 = time.perf_counter()
        oracle.adam_update(W, m, v, G, 101, hp.lr, hp.beta1, hp.beta2, hp.eps)
        ta = time.perf_counter() - t1
        # the GPU passes' algorithmic bytes at fp32 storage: predict 16 B/param, Adam 28
        return {"predict_GB_s": round(16.0 * sweep_n / tp / 1e9, 3),
                "adam_GB_s": round(28.0 * sweep_n / ta / 1e9, 3)}

    with threadpool_limits(limits=1):
        sw1 = sweep()
    swn = sweep()
    return {"value": round(samples / sec, 3), "unit": "samples/s", "cores": int(threads),
            "kind": "oracle", "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": (f"one full step ({samples} samples: 2 predictions, {w.T} forwards, {w.T} "
                       f"backwards with recompute, Adam) of the same stage in fp64 numpy with "
                       f"{storage} storage rounding; {sec:.1f} s on {threads} BLAS threads"),
            "single_thread": {"forward_one_micro_batch_s": round(fwd1, 3),
                              "samples_per_s": round(w.micro_batch / fwd1, 3),
                              "note": "forward of one micro-batch only, one thread"},
            "predict_adam_sweep": {"n_params": sweep_n, "one_thread": sw1, "all_threads": swn,
                                   "note": "numpy element-wise passes run on one thread either way"}}


def is_gemm(name):
    return name.startswith(("k_conv_gemm", "k_conv_direct", "k_wgrad"))


class KernelTable:
    """Per-kernel event timings of a timing pass (name -> (ms, launches, work))
    with the per-launch event offset removed: average launch time, achieved
    rate and roofline fraction (GEMMs against the MFMA peak of the type they
    multiply in, everything else against HBM)."""

    def __init__(self, classes, steps, off_us, peak_key):
        self.c, self.steps, self.off_us, self.peak_key = classes, steps, off_us, peak_key

    def ms(self, k):
        kms, kn, _ = self.c[k]
        return max(kms - kn * self.off_us / 1e3, 1e-9)

    def dominant(self, pred=lambda k: True):
        ks = [k for k in self.c if pred(k)]
        return max(ks, key=self.ms) if ks else None

    def roofline(self, k):
        kms, kn, kwork = self.c[k]
        ms = self.ms(k)
        if is_gemm(k):
            ach = kwork / (ms / 1e3) / 1e12
            peak = PEAK_TFLOPS[self.peak_key]
            r = {"bound": "mfma", "achieved": round(ach, 3), "peak": peak, "unit": "TFLOP/s",
                 "frac": round(ach / peak, 5)}
        else:
            ach = kwork / (ms / 1e3) / 1e9
            r = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": round(ach / HBM_PEAK_GBS, 4)}
        r.update({"kernel": k, "launches_per_step": kn / self.steps,
                  "avg_launch_us": round(1e3 * ms / max(kn, 1), 3),
                  "avg_launch_us_raw_events": round(1e3 * kms / max(kn, 1), 3),
                  "work_per_launch": kwork / max(kn, 1)})
        return r

    def summary(self, k):
        r = self.roofline(k)
        return {"kernel": k, "ms_per_step": round(self.ms(k) / self.steps, 4),
                "launches_per_step": r["launches_per_step"], "avg_us": round(r["avg_launch_us"], 2),
                "achieved": r["achieved"], "unit": r["unit"], "frac": r["frac"]}

    def top(self, n):
        return sorted(self.c, key=lambda k: -self.ms(k))[:n]

    def all_gemm_frac(self):
        ms = sum(self.ms(k) for k in self.c if is_gemm(k))
        work = sum(self.c[k][2] for k in self.c if is_gemm(k))
        return round(work / (ms / 1e3) / 1e12 / PEAK_TFLOPS[self.peak_key], 5) if ms > 0 else None

    def launches_per_step(self):
        return sum(v[1] for v in self.c.values()) / self.steps


def config_legs(args, off_us):
    """The other stage configurations, each timed the same way as the main
    line (whole steps with HIP events, then a per-kernel timing pass): the
    Tiny MLP (fp32, micro-seconds per step: launch-bound, no roofline), the
    VGG-16 first stage (bf16 and fp32, s_f = 2 and the half-down reading's 1),
    the ResNet middle stage and the Inception-A stage in both storage types.
    fp32 storage multiplies on fp64 MFMA, so its GEMMs are held to the fp64
    peak."""
    legs = [("tiny_mlp", "f32", None), ("vgg16_stage0", "bf16", None), ("vgg16_stage0", "bf16", 1),
            ("vgg16_stage0", "f32", None), ("vgg16_stage0", "f32", 1),
            ("resnet101_mid_stage", "bf16", None), ("resnet101_mid_stage", "f32", None),
            ("inception_v3_stage", "f32", None)]
    out = []
    for name, dt, sf in legs:
        w, ms, wall, classes, fin = time_stage(args, workload=name, dtype=dt, s_fwd=sf,
                                               steps=max(10, min(args.steps, 20)), warmup=3)
        steps = max(10, min(args.steps, 20))
        tab = KernelTable(classes, steps, off_us, "bf16" if dt == "bf16" else "f64")
        samples = w.T * w.micro_batch
        leg = {"workload": name, "dtype": dt, "micro_batch": w.micro_batch, "T": w.T,
               "s_fwd": w.s_fwd, "s_bwd": w.s_bwd, "ms_per_step": round(ms, 4),
               "samples_per_s": round(samples / (ms / 1e3), 1), "finite": fin,
               "launches_per_step": tab.launches_per_step()}
        if name == "tiny_mlp":
            leg["us_per_step"] = round(ms * 1e3, 1)
        else:
            dom = tab.dominant()
            leg["roofline"] = tab.roofline(dom)
            cg = tab.dominant(lambda k: k.startswith(("k_conv_gemm", "k_conv_direct")))
            wg = tab.dominant(lambda k: k.startswith("k_wgrad"))
            leg["roofline_conv_gemm"] = tab.roofline(cg) if cg else None
            leg["roofline_weight_gradient"] = tab.roofline(wg) if wg else None
            leg["mfma_util_all_gemm"] = tab.all_gemm_frac()
        leg["top_kernels"] = [tab.summary(k) for k in tab.top(5)]
        out.append(leg)
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this library runs one pipeline stage on one GPU; --gpus must be 1 "
                                   "(each pipeline stage would run as its own one-GPU process)"}))
        sys.exit(2)
    if args.traffic_summarize:
        traffic_summarize(*args.traffic_summarize)
        return
    import torch
    import paper_1911_04610_amd as xp
    torch.cuda.set_device(0)
    if args.traffic_run:
        traffic_run(args)
        return
    w, ms, wall, classes, finite = time_stage(args)
    samples = w.T * w.micro_batch
    value = samples / (ms / 1e3)
    peak_key = "bf16" if args.dtype == "bf16" else "f64"
    off_us, off_bracket, off_period = event_offset_us()
    tab = KernelTable(classes, args.steps, off_us, peak_key)
    # the dominant kernel: largest summed launch time once the per-launch
    # event offset is removed (what the kernel-trace profiler ranks by)
    dom = tab.dominant()
    rf = tab.roofline(dom)
    rf.update({"traffic": stored_traffic(dom), "traffic_unit": "bytes per launch",
               "event_offset_us": round(off_us, 3)})
    wg = tab.dominant(lambda k: k.startswith("k_wgrad"))
    cg = tab.dominant(lambda k: k.startswith(("k_conv_gemm", "k_conv_direct")))
    top = tab.top(12)
    out = {
        "metric": "stage samples/sec (predict+fwd+bwd+Adam); predict/Adam HBM GB/s; MFMA util",
        "value": round(value, 2),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic (seeded N(0,1) inputs, Kaiming-uniform weights, paper moment init)",
        "config": {"workload": w.name, "micro_batch": w.micro_batch, "T": w.T,
                   "mini_batch": samples, "input_hwc": list(w.in_shape), "s_fwd": w.s_fwd,
                   "s_bwd": w.s_bwd, "rank": w.rank, "size": w.size,
                   "update": "adam fused with next predictions", "parallelism": "one stage, 1 GPU"},
        "roofline": rf,
        "roofline_conv_gemm": tab.roofline(cg) if cg else None,
        "roofline_weight_gradient": tab.roofline(wg) if wg else None,
        "mfma_util_all_gemm": tab.all_gemm_frac(),
        "launches_per_step": tab.launches_per_step(),
        "kernels_timed_sum_ms_per_step": round(sum(v[0] for v in classes.values()) / args.steps, 4),
        "pass_us_per_micro_batch": getattr(time_stage, "passes", None),
        "top_kernels": [tab.summary(k) for k in top],
        "finite": finite,
    }
    pk = measured_peaks()
    if not args.no_sweep:
        # (left out with --no-sweep: its spin launches would dominate a kernel trace)
        pk["graph_fork_join"] = graph_costs()
    out["peaks_measured"] = pk
    if rf["unit"] == "TFLOP/s" and peak_key == "bf16":
        rf["frac_of_measured_peak"] = round(rf["achieved"] / pk["mfma_bf16_TFLOP_s"], 5)
    elif rf["unit"] == "GB/s":
        rf["frac_of_measured_peak"] = round(rf["achieved"] / pk["hbm_copy_GB_s"], 4)
    if not args.no_sweep:
        sw = time_sweep(args.sweep_n, args.steps)
        ceil = sw.pop("stream_ceiling")
        out["predict_adam_sweep"] = {"n_params": args.sweep_n, "t": 100,
                                     **{k: {"ms": round(v["ms"], 4), "GB_s": round(v["GB_s"], 1),
                                            "frac_hbm": round(v["GB_s"] / HBM_PEAK_GBS, 4),
                                            "frac_measured_copy": round(v["GB_s"] / pk["hbm_copy_GB_s"], 4),
                                            **({"frac_of_stream_ceiling": v["frac_of_stream_ceiling"]}
                                               if "frac_of_stream_ceiling" in v else {})}
                                        for k, v in sw.items()},
                                     "stream_ceiling": {k: {"reads": v["reads"], "writes": v["writes"],
                                                            "GB_s": round(v["GB_s"], 1),
                                                            "frac_hbm": round(v["GB_s"] / HBM_PEAK_GBS, 4)}
                                                        for k, v in ceil.items()}}
    if not args.no_sweep:
        out["interleaved_schedule"] = time_interleaved(args)
        out["vgg16_partitioned"] = time_partitioned(args, "vgg16")
        out["resnet101_partitioned"] = time_partitioned(args, "resnet101")
        out["inception_v3_partitioned"] = time_partitioned(args, "inception_v3")
        out["vendor_reference"] = vendor_reference(off_us)
    if not args.no_legs:
        out["configs"] = config_legs(args, off_us)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.dtype)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
