"""Benchmark: one training step of the CosmoFlow conv hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--extra-workload NAME|none]
                    [--no-cpu-baseline]

A step is the whole hot path over one batch of synthetic cubes: forward
(conv, bias + leaky ReLU, 2^3 average pool per layer) and backward (pool
backward, leaky-ReLU backward + bias grad, weight grad, data grad) through
the C ABI.  Inputs, weights and the upstream gradient are resident in HBM
before timing starts.  Warm-up: the W steps, then untimed steps until 0.3 s
have passed (the GPU's clocks need tens of milliseconds of sustained work to
settle).  Prints ONE JSON line.

value = algorithmic conv FLOPs per step (fwd + wgrad + dgrad, padded taps
included, layer-1 dgrad skipped) x steps / wall time of the timed steps, for
the headline workload: the 128^3 stack at the paper's precision (fp32, batch
1, as Table I times it).  The same measurement of the bf16 batch-8 128^3
stack is reported under its own key.  The roofline entry is for the op that
takes the most time per step, timed with events on the launch stream over
the same timed steps.

The parameter update that follows each step in training (Adam + LARC +
linear decay, Section III-B) is timed on its own after the timed steps and
reported under "update"; --with-update also runs it inside every step.
The fully-connected head and loss on the stack's output (three FC layers
with leaky ReLU, mean squared error) is likewise timed on its own and
reported under "head"; --with-head runs it inside every step, the stack's
upstream gradient then being the loss gradient instead of a fixed N(0,1)
tensor.
"hbm_passes" times the unfused elementwise and pooling kernels alone at the
first layer's activation shape.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK = {"bf16": 2516.6, "f32": 157.3}  # dense MFMA TFLOP/s, MI355X
HBM_PEAK_GBS = 8000.0
METRIC = "fwd+bwd 3D-conv TFLOP/s & samples/s, 128^3 CosmoFlow stack; % MFMA peak"
RAMP_S = 0.3  # minimum seconds of untimed warm-up work (clock ramp), after the W warm-up steps


def describe(name, wl):
    pads = {L.get("pad", "same") for L in wl["layers"]}
    pad = "TF-SAME padding" if pads == {"same"} else "VALID padding" if pads == {"valid"} else "mixed padding"
    pooled = sum(1 for L in wl["layers"] if L["pool"])
    what = "CosmoFlow conv stack" if name.startswith("stack") else "the paper's first three conv layers"
    return (f"{what}, {wl['size']}^3 x {wl['c0']} input, batch {wl['batch']}, {wl['dtype']}, "
            f"{len(wl['layers'])} conv layers ({pooled} pooled), {pad}, fwd+bwd")


def cpu_baseline(name, seconds_hint=True):
    """Time the oracle (fp64 CPU) on one sample of the workload: forward and
    backward of every layer (layer-1 dgrad skipped, like the GPU step)."""
    import numpy as np

    import oracle
    from paper_1808_04728_amd import inputs

    wl = dict(inputs.WORKLOADS[name])
    x = inputs.make_input(name)[:1]
    ws, bs = inputs.make_weights(name)
    layers = [dict(k=L["k"], stride=L["stride"], pool=L["pool"], pad=L.get("pad", "same")) for L in wl["layers"]]
    oracle.build(force=False)
    # one sample's step, repeated until about 10 s of CPU work
    reps, t0 = 0, time.perf_counter()
    while True:
        acts = oracle.stack_forward(x, layers, ws, bs, inputs.ALPHA)
        dout = inputs.normal(acts[-1]["out"].shape, 30000 + wl["cfg"])
        oracle.stack_backward(acts, layers, ws, dout, inputs.ALPHA, skip_first_dgrad=True)
        reps += 1
        if time.perf_counter() - t0 > 10.0 or reps >= 8:
            break
    dt = (time.perf_counter() - t0) / reps
    flops = 0
    size = wl["size"]
    for i, L in enumerate(wl["layers"]):
        out = -(-size // L["stride"]) if L.get("pad", "same") == "same" else (size - L["k"]) // L["stride"] + 1
        macs = out ** 3 * L["cout"] * L["k"] ** 3 * L["cin"]
        flops += 2 * macs * (2 if i == 0 else 3)
        size = out // 2 if L["pool"] else out
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or os.cpu_count()
    return dict(value=flops / dt / 1e12, unit="TFLOP/s", cores=threads, kind="oracle",
                sample=f"1 of {wl['batch']} samples (batch 1), full {wl['size']}^3 stack fwd+bwd in fp64, "
                       f"{reps} repetitions, {dt:.2f} s each, {1.0 / dt:.4f} samples/s")


def measured_traffic(workload, op):
    """HBM bytes per launch of `op` from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy), or None when
    there is none for this op or a source it was measured on has changed."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hbm_traffic.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        if not line.startswith("traffic:"):
            continue
        kv = dict(t.split("=", 1) for t in line.split()[1:])
        if kv.get("workload") != workload or kv.get("op") != op:
            continue
        for spec in kv["sources"].split(","):
            f, h = spec.rsplit(":", 1)
            fp = os.path.join(ROOT, f)
            if not os.path.exists(fp) or hashlib.sha256(open(fp, "rb").read()).hexdigest()[:len(h)] != h:
                return None
        return int(kv["bytes"])
    return None


def copy_probe(mib):
    """A plain copy of known size: what the FETCH_SIZE / WRITE_SIZE counters
    read for it is the scale that turns their readings into HBM bytes."""
    import torch

    torch.cuda.set_device(0)
    src = torch.ones(mib << 20, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": mib << 20, "copies": 5}), flush=True)


def update_at_paper_size(step, B, np, torch, bf16):
    """The update over as many parameters as the paper's network holds
    (28.15 MB of fp32, Section IV: about 7.04 M) in 20 groups of seeded sizes
    (its layer widths are not recoverable), queued behind a step; there the
    pass is bound by HBM bandwidth, not latency."""
    total = 7_037_500
    r = np.random.default_rng(11)
    w = r.uniform(0.2, 1.0, 20)
    sizes = np.floor(w / w.sum() * total).astype(np.int64) // 4 * 4
    off = [0] + np.cumsum(sizes).tolist()
    n = off[-1]
    v = torch.randn(n, device="cuda:0") * 0.05
    g = torch.randn(n, device="cuda:0")
    m = torch.zeros(n, device="cuda:0")
    s = torch.zeros(n, device="cuda:0")
    v16 = torch.empty(n, dtype=torch.bfloat16, device="cuda:0") if bf16 else None
    ws = torch.empty(max(B.cf_adam_larc_workspace_size(off), 16), dtype=torch.uint8, device="cuda:0")
    offc = B.adam_offsets(off)
    hp = B.make_hparams(100000)
    times = []
    for rep in range(3):
        step()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for t in range(10):
            B.cf_adam_larc_step(offc, 10 * rep + t, hp, v, g, m, s, v16, ws)
        e1.record()
        times.append((e0, e1))
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in times])) / 10
    nbytes = n * (28 + (2 if bf16 else 0))
    gbs = nbytes / (ms * 1e-3) / 1e9
    return dict(params=n, groups=20, launch_ms=round(ms, 4), algorithmic_bytes=nbytes, achieved=round(gbs, 1),
                frac=round(gbs / HBM_PEAK_GBS, 4))


def hbm_passes(B, np, torch, wl):
    """The unfused elementwise and pooling passes (bias + leaky ReLU forward and
    backward, 2^3 average pool forward and backward) at the first layer's
    activation shape of the workload, each timed alone: 10 launches back to
    back on resident tensors, HIP events around them.  Inside the unfused step
    the same kernels also absorb the write-back of the previous kernel's
    output, so their in-sequence times (--unfused --op-breakdown) are longer."""
    dt = wl["dtype"]
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    n, s, c = wl["batch"], wl["size"], wl["layers"][0]["cout"]
    nvox = n * s ** 3
    dev = "cuda:0"
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    z = torch.randn((n, s, s, s, c), generator=g, device=dev).to(tdt)
    y = torch.empty_like(z)
    dy = torch.randn((n, s, s, s, c), generator=g, device=dev).to(tdt)
    dz = torch.empty_like(z)
    dp = torch.randn((n, s // 2, s // 2, s // 2, c), generator=g, device=dev).to(tdt)
    pool = torch.empty_like(dp)
    dy2 = torch.empty_like(z)
    bias = torch.zeros(c, device=dev)
    db = torch.empty(c, device=dev)
    ws = torch.empty(max(B.cf_bias_lrelu_bwd_workspace_size(nvox, c), 16), dtype=torch.uint8, device=dev)
    zb = z.numel() * z.element_size()
    pb = pool.numel() * pool.element_size()
    ops = {
        "bias_lrelu_fwd": (lambda: B.cf_bias_lrelu_fwd(nvox, c, dt, z, bias, 0.01, y), 2 * zb),
        "bias_lrelu_bwd": (lambda: B.cf_bias_lrelu_bwd(nvox, c, dt, dy, y, 0.01, dz, db, ws), 3 * zb),
        "avgpool_fwd": (lambda: B.cf_avgpool3d_fwd(n, s, s, s, c, 2, 2, dt, y, pool), zb + pb),
        "avgpool_bwd": (lambda: B.cf_avgpool3d_bwd(n, s, s, s, c, 2, 2, dt, dp, dy2), zb + pb),
    }
    out = {}
    for name, (fn, nbytes) in ops.items():
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            fn()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / 10
        gbs = nbytes / (us * 1e-6) / 1e9
        out[name] = dict(us=round(us, 1), algorithmic_bytes=nbytes, achieved=round(gbs, 1),
                         frac=round(gbs / HBM_PEAK_GBS, 4))
    return dict(shape=[n, s, s, s, c], dtype=dt, unit="GB/s", peak=HBM_PEAK_GBS, passes=out)


def run_stack(name, args, steps, warmup, extras):
    """Warm up, find the dominant op (events around every call over 3 steps),
    then time `steps` steps with events around the dominant op only.  extras:
    also time the FC head and the parameter update on their own (after the
    timed steps)."""
    import numpy as np
    import torch

    from paper_1808_04728_amd import binding as B
    from paper_1808_04728_amd import inputs
    from paper_1808_04728_amd.stack import ConvStack

    wl = inputs.WORKLOADS[name]
    st = ConvStack(wl["layers"], wl["size"], wl["batch"], wl["dtype"], inputs.ALPHA, "cuda:0", fused=not args.unfused)
    ws, bs = inputs.make_weights(name)
    st.set_params(ws, bs)
    st.set_input(inputs.make_input(name))
    dout = torch.as_tensor(inputs.normal((wl["batch"],) + st.out_dhw + (wl["layers"][-1]["cout"],),
                                         30000 + wl["cfg"]), device="cuda:0").to(st.tdt)

    hp = B.make_hparams(100000)  # the paper's constants; its decay length is not given

    from paper_1808_04728_amd.head import FCHead
    feats = int(np.prod(st.out_dhw)) * wl["layers"][-1]["cout"]
    head = FCHead(wl["batch"], feats, inputs.HEAD_WIDTHS, wl["dtype"], inputs.ALPHA, "cuda:0")
    head.set_params(*inputs.make_head(name, feats))
    head_dout = head.dx[0].view(dout.shape)

    def step():
        st.forward()
        if args.with_head:
            head.step(st.output())
            st.backward(head_dout)
        else:
            st.backward(dout)
        if args.with_update:
            st.update(hp)

    # warm-up: W steps, then more untimed steps until RAMP_S seconds have passed.
    # The GPU's clocks take tens of milliseconds of sustained work to reach their
    # steady state (measured on the 128^3 stacks: the first ~40 steps after an
    # idle period run 3-50% slower), and a training job runs in that state.
    t_w = time.perf_counter()
    done, prev = 0, None
    while done < warmup or time.perf_counter() - t_w < RAMP_S:
        for _ in range(8):
            step()
        done += 8
        ev = torch.cuda.Event()
        ev.record()
        if prev is not None:
            prev.synchronize()  # bounds the queue without letting the GPU go idle
        prev = ev
    torch.cuda.synchronize()

    # per-op times (events around every call) to find the dominant op
    st.timer = {}
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    op_ms = {k: float(np.mean([a.elapsed_time(b) for a, b in v])) for k, v in st.timer.items()}
    dominant = max(op_ms, key=op_ms.get)
    if args.op_breakdown:
        # in call order (the order of the ops' launches within a step), with each
        # op's FLOPs and algorithmic bytes
        print(f"{name}:", file=sys.stderr)
        for k, v in op_ms.items():
            fl, nb = st.op_flops(k), st.op_bytes(k)
            extra = f"{fl / v / 1e9:8.1f} TFLOP/s" if fl else f"{nb / v / 1e6:8.1f} GB/s"
            print(f"  op {k:30s} {v * 1e3:9.1f} us {fl / 1e9:10.4f} GFLOP {nb / 1e6:10.4f} MB  {extra}",
                  file=sys.stderr)

    # timed region: events bracket only the dominant op
    st.timer = {}
    st.timed_ops = {dominant}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom_ms = float(np.mean([a.elapsed_time(b) for a, b in st.timer[dominant]]))
    st.timer = None

    ms = wall * 1e3 / steps
    flops = st.conv_flops()
    tflops = flops / (ms * 1e-3) / 1e12
    peak = PEAK[wl["dtype"]]
    dom_flops = st.op_flops(dominant)
    if dom_flops:
        ach = dom_flops / (dom_ms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(ach, 2), peak=peak, unit="TFLOP/s", frac=round(ach / peak, 4),
                    traffic=measured_traffic(name, dominant), kernel=dominant, launch_ms=round(dom_ms, 4),
                    per_launch=f"{dom_flops / 1e9:.2f} GFLOP", algorithmic_bytes=st.op_bytes(dominant))
    else:
        gbs = st.op_bytes(dominant) / (dom_ms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(gbs, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=round(gbs / HBM_PEAK_GBS, 4), traffic=measured_traffic(name, dominant), kernel=dominant,
                    launch_ms=round(dom_ms, 4), per_launch=f"{st.op_bytes(dominant) / 2**20:.1f} MiB",
                    algorithmic_bytes=st.op_bytes(dominant))
    out = dict(wl=wl, ms=ms, tflops=tflops, flops=flops, peak=peak, roofline=roof,
               op_ms={k: round(v, 4) for k, v in sorted(op_ms.items(), key=lambda kv: -kv[1])},
               samples_per_s=round(wl["batch"] / (ms * 1e-3), 2))
    if not extras:
        return out

    # the FC head + loss alone (before any parameter update): forward and
    # backward twice, queued behind a step so that the device never waits for
    # the host to submit the launches; the one-call head (four launches) and,
    # for reference, the per-layer calls (22 launches)
    def head_time(fn):
        hts = []
        for _ in range(5):
            step()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(2):
                fn()
            e1.record()
            hts.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in hts])) / 2

    def per_layer():
        head.forward(st.output())
        head.backward()

    per_layer_ms = head_time(per_layer)
    head_ms = head_time(lambda: head.step(st.output()))
    head_bytes = head.weight_bytes()
    head_gbs = head_bytes / (head_ms * 1e-3) / 1e9
    out["head"] = dict(widths=[feats, *inputs.HEAD_WIDTHS], ms=round(head_ms, 4),
                       algorithmic_bytes=head_bytes, achieved=round(head_gbs, 1), unit="GB/s", peak=HBM_PEAK_GBS,
                       frac=round(head_gbs / HBM_PEAK_GBS, 4), in_step=args.with_head, one_call=head.fused,
                       per_layer_ms=round(per_layer_ms, 4),
                       loss=round(float(head.loss[0].item()), 6))

    # the parameter update alone, after the timed steps (it changes the weights):
    # K updates queued behind a step, so that the device never waits for the host
    # to submit the next one, bracketed by events
    ups = []
    for _ in range(3):
        step()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            st.update(hp)
        e1.record()
        ups.append((e0, e1))
    torch.cuda.synchronize()
    upd_ms = float(np.mean([a.elapsed_time(b) for a, b in ups])) / 10
    upd_bytes = st.update_bytes()
    upd_gbs = upd_bytes / (upd_ms * 1e-3) / 1e9
    update = dict(kernel="adam_norms + adam_update", params=st.param_offsets[-1], groups=len(st.param_offsets) - 1,
                  launch_ms=round(upd_ms, 4), algorithmic_bytes=upd_bytes, achieved=round(upd_gbs, 1),
                  unit="GB/s", peak=HBM_PEAK_GBS, frac=round(upd_gbs / HBM_PEAK_GBS, 4), in_step=args.with_update)
    update["paper_network_size"] = update_at_paper_size(step, B, np, torch, wl["dtype"] == "bf16")
    out["update"] = update
    return out


def config_of(name, wl, flops, args):
    return {"workload": describe(name, wl) + (", unfused entry points" if args.unfused else "")
            + (", Adam + LARC update in every step" if args.with_update else "")
            + (", FC head + loss in every step" if args.with_head else ""),
            "name": name, "edge": wl["size"], "batch": wl["batch"],
            "input_channels": wl["c0"], "conv_gflop_per_step": round(flops / 1e9, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="stack_128c_b1_f32",
                    help="headline workload (default: the 128^3 stack at the paper's fp32, batch 1)")
    ap.add_argument("--extra-workload", default="stack_128c_b8_bf16",
                    help="second workload reported under its own key ('none' to skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--op-breakdown", action="store_true", help="print per-op times to stderr")
    ap.add_argument("--with-update", action="store_true",
                    help="apply the Adam + LARC parameter update inside every timed step")
    ap.add_argument("--with-head", action="store_true",
                    help="run the FC head + loss inside every step (its input gradient drives the backward pass)")
    ap.add_argument("--unfused", action="store_true",
                    help="run every layer through the unfused entry points (conv, bias + lReLU, pool separately)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device copies of MIB MiB (calibrates the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the step would shard "
              "data-parallel, with one allreduce of the weight and bias gradients per step, which is not "
              "implemented); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    from paper_1808_04728_amd import binding as B
    from paper_1808_04728_amd import inputs

    torch.cuda.set_device(0)
    name = args.workload
    r = run_stack(name, args, args.steps, args.warmup, extras=True)
    wl = r["wl"]
    res = {
        "metric": METRIC,
        "value": round(r["tflops"], 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl["dtype"],
        "data": "synthetic",
        "config": config_of(name, wl, r["flops"], args),
        "samples_per_s": r["samples_per_s"],
        "mfma_peak_frac": round(r["tflops"] / r["peak"], 4),
        "roofline": r["roofline"],
        "op_ms": r["op_ms"],
        "update": r["update"],
        "head": r["head"],
    }
    if args.extra_workload != "none" and args.extra_workload != name:
        x = run_stack(args.extra_workload, args, args.steps, args.warmup, extras=False)
        xw = x["wl"]
        res[args.extra_workload] = dict(
            value=round(x["tflops"], 3), unit="TFLOP/s", ms_per_step=round(x["ms"], 4), dtype=xw["dtype"],
            samples_per_s=x["samples_per_s"], mfma_peak_frac=round(x["tflops"] / x["peak"], 4),
            config=config_of(args.extra_workload, xw, x["flops"], args), roofline=x["roofline"], op_ms=x["op_ms"])
    # the unfused elementwise and pool passes at the largest first-layer activation
    # of the two workloads (the bf16 batch-8 one: 512 MiB, beyond the last-level cache)
    pw = inputs.WORKLOADS[args.extra_workload] if args.extra_workload in inputs.WORKLOADS else wl
    res["hbm_passes"] = hbm_passes(B, np, torch, pw)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(name)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
