"""Benchmark of the MI355X SGD-step hot path.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--quick] [--no-cpu]

Headline workload: one SGD step of the wide regression MLP (batch 4096,
1024 -> 4 x 4096 ReLU -> 1, MSE, fp16 storage, fp32 accumulation and master
weights, dynamic loss scaling, momentum 0.9): forward, loss, backward and
update of one minibatch of synthetic inputs already resident in HBM.  `value`
is train samples per second.

Also on the same JSON line:
  roofline      the step's dominant kernel: its average launch duration from
                HIP events around each launch of a replay of exactly its
                launches in the step (same shapes and buffers), against the
                fp16 MFMA peak; HBM traffic per launch from rocprofv3 counters
                (profiles/) while the kernel source is unchanged;
  cpu_baseline  the fp64 oracle's step on this host on one full batch;
  gemm_sweep    the fp16 GEMM sweep (M = N = K in 1024/4096/8192, NN/NT/TN);
  conv          the ResNet-style 3x3 layers (batch 128) fwd / bwd-data /
                bwd-filter;
  gemm_fp32_split3  fp32 GEMMs (4096, 8192) through three fp16 MFMA
                products of the Eq. (1) splits, next to the native fp32 kernel;
  workloads     samples/s of the LeNet-style bf16 step and the fp32 MLP step;
  async_sgd     the same two nets trained asynchronously (section 3.1) by
                several workers on separate streams sharing one parameter
                vector, samples/s over all workers;
  sustained_clock  the shader clock rocm-smi reports while the headline step,
                and the NN 8192^3 fp16 GEMM on the sweep's operands and on
                all-zero operands, run back to back for a few seconds: the
                rate the matrix cores keep at the clock the power limit allows.
Every timed region follows sustained untimed load (about a second of the
same work, or 3 runs of at least 50 ms with the median kept for the
sub-benchmarks): the GPU's clocks settle under sustained load, which is the
state a training run spends its time in.
Only one GPU is used; --gpus > 1 exits with a message.
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

METRIC = "train samples/sec per step; mixed-precision GEMM/conv TFLOP/s (% MFMA peak)"
PEAK_F16_TFLOPS = 2516.6   # MI355X dense fp16/bf16 MFMA (256 CU x 4096 FLOP/clk x 2.4 GHz)
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def _sync():
    import torch
    torch.cuda.synchronize()


class _Timer:
    """HIP events on torch's current stream (the stream every call uses)."""

    def __init__(self):
        import torch
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def __enter__(self):
        _sync()
        self.a.record()
        return self

    def __exit__(self, *exc):
        self.b.record()
        _sync()
        self.ms = self.a.elapsed_time(self.b)


def _train_setup(mdnn, cfg, n_batches=10, fuse_update=False):
    import torch
    import workloads as W
    net = mdnn.Net(cfg.layers, cfg.batch, {"f32": 0, "f16": 1, "bf16": 2}[cfg.dtype], cfg.loss,
                   cfg.lr, cfg.momentum, cfg.loss_scaling, cfg.init_scale, cfg.n_classes,
                   fuse_update=fuse_update)
    net.set_params(W.init_params(cfg))
    xs, ts = [], []
    for s in range(n_batches):
        x, t = W.batch_inputs(cfg, s)
        xs.append(torch.from_numpy(x).cuda())
        ts.append(torch.from_numpy(t).cuda())
    _sync()
    return net, xs, ts


WARM_SECONDS = 1.0   # sustained load before a timed region: the GPU's clock settles under it


def _warm(fn, seconds=WARM_SECONDS):
    """Run fn back to back for about `seconds` (untimed): GPU clocks ramp up
    under sustained load, and a training run spends its life in that state."""
    fn()
    _sync()
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(max(1, 2 ** min(n, 6))):
            fn()
        _sync()
        n += 1


def _measure(fn, min_ms=50.0, chunks=3):
    """Median per-call time (ms) over `chunks` back-to-back runs of at least
    `min_ms` each, after a short warm-up."""
    for _ in range(3):
        fn()
    with _Timer() as tm:
        fn()
    reps = max(3, int(min_ms / max(tm.ms, 1e-3)))
    res = []
    for _ in range(chunks):
        with _Timer() as tm:
            for _ in range(reps):
                fn()
        res.append(tm.ms / reps)
    return sorted(res)[len(res) // 2]


def _time_steps(net, xs, ts, steps, warmup, check=None):
    it = iter(range(1 << 62))

    def one():
        i = next(it)
        net.step(xs[i % len(xs)], ts[i % len(ts)])
    _warm(one)
    for i in range(warmup):
        net.step(xs[i % len(xs)], ts[i % len(ts)])
    _sync()
    if check is not None:
        check.start()
    with _Timer() as tm:
        for i in range(steps):
            net.step(xs[i % len(xs)], ts[i % len(ts)])
    return tm.ms / steps


class _UpdateCheck:
    """Whether every step between start() and stop() applied its update.  A
    loss-scaled step that overflows skips its update (and halves the scale);
    a timed step must do the whole step's work, so the benchmark checks the
    scaler's state machine: with no overflow, good_steps advanced by exactly
    the number of steps (modulo growth_interval, where the scale grows)."""

    def __init__(self, mdnn, net):
        self.mdnn, self.net = mdnn, net
        self.before = None

    def start(self):
        if self.net.scaler is not None:
            self.before = self.mdnn.read_scaler(self.net.scaler)

    def stop(self, steps: int) -> bool:
        if self.net.scaler is None:
            return True
        b, a = self.before, self.mdnn.read_scaler(self.net.scaler)
        total = b["good_steps"] + steps
        gi = b["growth_interval"]
        grown = b["scale"] * b["growth"] ** (total // gi)
        return a["good_steps"] == total % gi and a["scale"] == grown


def _time_graph_steps(net, xs, ts, steps, warmup, check=None):
    """As _time_steps, with each batch's step recorded once into a HIP graph
    and replayed (one launch per step instead of one per kernel)."""
    graphs = [net.record_step(x, t) for x, t in zip(xs, ts)]
    it = iter(range(1 << 62))

    def one():
        graphs[next(it) % len(graphs)].launch()
    _warm(one)
    for i in range(warmup):
        graphs[i % len(graphs)].launch()
    _sync()
    if check is not None:
        check.start()
    with _Timer() as tm:
        for i in range(steps):
            graphs[i % len(graphs)].launch()
    for g in graphs:
        g.close()
    return tm.ms / steps


def _under_profiler() -> bool:
    """True inside rocprofv3: its preloaded library would initialise the GPU
    in every child process too, so no helper programs are started then."""
    return "rocprof" in os.environ.get("LD_PRELOAD", "") or any(k.startswith("ROCPROF") for k in os.environ)


def _clocks():
    """Current shader / memory clocks (MHz) as rocm-smi reports them, or None
    (also when running under the profiler)."""
    import re
    import subprocess
    if _under_profiler():
        return None
    try:
        out = subprocess.run(["rocm-smi", "--showclocks", "--json"], capture_output=True, text=True,
                             timeout=30).stdout
        d = json.loads(out)
    except Exception:
        return None
    res = {}
    for card in d.values():
        if not isinstance(card, dict):
            continue
        for k, v in card.items():
            m = re.search(r"(\d+)\s*mhz", str(v), re.I)
            if m and "speed" in k.lower():
                for clk in ("sclk", "mclk", "fclk", "socclk"):
                    if k.lower().startswith(clk):
                        res[clk + "_mhz"] = int(m.group(1))
        break
    return res or None


UPDATE_OUT = "f32 + SGD update"   # a weight-gradient product that applies the update (fuse_update)


def _fused(cfg, i) -> bool:
    """Whether the train step with fuse_update updates FC layer i inside its
    weight-gradient product (the library's rule: in and out multiples of 256,
    a batch multiple of 64, 16-bit storage (fp16 when the loss is scaled), and
    a product the unfused step would not split over K: at least 128 tiles of
    128 x 128, or K < 256)."""
    import workloads as W
    l = cfg.layers[i]
    if l.kind != W.FC or cfg.dtype == "f32" or (cfg.loss_scaling and cfg.dtype != "f16"):
        return False
    if l.c_in % 256 or l.c_out % 256 or cfg.batch % 64:
        return False
    return (l.c_in // 128) * (l.c_out // 128) >= 128 or cfg.batch < 256


def _step_gemms(cfg, fuse_update=False):
    """Every GEMM one step of an FC chain issues, as (layout, M, N, K, out)."""
    import workloads as W
    out, B = [], cfg.batch
    n = len(cfg.layers)
    for i, l in enumerate(cfg.layers):
        if l.kind != W.FC:
            continue
        out.append(("NN", B, l.c_out, l.c_in, "f32" if i == n - 1 else cfg.dtype, i))
        out.append(("TN", l.c_in, l.c_out, B, UPDATE_OUT if fuse_update and _fused(cfg, i) else "f32", i))
        if i > 0:
            out.append(("NT", B, l.c_in, l.c_out, cfg.dtype, i))
    return out


def _kernel_choice(layout: str, m: int, n: int, k: int) -> str:
    """The GEMM engine's automatic kernel choice for the step's plain,
    aligned operands (mirrors the library's fixed table)."""
    cd = lambda a, b: -(-a // b)  # noqa: E731
    if k <= 4:
        return "skinny depth kernel"
    if n <= 4 and layout != "TN":
        return "skinny rows kernel"
    if n <= 16 and layout == "TN":
        return "skinny cols kernel"
    mn_contig = {"NN": [n], "NT": [], "TN": [m, n]}[layout]
    if k % 64 == 0 and all(d % 8 == 0 for d in mn_contig) and cd(m, 128) * cd(n, 128) >= 32:
        if n <= 64 and m > 64:
            return "gemm_lds_kernel (256x64 direct-to-LDS pipeline)"
        if m <= 64 and n > 64:
            return "gemm_lds_kernel (64x256 direct-to-LDS pipeline)"
        if n > 128 and m > 128 and cd(m, 256) * cd(n, 256) >= 256:
            return "gemm_lds_kernel (256x256 direct-to-LDS pipeline)"
        if cd(m, 128) * cd(n, 128) < 128 and cd(m, 64) * cd(n, 64) >= 128:
            return "gemm_lds_kernel (64x64 direct-to-LDS pipeline)"
        if cd(m, 128) * cd(n, 128) <= 256:
            return "gemm_lds_kernel (128x128 direct-to-LDS pipeline with 3 stages)"
        return "gemm_lds_kernel (128x128 direct-to-LDS pipeline)"
    if m <= 64 or n <= 64:
        return "gemm_mfma_kernel 64x64"
    if cd(m, 256) * cd(n, 256) >= 256 and m > 128 and n > 128:
        return "gemm_mfma_kernel 256x256"
    if cd(m, 128) * cd(n, 128) >= 160:
        return "gemm_mfma_kernel 128x128"
    return "gemm_mfma_kernel 64x64"


def _replay_group(mdnn, net, cfg, group, reps):
    """Replay the launches of one kernel instantiation exactly as the step
    issues them (same shapes, leading dimensions, epilogues and buffers),
    `reps` times; returns (mean ms per launch, mean FLOP per launch)."""
    lp = {"f32": 0, "f16": 1, "bf16": 2}[cfg.dtype]
    es = 2 if lp else 4
    offs = cfg.param_offsets()
    wbase = net.lowp.data_ptr() if net.lowp is not None else net.master.data_ptr()
    # the step's own activation-gradient buffers ([batch, widest] each), holding
    # the last step's gradients: the replayed products see the step's data
    # (masked, partly zero), which the GPU's power and clock depend on
    g0, g1 = net.output_grad_ptr(0), net.output_grad_ptr(1)
    assert g0 and g1
    import torch
    calls, keep = [], []
    for (layout, M, N, K, out_t, i) in group:
        l = cfg.layers[i]
        a_in = net.activation_ptr(i)
        a_out = net.activation_ptr(i + 1)
        wptr = wbase + offs[i][0] * es
        bias = net.master.data_ptr() + offs[i][1] * 4
        if out_t == UPDATE_OUT:
            # the fused update, on copies of the layer's weights, momentum and
            # working copy (replays must not move the net's own parameters)
            w0, nw = offs[i][0], M * N
            cp = (net.master[w0:w0 + nw].clone(), net.mom[w0:w0 + nw].clone() if net.mom is not None else None,
                  net.lowp[w0:w0 + nw].clone())
            keep.append(cp)
            calls.append(("upd", M, N, K, a_in, M, g0, N, cp))
            continue
        if layout == "NN":
            calls.append((0, M, N, K, a_in, K, wptr, N, a_out, N, 0 if out_t == "f32" else lp,
                          bias, l.act, None, 0))
        elif layout == "TN":
            calls.append((2, M, N, K, a_in, M, g0, N, net.grads.data_ptr() + offs[i][0] * 4,
                          N, 0, None, 0, None, 0))
        else:
            calls.append((1, M, N, K, g0, K, wptr, K, g1, N, lp, None, 0,
                          a_in, N))
    flops = sum(2.0 * c[1] * c[2] * c[3] for c in calls) / len(calls)
    # one event pair around the timed replay: reps x the group's launches back
    # to back, queued behind a bounded spin kernel so that the GPU never waits
    # for the host; the mean launch duration is the elapsed time over the
    # launches (an event pair around every launch added about 5 us to each,
    # against the kernel trace's durations of the same launches)
    # the step's split-K workspace and, for the weight gradients, its loss
    # scaler's overflow flag: the replay takes the kernel paths the step takes
    ws_bytes = max([mdnn.mdnn_gemm_workspace(lp, c[1], c[2], c[3]) for c in calls] + [256])
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")

    def launch(c):
        if c[0] == "upd":
            w, v, wl = c[8]
            mdnn.mdnn_gemm_tn_update(c[1], c[2], c[3], c[4], c[5], c[6], c[7], lp, w, v, wl, c[2], cfg.lr,
                                     cfg.momentum, net.scaler)
            return
        mdnn.mdnn_gemm_mixed_ws(c[0], c[1], c[2], c[3], 1.0, c[4], c[5], c[6], c[7], lp, 0.0,
                                None, 0, c[8], c[9], c[10], c[11], c[12], c[13], c[14], ws, ws_bytes,
                                nonfinite=flag if c[0] == 2 and c[10] == 0 else None)
    for _ in range(3):
        for c in calls:
            launch(c)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if hasattr(torch.cuda, "_sleep"):
        torch.cuda._sleep(4_000_000)
    e0.record()
    for _ in range(reps):
        for c in calls:
            launch(c)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / (reps * len(calls)), flops


GRAPH_CALLS = 32
# the headline step updates its hidden layers inside their weight-gradient
# products (mdnn_train_cfg_t.fuse_update: bitwise the same step)
FUSE_UPDATE = True


def _graph_measure(fn, reps_scale=1.0):
    """Per-call time (ms) of GRAPH_CALLS calls of fn recorded into one HIP
    graph and replayed: the launches reach the GPU back to back, without the
    host's per-call cost (which exceeds the kernel itself for a 1024^3
    product)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()   # first call outside the capture
    torch.cuda.current_stream().wait_stream(side)
    _sync()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(GRAPH_CALLS):
            fn()
    ms = _measure(g.replay, min_ms=50.0 * reps_scale) / GRAPH_CALLS
    del g
    return ms


def _gemm_sweep(mdnn, reps_scale=1.0):
    import torch
    import workloads as W
    res = {}
    for size in W.GEMM_SIZES:
        for layout in W.GEMM_LAYOUTS:
            a, b = W.gemm_operands(layout, size, size, size)
            A, B = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
            D = torch.empty((size, size), dtype=torch.float32, device="cuda")
            lay = {"NN": 0, "NT": 1, "TN": 2}[layout]

            def run():
                mdnn.mdnn_gemm_mixed(lay, size, size, size, 1.0, A, A.stride(0), B, B.stride(0), 1,
                                     0.0, None, 0, D, size, 0)
            ms = _measure(run, min_ms=50.0 * reps_scale)
            tf = 2.0 * size ** 3 / (ms * 1e-3) / 1e12
            gms = _graph_measure(run, reps_scale)
            gtf = 2.0 * size ** 3 / (gms * 1e-3) / 1e12
            res[f"{layout}_{size}"] = {"ms": round(ms, 4), "tflops": round(tf, 1),
                                       "mfma_frac": round(tf / PEAK_F16_TFLOPS, 4),
                                       "graph_ms": round(gms, 4), "graph_tflops": round(gtf, 1)}
            del A, B, D
    return res


CLOCK_MAX_MHZ = 2400   # the shader clock PEAK_F16_TFLOPS assumes


def _sampled_clock(fn, seconds=3.0):
    """Run fn back to back for about `seconds` (after _warm) while a thread
    samples rocm-smi's shader clock; returns (ms per call, median sclk MHz or
    None, samples)."""
    import statistics
    import threading
    import torch
    _warm(fn)
    samples, stop = [], threading.Event()

    def sample():
        while not stop.is_set():
            c = _clocks()
            if c and c.get("sclk_mhz"):
                samples.append(c["sclk_mhz"])
            stop.wait(0.2)
    th = threading.Thread(target=sample, daemon=True)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    th.start()
    a.record()
    n, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            fn()
        n += 8
        _sync()
    b.record()
    _sync()
    stop.set()
    th.join()
    return a.elapsed_time(b) / n, (statistics.median(samples) if samples else None), len(samples)


def _sustained_clock(mdnn, net=None, xs=None, ts=None, cfg=None):
    """The shader clock under sustained load.  MI355X's matrix-core peak
    assumes 2.4 GHz; with N(0,1) fp16 operands the GEMMs draw enough power
    that the clock settles well below it, while the same product on all-zero
    operands (far less switching) holds 2.4 GHz.  frac_at_sclk is the GEMM's
    rate over the peak scaled to the sampled clock."""
    import torch
    import workloads as W
    res = {}
    if net is not None:
        it = iter(range(1 << 62))

        def step():
            i = next(it)
            net.step(xs[i % len(xs)], ts[i % len(ts)])
        ms, mhz, ns = _sampled_clock(step)
        tf = cfg.flops_per_step() / (ms * 1e-3) / 1e12
        res["wide_mlp_step"] = {"ms": round(ms, 4), "tflops": round(tf, 1), "sclk_mhz": mhz, "sclk_samples": ns,
                                "frac_at_sclk": round(tf / (PEAK_F16_TFLOPS * mhz / CLOCK_MAX_MHZ), 4)
                                if mhz else None}
    size = 8192
    a, b = W.gemm_operands("NN", size, size, size)
    A, B = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    D = torch.empty((size, size), dtype=torch.float32, device="cuda")

    def run():
        mdnn.mdnn_gemm_mixed(0, size, size, size, 1.0, A, A.stride(0), B, B.stride(0), 1,
                             0.0, None, 0, D, size, 0)
    for name in ("NN_8192", "NN_8192_zero_operands"):
        if name.endswith("zero_operands"):
            A.zero_()
            B.zero_()
        ms, mhz, ns = _sampled_clock(run)
        tf = 2.0 * size ** 3 / (ms * 1e-3) / 1e12
        res[name] = {"ms": round(ms, 4), "tflops": round(tf, 1), "mfma_frac": round(tf / PEAK_F16_TFLOPS, 4),
                     "sclk_mhz": mhz, "sclk_samples": ns,
                     "frac_at_sclk": round(tf / (PEAK_F16_TFLOPS * mhz / CLOCK_MAX_MHZ), 4) if mhz else None}
    del A, B, D
    return res


def _fuse_ab(mdnn, rounds=3, steps=50):
    """The headline step with and without fuse_update, alternating in one
    process (the same box and clock state for both): ms per step of each
    round, and whether every timed step applied its update."""
    import torch
    import workloads as W
    cfg = W.wide_mlp_fp16()
    res = {"unfused_ms": [], "fused_ms": [], "every_update_applied": True}
    for _ in range(rounds):
        for fuse in (False, True):
            net, xs, ts = _train_setup(mdnn, cfg, fuse_update=fuse)
            check = _UpdateCheck(mdnn, net)
            ms = _time_steps(net, xs, ts, steps, 5, check)
            res["every_update_applied"] &= bool(check.stop(steps))
            res["fused_ms" if fuse else "unfused_ms"].append(round(ms, 4))
            net.close()
            del net, xs, ts
            torch.cuda.empty_cache()
    return res


def _split3_sweep(mdnn):
    """fp32 GEMMs through three fp16 MFMA products (section 3.2, Eq. (1)),
    next to the native fp32 (VALU) kernel; inputs fp32 N(0,1)/sqrt(K)."""
    import torch
    import workloads as W
    res = {}
    for size in (4096, 8192):
        for layout in W.GEMM_LAYOUTS:
            a, b = W.gemm_operands(layout, size, size, size, dtype="f32")
            A, B = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
            D = torch.empty((size, size), dtype=torch.float32, device="cuda")
            lay = {"NN": 0, "NT": 1, "TN": 2}[layout]
            wsb = mdnn.mdnn_gemm_split3_workspace(size, size, size)
            ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
            fns = {"split3": lambda: mdnn.mdnn_gemm_split3(lay, size, size, size, 1.0, A, A.stride(0), 1.0,
                                                           B, B.stride(0), 1.0, 0.0, None, 0, D, size,
                                                           ws, wsb)}
            if size == 4096:
                fns["native_f32"] = lambda: mdnn.mdnn_gemm_mixed(lay, size, size, size, 1.0, A, A.stride(0), B,
                                                                 B.stride(0), 0, 0.0, None, 0, D, size, 0)
            for name, fn in fns.items():
                ms = _measure(fn, min_ms=40.0, chunks=3)
                tf = 2.0 * size ** 3 / (ms * 1e-3) / 1e12
                ent = {"ms": round(ms, 4), "fp32_tflops": round(tf, 1),
                       "vs_fp32_peak": round(tf / PEAK_F32_TFLOPS, 3)}
                if name == "split3":   # three fp16 products of depth K on the matrix cores
                    ent["mfma_frac"] = round(3 * tf / PEAK_F16_TFLOPS, 4)
                res[f"{name}_{layout}_{size}"] = ent
            del A, B, D, ws
    return res


def _conv_bench(mdnn, reps=20):
    import torch
    import workloads as W
    res = {}
    for li, sh in enumerate(W.RESNET_LAYERS):
        x, w, dy = W.conv_operands(sh)
        X, Wt, DY = (torch.from_numpy(v).cuda() for v in (x, w, dy))
        cs = mdnn.ConvShape(sh.n, sh.h, sh.w, sh.c_in, sh.c_out, sh.r, sh.s, sh.pad)
        y = torch.empty(dy.shape, dtype=torch.float16, device="cuda")
        dx = torch.empty(x.shape, dtype=torch.float16, device="cuda")
        dw = torch.empty(w.shape, dtype=torch.float32, device="cuda")
        wsb = mdnn.mdnn_conv2d_bwd_filter_workspace(cs, 1)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        # one workspace big enough for every forward algorithm
        awb = max(mdnn.mdnn_conv2d_fwd_algo_workspace(cs, 1, a) for a in (mdnn.CONV_IM2COL_GEMM, mdnn.CONV_WINOGRAD))
        aws = torch.empty(max(awb, 256), dtype=torch.uint8, device="cuda")
        fns = {
            "fwd": lambda: mdnn.mdnn_conv2d_fwd(cs, X, Wt, 1, None, 0, y, 1),
            "bwd_data": lambda: mdnn.mdnn_conv2d_bwd_data(cs, DY, Wt, 1, None, dx, 1),
            "bwd_filter": lambda: mdnn.mdnn_conv2d_bwd_filter(cs, X, DY, 1, dw, None, ws, wsb),
            # the alternative forward algorithms (section 2.1); their "tflops"
            # count the direct convolution's FLOP (equivalent rate)
            "fwd_im2col_gemm": lambda: mdnn.mdnn_conv2d_fwd_algo(cs, X, Wt, 1, None, 0, y, 1, mdnn.CONV_IM2COL_GEMM,
                                                                 aws, awb),
            "fwd_winograd": lambda: mdnn.mdnn_conv2d_fwd_algo(cs, X, Wt, 1, None, 0, y, 1, mdnn.CONV_WINOGRAD,
                                                              aws, awb),
        }
        for op, fn in fns.items():
            ms = _measure(fn, min_ms=30.0)
            tf = sh.flops() / (ms * 1e-3) / 1e12
            res[f"L{li + 1}_{sh.c_in}x{sh.h}_{op}"] = {"ms": round(ms, 4), "tflops": round(tf, 1),
                                                       "mfma_frac": round(tf / PEAK_F16_TFLOPS, 4)}
        key = f"L{li + 1}_{sh.c_in}x{sh.h}"
        # the library's own per-layer choice given room for every algorithm
        res[f"{key}_fwd_selected"] = {mdnn.CONV_IMPLICIT_GEMM: "implicit_gemm", mdnn.CONV_IM2COL_GEMM: "im2col_gemm",
                                      mdnn.CONV_WINOGRAD: "winograd"}[mdnn.mdnn_conv2d_fwd_choose(cs, 1, awb)]
    return res


def _async_bench(mdnn, steps=40):
    """Asynchronous SGD (section 3.1): W workers on W streams share one fp32
    parameter vector (mdnn_train_step_async), next to the synchronous step of
    the same net; samples/s over all workers' steps."""
    import torch
    import workloads as W
    res = {}
    for cfg, workers in ((W.mlp784_fp32(), 4), (W.lenet_bf16(), 2)):
        lp = {"f32": 0, "f16": 1, "bf16": 2}[cfg.dtype]
        params = torch.as_tensor(W.init_params(cfg), dtype=torch.float32)
        nets = []
        for k in range(workers):
            n = mdnn.Net(cfg.layers, cfg.batch, lp, cfg.loss, cfg.lr, cfg.momentum, cfg.loss_scaling,
                         cfg.init_scale, cfg.n_classes, shared_master=nets[0].master if nets else None)
            if not nets:
                n.set_params(params)
            nets.append(n)
        streams = [torch.cuda.Stream() for _ in range(workers)]
        data = []
        for s in range(8):
            x, t = W.batch_inputs(cfg, s)
            tt = torch.from_numpy(t).cuda()
            data.append((torch.from_numpy(x).cuda(), tt))
        losses = [torch.zeros(1, device="cuda") for _ in range(workers)]

        def round_():
            for k in range(workers):
                x, t = data[k % len(data)]
                nets[k].step_async(x, t, loss_out=losses[k], stream=streams[k])
        _warm(round_, 0.3)
        with _Timer() as tm:
            for _ in range(steps):
                round_()
            for st in streams:
                torch.cuda.current_stream().wait_stream(st)
        ms = tm.ms / (steps * workers)
        res[f"{cfg.name}_async{workers}"] = {"workers": workers, "ms_per_step": round(ms, 4),
                                             "samples_per_s": round(cfg.batch / (ms * 1e-3), 1)}
        for n in nets:
            n.close()
    return res


def _traffic_key(kernel_desc: str) -> str:
    """'NN f16 -> f16 256x256' style key of a step kernel description."""
    tile = "256x256" if "256x256" in kernel_desc else "128x128"
    if "3 stages" in kernel_desc:
        tile += " (3 stages)"
    parts = kernel_desc.split(", ")
    return f"{parts[1]} {tile}"


TRAFFIC_SOURCES = ("gemm_lds.h", "gemm_core.h", "common.h")


def gemm_lds_source_digest() -> str:
    """SHA-256 over the pipelined GEMM kernel's sources, in TRAFFIC_SOURCES order."""
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2011_11188_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def _traffic_record(kernel_desc: str):
    """HBM bytes per launch of a step kernel measured with rocprofv3 counters
    (profiles/), used only while the kernel's source (the pipeline, its
    epilogue and the shared device helpers) is unchanged."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "gemm_lds_kernel_traffic.txt")
    if not os.path.exists(path) or "gemm_lds_kernel" not in kernel_desc:
        return None
    sha, recs = None, {}
    for ln in open(path):
        if ln.startswith("source_sha256:"):
            sha = ln.split(":", 1)[1].strip()
        elif ln.startswith("record:"):
            f = [x.strip() for x in ln.split(":", 1)[1].split("|")]
            recs[f[0]] = float(f[-1].split()[-1])
    if sha != gemm_lds_source_digest():
        return None
    return recs.get(_traffic_key(kernel_desc))


def _cpu_baseline(cfg):
    """The fp64 oracle's step on one full batch of the headline workload."""
    import numpy as np
    import workloads as W
    from oracle import train
    # the host cores this process may run on (numpy's BLAS pool is sized to them)
    threads = len(os.sched_getaffinity(0))
    orc = train.from_config(cfg, W.init_params(cfg))
    x, t = W.batch_inputs(cfg, 0)
    t0 = time.perf_counter()
    orc.step(x, t)
    dt = time.perf_counter() - t0
    del np
    return {"value": round(cfg.batch / dt, 2), "unit": "samples/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"one full SGD step (batch {cfg.batch}) of {cfg.name} in fp64 numpy "
                      f"(its products through numpy's BLAS), {dt:.1f} s wall"}


def _copy_calibration(mdnn):
    """Calibration for HBM-traffic counters: a plain fp32 copy of known size
    (256 MiB read + 256 MiB written per launch), three launches."""
    import torch
    ncopy = 64 << 20
    csrc = torch.empty(ncopy, dtype=torch.float32, device="cuda").normal_()
    cdst = torch.empty_like(csrc)
    for _ in range(3):
        mdnn.mdnn_cast(ncopy, csrc, mdnn.F32, cdst, mdnn.F32)
    _sync()
    del csrc, cdst


def _workloads_bench(mdnn):
    """The LeNet bf16 and fp32 MLP training steps, eager and as recorded graphs."""
    import workloads as W
    wl = {}
    for c in (W.lenet_bf16(), W.mlp784_fp32()):
        n2, xs2, ts2 = _train_setup(mdnn, c)
        m2 = _time_steps(n2, xs2, ts2, 50, 5)
        g2 = _time_graph_steps(n2, xs2, ts2, 200, 5)
        wl[c.name] = {"ms_per_step": round(m2, 4), "samples_per_s": round(c.batch / (m2 * 1e-3), 1),
                      "tflops": round(c.flops_per_step() / (m2 * 1e-3) / 1e12, 2),
                      "graph_ms_per_step": round(g2, 4),
                      "graph_samples_per_s": round(c.batch / (g2 * 1e-3), 1)}
        n2.close()
    return wl


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--quick", action="store_true", help="headline only (no sub-benchmarks)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--only", choices=["gemm", "conv", "split3", "workloads", "async", "clock", "fuse_ab"],
                    help="profiling runs: the counter calibration copy and one sub-benchmark, printed as JSON "
                         "(no headline line)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the step runs on one GPU (no collectives are implemented); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2011_11188_amd as mdnn
    import workloads as W
    if not torch.cuda.is_available():
        print("bench.py: no GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)

    if args.only:
        _copy_calibration(mdnn)
        subs = {"gemm": _gemm_sweep, "conv": _conv_bench, "split3": _split3_sweep, "workloads": _workloads_bench,
                "async": _async_bench, "clock": _sustained_clock, "fuse_ab": _fuse_ab}
        print(json.dumps({args.only: subs[args.only](mdnn), "clocks": _clocks()}), flush=True)
        return

    clocks_before = _clocks()
    cfg = W.wide_mlp_fp16()
    net, xs, ts = _train_setup(mdnn, cfg, fuse_update=FUSE_UPDATE)
    check = _UpdateCheck(mdnn, net)
    ms = _time_steps(net, xs, ts, args.steps, args.warmup, check)
    applied = check.stop(args.steps)
    if not applied:
        print("[bench] WARNING: a timed step overflowed and skipped its update", file=sys.stderr, flush=True)
    samples = cfg.batch / (ms * 1e-3)
    step_tf = cfg.flops_per_step() / (ms * 1e-3) / 1e12
    print(f"[bench] {cfg.name}: {ms:.3f} ms/step, {samples:.0f} samples/s, "
          f"{step_tf:.1f} TFLOP/s", file=sys.stderr, flush=True)
    graph_ms = _time_graph_steps(net, xs, ts, args.steps, args.warmup, check)
    graph_applied = check.stop(args.steps)
    print(f"[bench] {cfg.name} as a recorded graph: {graph_ms:.3f} ms/step", file=sys.stderr, flush=True)

    # every kernel instantiation (layout, output type, tile) of the step's
    # GEMMs, its launches replayed as the step issues them; the dominant
    # kernel is the one whose launches take the most time per step
    gemms = _step_gemms(cfg, FUSE_UPDATE)
    groups = {}
    for g in gemms:
        groups.setdefault((g[0], g[4], _kernel_choice(g[0], g[1], g[2], g[3])), []).append(g)
    best, step_groups = None, {}
    for key, grp in groups.items():
        mpl, fpl = _replay_group(mdnn, net, cfg, grp, reps=max(5, args.steps // 2))
        total = mpl * len(grp)
        tf = fpl / (mpl * 1e-3) / 1e12
        step_groups[f"{key[0]} f16 -> {key[1]}, {key[2]}"] = {
            "launches_per_step": len(grp), "avg_launch_ms": round(mpl, 4), "flop_per_launch": fpl,
            "tflops": round(tf, 1), "mfma_frac": round(tf / PEAK_F16_TFLOPS, 4), "ms_per_step": round(total, 4)}
        if best is None or total > best[0]:
            best = (total, key, mpl, fpl, len(grp))
    _, key, mpl, fpl, nl = best
    achieved = fpl / (mpl * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_F16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_F16_TFLOPS, 4), "traffic": None,
                "kernel": f"{key[2]}, {key[0]} f16 -> {key[1]}, {nl} launches per step",
                "avg_launch_ms": round(mpl, 4), "flop_per_launch": fpl}
    if key[1] == UPDATE_OUT:
        # the product's MFMA work and then its update's HBM bytes (operands,
        # then weights and momentum read and written, the fp16 copy written),
        # one after the other in each workgroup: the bound is their sum
        g = groups[key][0]
        mn = g[1] * g[2]
        upd_bytes = 2.0 * (g[1] + g[2]) * g[3] + mn * (18 if cfg.momentum else 10)
        t_bound = fpl / (PEAK_F16_TFLOPS * 1e12) + upd_bytes / (PEAK_HBM_GBS * 1e9)
        roofline["update_bytes_per_launch"] = upd_bytes
        roofline["mfma_then_hbm_bound_frac"] = round(t_bound / (mpl * 1e-3), 4)
    print(f"[bench] dominant kernel {roofline['kernel']}: {mpl:.4f} ms/launch, "
          f"{achieved:.1f} TFLOP/s", file=sys.stderr, flush=True)

    _copy_calibration(mdnn)
    traffic = _traffic_record(roofline["kernel"])
    if traffic is not None:
        roofline["traffic"] = traffic

    line = {
        "metric": METRIC, "value": round(samples, 1), "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic (seeded N(0,1) inputs and targets, He-normal weights)",
        "config": {"workload": f"{cfg.name}: wide regression MLP 1024->4x4096(ReLU)->1, MSE, "
                               "fp16 storage, fp32 accumulate + master weights, dynamic loss "
                               f"scaling (2^16), SGD momentum {cfg.momentum}, lr {cfg.lr:g}",
                   "global_batch": cfg.batch, "parallelism": "single GPU", "fuse_update": FUSE_UPDATE,
                   "step_tflops": round(step_tf, 1),
                   "graph_ms_per_step": round(graph_ms, 4),
                   "every_timed_update_applied": bool(applied and graph_applied),
                   "step_mfma_frac": round(step_tf / PEAK_F16_TFLOPS, 4),
                   "flop_per_step": cfg.flops_per_step()},
        "roofline": roofline,
        "step_gemm_kernels": step_groups,
    }
    if not args.quick:
        line["gemm_sweep"] = _gemm_sweep(mdnn)
        print("[bench] gemm sweep done", file=sys.stderr, flush=True)
        line["conv"] = _conv_bench(mdnn)
        print("[bench] conv done", file=sys.stderr, flush=True)
        line["gemm_fp32_split3"] = _split3_sweep(mdnn)
        print("[bench] fp32 split3 sweep done", file=sys.stderr, flush=True)
        line["workloads"] = _workloads_bench(mdnn)
        print("[bench] workloads done", file=sys.stderr, flush=True)
        line["async_sgd"] = _async_bench(mdnn)
        print("[bench] async sgd done", file=sys.stderr, flush=True)
        if not _under_profiler():
            line["sustained_clock"] = _sustained_clock(mdnn, net, xs, ts, cfg)
            print("[bench] sustained clock done", file=sys.stderr, flush=True)
    line["clocks"] = {"before": clocks_before, "after": _clocks()}
    if not args.no_cpu:
        line["cpu_baseline"] = _cpu_baseline(cfg)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
