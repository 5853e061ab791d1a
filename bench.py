#!/usr/bin/env python3
"""Throughput of the DP-masked linear path on one MI355X.

Default workload: one step = the whole hot path for the 36-layer Qwen3-4B-shaped
projection stack at a 1024-token prefill: for each layer and projection group (QKV
2560->6144, O 4096->2560, gate/up 2560->19456, down 9728->2560) noise + mask (one
kernel) and the GEMM with the fused unmask epilogue (one kernel).  Weights are bf16
~ N(0, 0.02^2) (random init, stored once in the MFMA kernels' tiled load order),
activations float32 ~ N(0, 1), Gaussian mechanism (Prop. 2) with Delta = 1, eps = 1
(the work does not depend on the noise scale); the corrections eta W^T are
precomputed outside the timed region (the paper's offline step) and reported
separately.  The timed steps are captured, in order, as one HIP graph and replayed
once (after an untimed replay), so the host launches once for all of them.

The same line carries `legs`, the other workloads measured the same way: the
28-layer Llama-3.2-3B stack at 512 tokens, one Llama layer at 128 tokens (8 weight
sets cycled so the 201 MB per layer streams from HBM, not the 256 MB MALL), and
Qwen3-4B decode steps of M = 1, 4, 16, 64 tokens at position 1024 of a 2048-position
correction bank (per step one launch draws every layer's masks, then each projection
is one launch that forms fl32(X + eta), multiplies and unmasks).  --workload selects
another workload as the headline (legs are then skipped), e.g. the single float32
projection or the LM heads.

Fields beyond the common contract: ``roofline`` -- the dominant launch (the
projection group with the most flops: gate/up) against the MFMA or HBM peak by its
algorithmic intensity, each group's launches for every layer back to back in one HIP
graph, bracketed by HIP events on the stream they run on; ``traffic`` from the
committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary of the workload when the kernel
sources still match it, else null; ``step``, the whole step's fraction; ``launches``,
every group's GEMM launch; the noise + mask launch times and their share of the
step.  ``cpu_baseline`` (the oracle on a bounded sample of the same workload) and
``fp_error`` (the analogue of the paper's Table 4: the GPU path's error against the
oracle per mechanism and eps at the paper's noise scale), both from the one CPU leg
that runs the oracle; ``modes`` (the other precision modes); ``correction_ms``
(offline precompute); ``down_f64`` (the Down projection at Theorem 3's noise scale
through the binary64 path against the bf16x3 one: time and error); ``noise_bank`` (one
layer's correction banks for 2048 positions: created from the GPU corrections into
files, then loaded as decode steps and as one batch); ``noise_scale`` (the offline
noise-scale step of the same model: spectral norms of W_val, W_up, W_gate and W_down
by the power method, the sensitivity bounds of Theorems 1-3 from them, and the time
of one power-method round against the HBM roofline of reading W once).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "masked-linear TFLOP/s (noise+mask+GEMM+unmask) and % MFMA/HBM roofline"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFS = 2500.0
FP32_PEAK_TFS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=WORKLOADS)
    ap.add_argument("--prec", default="bf16x3", choices=["bf16x3", "bf16", "f32"])
    ap.add_argument("--mech", default="gaussian", choices=["gaussian", "laplace", "none"])
    ap.add_argument("--eps", type=float, default=1.0)
    ap.add_argument("--delta", type=float, default=1.0)
    ap.add_argument("--weight-sets", type=int, default=8)
    ap.add_argument("--layout", default="auto", choices=["auto", "tiled", "row-major"],
                    help="bfloat16 weights in the tiled load order (splitee_tile_weights) or row-major; "
                         "auto: row-major for one or two tokens of projections under 16384 rows (the "
                         "vector-ALU GEMV reads whole rows), tiled otherwise (gate/up and the LM heads "
                         "at one or two tokens; 'mixed' when a workload has both)")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of HIP graphs")
    ap.add_argument("--step-masks-max-m", type=int, default=STEP_MASKS_MAX_M,
                    help="up to this many tokens, draw the masks of a step in one launch")
    ap.add_argument("--no-modes", action="store_true", help="skip the other precision modes")
    ap.add_argument("--no-legs", action="store_true",
                    help="skip the other workloads measured beside the default one")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-noise-scale", action="store_true", help="skip the noise-scale leg")
    ap.add_argument("--noise-scale-only", action="store_true", help="run only the noise-scale leg")
    ap.add_argument("--power-iters", type=int, default=300)
    ap.add_argument("--no-noise-bank", action="store_true", help="skip the noise-bank leg")
    ap.add_argument("--no-down-f64", action="store_true", help="skip the binary64 Down leg")
    ap.add_argument("--down-f64-only", action="store_true", help="run only the binary64 Down leg")
    ap.add_argument("--noise-bank-only", action="store_true", help="run only the noise-bank leg")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (HBM counter calibration) and exit")
    ap.add_argument("--counter-launches", type=int, default=0,
                    help="only run each projection group's GEMM launch this many times, eagerly and in order "
                         "(for rocprofv3 counter runs), and exit")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample")
    return ap.parse_args()


DEFAULT_WORKLOAD = "qwen3-4b-36l-m1024"
WORKLOADS = ["llama3b-layer-m128", "single-fp32-m32", "llama3b-28l-m512", "qwen3-4b-36l-m1024",
             "qwen3-4b-decode-m1", "qwen3-4b-decode-m4", "qwen3-4b-decode-m16", "qwen3-4b-decode-m64",
             "llama3b-lmhead-m1", "llama3b-lmhead-m15", "llama3b-lmhead-m128",
             "qwen3-4b-lmhead-m1", "qwen3-4b-lmhead-m15"]
STEP_MASKS_MAX_M = 64  # up to this many tokens the masks of a step are drawn in one launch
DECODE_POS = 1024  # decode position t: rows [t, t+M) of the 2048-position correction bank


def workload_spec(WL, name):
    """(projections, tokens, layers per step, weight sets, weight dtype, bank rows, row0)."""
    if name == "single-fp32-m32":
        c = WL.SINGLE_FP32
        return [WL.Projection("single", c["K"], c["N"], 0)], c["M"], 1, 8, "f32", 0, 0
    if name == "llama3b-layer-m128":
        return WL.LLAMA_3B.projections(), 128, 1, 8, "bf16", 0, 0
    if name == "llama3b-28l-m512":
        return WL.LLAMA_3B.projections(), 512, WL.LLAMA_3B.layers, 1, "bf16", 0, 0
    if name == "qwen3-4b-36l-m1024":
        return WL.QWEN3_4B.projections(), 1024, WL.QWEN3_4B.layers, 1, "bf16", 0, 0
    if name.startswith("qwen3-4b-decode-m"):
        m = int(name.rsplit("m", 1)[1])
        return WL.QWEN3_4B.projections(), m, WL.QWEN3_4B.layers, 1, "bf16", 2048, DECODE_POS
    if "-lmhead-m" in name:
        # the vocabulary projection alone (788 / 778 MB of bf16 W, past the MALL by itself):
        # decode sizes read their correction rows from a 2048-position bank
        model = WL.QWEN3_4B if name.startswith("qwen") else WL.LLAMA_3B
        m = int(name.rsplit("m", 1)[1])
        bank, row0 = (2048, DECODE_POS) if m <= 16 else (0, 0)
        return [model.lm_head()], m, 1, 1, "bf16", bank, row0
    raise ValueError(name)


class Path:
    """Device buffers of one workload: per layer (or weight set) and projection
    group, the weights, the precomputed correction rows and the outputs.

    Prefill-sized M: per projection, noise + mask in one kernel, then the GEMM with
    the unmask epilogue.  Up to `step_masks_max_m` tokens (64: measured faster at 64,
    slower at 128 and 1024) the noise does not fill the chip one projection at a time, so
    one launch per step draws the masks of every layer and projection group (the noise
    does not depend on the input), and the fused call of each projection forms
    fl32(X + eta) from the drawn mask inside its GEMM: the skinny kernel at M <= 16, the
    streamed kernel's in-kernel mask above."""

    def __init__(self, torch, sp, WL, name, prec, mech, delta, eps, weight_sets, layout="auto",
                 step_masks_max_m=STEP_MASKS_MAX_M):
        self.torch, self.sp = torch, sp
        self.prec, self.mech, self.delta, self.eps = prec, mech, delta, eps
        (self.projs, self.M, self.layers_per_step, nsets, self.w_dtype, bank_rows,
         self.row0) = workload_spec(WL, name)
        if self.layers_per_step == 1 and weight_sets and nsets > 1:
            nsets = weight_sets
        self.nsets = nsets if self.layers_per_step == 1 else 1
        nlayers = self.layers_per_step * self.nsets
        dev = "cuda"
        M = self.M
        g = torch.Generator(device=dev)
        g.manual_seed(1)
        wt = sp.SPLITEE_F32 if self.w_dtype == "f32" else sp.SPLITEE_BF16
        can_tile = wt == sp.SPLITEE_BF16 and prec != sp.SPLITEE_PREC_F32
        self.tiled = [can_tile and weight_tiled(layout, M, p.N, p.K) for p in self.projs]
        self.wt = [sp.SPLITEE_BF16_TILED if t else wt for t in self.tiled]
        self.layout = "tiled" if all(self.tiled) else ("row-major" if not any(self.tiled) else "mixed")
        self.X, self.Xt, self.Y, self.ws = [], [], [], []
        for p in self.projs:
            self.X.append(torch.randn((M, p.K), generator=g, device=dev, dtype=torch.float32))
            planes = 3 if prec == sp.SPLITEE_PREC_BF16X3 else 1
            dt = torch.float32 if prec == sp.SPLITEE_PREC_F32 else torch.int16
            self.Xt.append(torch.empty((planes, M, p.K), dtype=dt, device=dev))
            self.Y.append(torch.empty((M, p.N), dtype=torch.float32, device=dev))
        self.step_masks = M <= step_masks_max_m and prec != sp.SPLITEE_PREC_F32
        for p in self.projs:
            self.ws.append(sp.workspace(M, p.N, p.K, prec, dev, gemm_only=not self.step_masks))
        # drawn per step: the masks of every layer of a step, [layer][token][k] per projection group
        self.eta = [torch.empty((self.layers_per_step, M, p.K), dtype=torch.float32, device=dev)
                    for p in self.projs] if self.step_masks else None
        self.sid_step = WL.stream_id(1, 0) - WL.stream_id(0, 0)
        self.W, self.C, self.sid = [], [], []
        for l in range(nlayers):
            Ws, sids = [], []
            for i, p in enumerate(self.projs):
                W = torch.randn((p.N, p.K), generator=g, device=dev) * 0.02
                if wt == sp.SPLITEE_BF16:
                    W = W.to(torch.bfloat16)
                    if self.tiled[i]:  # stored once in the kernels' load order, like loading a checkpoint
                        W = sp.tile_weights(W)
                Ws.append(W)
                sids.append(WL.stream_id(l, p.group))
            self.W.append(Ws)
            self.sid.append(sids)
        torch.cuda.synchronize()
        # offline corrections (binary32-accurate mode) for the rows the steps consume;
        # decode keeps them in a 2048-position bank and reads rows [t, t+M)
        cprec = sp.SPLITEE_PREC_F32 if wt == sp.SPLITEE_F32 else sp.SPLITEE_PREC_BF16X3
        t0 = time.perf_counter()
        for l in range(nlayers):
            Cs = []
            for i, p in enumerate(self.projs):
                c = sp.correction(self.W[l][i], M, mech, delta, eps, 0, self.sid[l][i], self.row0, cprec)
                if bank_rows:
                    bank = torch.zeros((bank_rows, p.N), dtype=torch.float32, device=dev)
                    bank[self.row0:self.row0 + M].copy_(c)
                    c = bank[self.row0:self.row0 + M]
                Cs.append(c)
            self.C.append(Cs)
        torch.cuda.synchronize()
        self.correction_ms = (time.perf_counter() - t0) * 1e3 / nlayers * self.layers_per_step

    def gemm(self, l, i):
        """The GEMM + unmask launch of projection group i of layer (or weight set) l
        (masks drawn per step: mask + GEMM + unmask, on the mask drawn for the layer)."""
        p, M = self.projs[i], self.M
        W, C = self.W[l][i], self.C[l][i]
        if self.step_masks:
            self.sp.splitee_masked_linear_fused(
                self.X[i], p.K, W, self.wt[i], p.K, C, C.stride(0), self.Y[i], p.N, M, p.N, p.K, self.mech,
                self.delta, self.eps, 0, self.sid[l][i], self.row0, self.eta[i][l % self.layers_per_step], self.prec,
                self.ws[i][0], self.ws[i][1])
        else:
            self.sp.splitee_masked_linear_unmask(self.Xt[i], self.prec, p.K, W, self.wt[i], p.K, C,
                                                 C.stride(0), self.Y[i], p.N, M, p.N, p.K,
                                                 self.ws[i][0], self.ws[i][1])

    def draw_masks(self, base):
        """Masks drawn per step: one launch draws the masks of all layers and projection groups of a step."""
        Ks = [p.K for p in self.projs]
        self.sp.splitee_noise_gen_multi(self.eta, Ks, Ks, self.sid[base], self.M, self.mech, self.delta,
                                        self.eps, 0, self.row0, reps=self.layers_per_step,
                                        rep_strides=[self.M * K for K in Ks], rep_sid_step=self.sid_step)

    def mask(self, l, i):
        """Prefill: the noise + mask launch of projection group i of layer (or weight set) l."""
        p = self.projs[i]
        self.sp.splitee_noise_mask(self.X[i], p.K, self.Xt[i], self.prec, p.K, self.M, p.K, self.mech,
                                   self.delta, self.eps, 0, self.sid[l][i], self.row0)

    def launches(self, s):
        """All kernels of step s: noise, mask, GEMM and unmask of every projection."""
        base = (s % self.nsets) * self.layers_per_step
        if self.step_masks:
            self.draw_masks(base)
        for l in range(base, base + self.layers_per_step):
            for i in range(len(self.projs)):
                if not self.step_masks:
                    self.mask(l, i)
                self.gemm(l, i)

    def flops(self):
        return self.layers_per_step * sum(2.0 * self.M * p.N * p.K for p in self.projs)

    def gemm_bytes(self):
        """Algorithmic bytes of each GEMM + unmask launch: W, float32 X (and, in the
        fused call that forms the masked input from a drawn mask, float32 eta), C and Y."""
        wb = 4.0 if self.w_dtype == "f32" else 2.0
        xb = 8.0 if self.step_masks else 4.0
        return [wb * p.N * p.K + xb * self.M * p.K + 8.0 * self.M * p.N for p in self.projs]


def run_mode(torch, sp, WL, name, prec, args, steps, warmup):
    path = Path(torch, sp, WL, name, prec, sp.MECHS[args.mech], args.delta, args.eps,
                args.weight_sets, args.layout, args.step_masks_max_m)
    nsets = path.nsets
    graphs = None
    if not args.no_graph:
        # one HIP graph per step variant; capturing records the same kernels
        for s in range(nsets):
            path.launches(s)  # warm the launch path before capture
        torch.cuda.synchronize()
        graphs = []
        for s in range(nsets):
            gph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gph):
                path.launches(s)
            graphs.append(gph)
        torch.cuda.synchronize()
        # the timed steps, in order, as one graph: the host launches once instead of once per
        # step (a graph launch costs tens of microseconds of host time, more than a small step)
        timed = torch.cuda.CUDAGraph()
        with torch.cuda.graph(timed):
            for s in range(steps):
                path.launches(s)
        torch.cuda.synchronize()

    def run(s):
        if graphs is not None:
            graphs[s % nsets].replay()
        else:
            path.launches(s)

    for s in range(warmup):
        run(s)
    if graphs is not None:
        timed.replay()  # its first launch uploads the graph: untimed
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if graphs is not None:
        timed.replay()
    else:
        for s in range(steps):
            run(s)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    if graphs is not None:
        del timed

    # per-launch duration of the GEMM + unmask kernel of each projection group, and of the
    # noise + mask launch (per projection group, or the one launch per step that draws
    # every layer's masks): the launches for every layer / weight set of the run,
    # back to back in one HIP graph (eager launches when --no-graph), bracketed by HIP
    # events recorded on the stream the kernels run on; averaged over launches and repeats
    nproj = len(path.projs)
    reps = max(2, min(steps, 20))
    stream = torch.cuda.current_stream()

    def time_launches(fn, n_launch):
        if graphs is not None:
            fn()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                fn()
            go = g.replay
        else:
            go = fn
        go()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            go()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (reps * n_launch)

    n_layers = path.nsets * path.layers_per_step

    def each_layer(f, i):
        for l in range(n_layers):
            f(l, i)

    per_proj_us = [time_launches(lambda i=i: each_layer(path.gemm, i), n_layers) for i in range(nproj)]
    if path.step_masks:
        # one launch per step: 16 of them per graph, so that the graph launch itself is amortised
        mask_us = [time_launches(lambda: [path.draw_masks((s % path.nsets) * path.layers_per_step)
                                          for s in range(16)], 16)]
    else:
        mask_us = [time_launches(lambda i=i: each_layer(path.mask, i), n_layers) for i in range(nproj)]
    return path, ms, per_proj_us, mask_us


def cpu_baseline_leg(torch, sp, WL, target_s, projs, tokens, w_dtype, workload, deltas=None):
    """The CPU leg, the only part of the bench that runs the oracle (test
    infrastructure): (1) the oracle (binary128 noise, mask, binary64 GEMM, correction
    GEMM, unmask) timed on a row sample of one layer of the workload on the host's
    cores, in TFLOP/s of the sample's algorithmic work (2 x rows x N x K per projection
    group); (2) the floating-point error of the GPU path against the oracle, the
    analogue of the paper's Table 4 (see fp_error_table)."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    Ws = [WL.gen_w(p.N, p.K, seed=2 + p.group, dtype=w_dtype) for p in projs]

    def run(rows):
        t0 = time.perf_counter()
        for p, W in zip(projs, Ws):
            X = WL.gen_x(rows, p.K, seed=1)
            sid = WL.stream_id(0, p.group)
            eta = O.noise(rows, p.K, O.MECH_GAUSSIAN, 1.0, 1.0, 0, sid, 0)
            Xt = O.mask(X, eta)
            R = O.gemm64(Xt, W).astype(np.float32)
            C = O.gemm64(eta, W).astype(np.float32)
            O.unmask(R, C)
        return time.perf_counter() - t0

    run(1)  # warm-up (library loads, first-touch)
    r0 = min(tokens, 8)
    per_row = run(r0) / r0  # includes the per-call fixed cost, so rows is not overestimated
    rows = int(max(1, min(tokens, target_s / 2 / per_row)))
    total, reps = 0.0, 0
    while reps == 0 or (total < target_s and reps < 100):
        total += run(rows)
        reps += 1
    flops = reps * sum(2.0 * rows * p.N * p.K for p in projs)
    base = {"value": flops / total / 1e12, "unit": "TFLOP/s",
            "cores": int(max(O.num_threads(), blas_threads)), "kind": "oracle",
            "sample": "%d x %d of %d tokens of one layer's %d projection group(s): noise, mask, GEMM, "
                      "correction GEMM, unmask; %.1f s" % (reps, rows, tokens, len(projs), total)}
    fp = None
    if w_dtype == "bf16":
        del Ws
        fp = fp_error_table(torch, sp, WL, O, np, projs, tokens, workload, deltas)
    return base, fp


def fp_error_table(torch, sp, WL, O, np, projs, M, workload, deltas=None, nrows=4, ncols=256,
                   eps_list=(0.5, 2.0, 8.0)):
    """Table 4 analogue: the fused bf16x3 call of the workload's launch configuration
    (full M, tiled W) per projection group, mechanism and eps at the paper's noise
    scale (Theorems 1-3: Delta_LN for QKV and gate/up, Delta_att for O, Delta_act for
    Down -- from the noise-scale leg when it ran, else the closed forms for alpha = 1,
    beta = 0 and ||W||_2 ~ 0.02 (sqrt(rows) + sqrt(cols))), against the oracle on
    nrows x ncols sampled outputs per group: mean |err|, mean Eq. fp-log-bound, their
    ratio, the share of elements above it, max err / Theorem-4 gate, and mean |err|
    eps.  QKV, O and gate/up are pooled (the paper's offloaded operators); Down, which
    the paper keeps in the TEE, is reported on its own."""
    model = WL.QWEN3_4B if workload.startswith("qwen") else WL.LLAMA_3B
    d = model.hidden
    if deltas is None:
        ln = 2.0 * d ** 0.75
        sn = lambda r, c: 0.02 * (r ** 0.5 + c ** 0.5)
        deltas = {"ln": ln, "att": ln * sn(model.kv_dim, d), "act": 2.0 * d * d * sn(model.ff, d) ** 2}
    dsel = {"qkv": deltas["ln"], "gate_up": deltas["ln"], "o": deltas["att"], "down": deltas["act"]}
    mechs = {"laplace": (sp.SPLITEE_MECH_LAPLACE, O.MECH_LAPLACE), "gaussian": (sp.SPLITEE_MECH_GAUSSIAN,
                                                                                 O.MECH_GAUSSIAN)}
    g = np.random.Generator(np.random.PCG64(5))
    acc = {}
    t0 = time.perf_counter()
    for p in projs:
        tg = torch.Generator(device="cuda")
        tg.manual_seed(100 + p.group)
        Wb = (torch.randn((p.N, p.K), generator=tg, device="cuda") * 0.02).to(torch.bfloat16)
        W = Wb.float().cpu().numpy()
        T = sp.tile_weights(Wb)
        del Wb
        X = WL.gen_x(M, p.K, seed=1)
        Xd = torch.from_numpy(X).cuda()
        rows = g.choice(M, size=min(M, nrows), replace=False)
        cols = g.choice(p.N, size=min(p.N, ncols), replace=False)
        Ws = W[cols]
        ref = O.gemm64(X[rows], Ws)
        sid = WL.stream_id(0, p.group)
        for mname, (gm, om) in mechs.items():
            for eps in eps_list:
                C = sp.correction(T, M, gm, dsel[p.name], eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
                Y = sp.masked_linear_fused(Xd, T, C, gm, dsel[p.name], eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
                Yh = Y[torch.from_numpy(rows).cuda()].cpu().numpy()[:, cols].astype(np.float64)
                del C, Y
                e = np.stack([O.noise(1, p.K, om, dsel[p.name], eps, 0, sid, int(i))[0] for i in rows])
                b = O.error_bounds(X[rows], e, O.mask(X[rows], e), Ws, O.PREC_BF16X3)
                err = np.abs(Yh - ref)
                key = (mname, eps, "down" if p.name == "down" else "offloaded")
                a = acc.setdefault(key, {"err": [], "logb": [], "gate": [], "y": []})
                a["err"].append(err.ravel())
                a["logb"].append(b["logb"].ravel())
                a["gate"].append((err / b["gate"]).ravel())
                a["y"].append(np.abs(ref).ravel())
        del T
        torch.cuda.empty_cache()
    table = {}
    for (mname, eps, grp), a in sorted(acc.items()):
        err, logb = np.concatenate(a["err"]), np.concatenate(a["logb"])
        y = np.concatenate(a["y"])
        table.setdefault(grp, {}).setdefault(mname, {})["%g" % eps] = {
            "mean_err": float("%.4g" % err.mean()), "mean_logb": float("%.4g" % logb.mean()),
            "logb_over_err": round(float(logb.mean() / err.mean()), 2),
            "pct_above_logb": round(100.0 * float(np.mean(err > logb)), 3),
            "max_err_over_gate": float("%.3g" % np.concatenate(a["gate"]).max()),
            "mean_err_times_eps": float("%.4g" % (err.mean() * eps)),
            "median_rel_err": float("%.3g" % np.median(err / y))}
    return {"what": "fused bf16x3 at full size (tiled W) against the oracle on %d x %d sampled outputs per "
                    "projection group; paper-scale Delta per group; 'offloaded' pools %s" %
                    (nrows, ncols, ", ".join(p.name for p in projs if p.name != "down")),
            "delta": {k: float("%.6g" % v) for k, v in dsel.items()}, "model": model.name, "tokens": M,
            "seconds": round(time.perf_counter() - t0, 1), "table": table}


GEMM_SOURCES = ["paper_2609_15039_amd/csrc/gemm.hip", "paper_2609_15039_amd/csrc/common.hpp"]


def gemm_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def weight_tiled(layout, M, N, K):
    """Whether a bfloat16 projection of N output rows and K columns at M tokens stores W
    tiled.  auto: one or two tokens run a vector-ALU GEMV, on row-major W (whole rows per
    wave) or on tiled W (32-row blocks); measured on the Llama-3.2-3B and Qwen3-4B
    projections and on 2560-24576 x 2560-4096 matrices, the tiled one is faster from 6144
    rows up at one token (Qwen3-4B QKV 9.6 -> 9.0 us, 6144 x 3072 10.8 -> 10.4 us, Llama-3.2-3B
    gate/up 21.9 -> 19.4 us; 5120 rows 9.3 against 9.8) and from about 12 M elements up at two
    (Qwen3-4B Down 20.2 -> 15.1 us), the row-major one below (Qwen3-4B O at one token 7.0 us
    against 8.9); every other M runs the MFMA kernels on tiled W."""
    if layout == "auto":
        if M == 1:
            return N >= 6144
        if M == 2:
            return N * K >= 12 * 2**20
        return True
    return layout == "tiled"


def measured_traffic(workload, prec_name, layout, names):
    """HBM bytes per GEMM + unmask launch from the committed rocprofv3 counter
    summary of this workload (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy's
    readings), or None when there is none or the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s_%s.md" % (workload, prec_name, layout))
    if not os.path.exists(path):
        return None
    sha, rows = None, {}
    with open(path) as fh:
        for line in fh:
            if line.startswith("source-sha256:"):
                sha = line.split(":", 1)[1].strip()
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            if len(cells) >= 7 and cells[0] in names:
                try:
                    rows[cells[0]] = float(cells[6])
                except ValueError:
                    pass
    if sha != gemm_source_sha() or set(rows) != set(names):
        return None
    return rows


def counter_launches(torch, sp, WL, args, prec):
    """The GEMM launches alone, for counter collection: after set-up, `n` rounds of
    one launch per projection group (layer 0), in projection order, each followed by
    a device synchronization; these are the run's last dispatches."""
    path = Path(torch, sp, WL, args.workload, prec, sp.MECHS[args.mech], args.delta, args.eps, 1, args.layout,
                args.step_masks_max_m)
    if path.step_masks:
        path.draw_masks(0)
    else:
        for i, p in enumerate(path.projs):
            sp.splitee_noise_mask(path.X[i], p.K, path.Xt[i], path.prec, p.K, path.M, p.K, path.mech,
                                  path.delta, path.eps, 0, path.sid[0][i], path.row0)
    torch.cuda.synchronize()
    for _ in range(args.counter_launches):
        for i in range(len(path.projs)):
            path.gemm(0, i)
            torch.cuda.synchronize()
    print(json.dumps({"counter_launches": args.counter_launches, "projections": [p.name for p in path.projs],
                      "algorithmic_bytes": [int(b) for b in path.gemm_bytes()]}), flush=True)


def copy_probe(mib):
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(2):
        torch.mul(x, 1.0, out=y)  # reads mib MiB, writes mib MiB
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_mib": mib, "read_bytes": n * 4, "write_bytes": n * 4}), flush=True)


def noise_scale_leg(torch, sp, WL, workload, iters):
    """Offline noise scale of one layer of the workload's model (random-init weights,
    normalisation parameters from workloads.gen_norm): ||W||_2 by the power method,
    Delta of Theorems 1-3, and the time of one round (difference of two runs of
    different lengths, HIP events on the stream the kernels run on)."""
    model = WL.QWEN3_4B if workload.startswith("qwen") else WL.LLAMA_3B
    d = model.hidden
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    mats = {"w_val": (model.kv_dim, d), "w_up": (model.ff, d), "w_gate": (model.ff, d),
            "w_down": (d, model.ff)}
    Ws = {k: (torch.randn(s, generator=g, device="cuda") * 0.02).to(torch.bfloat16) for k, s in mats.items()}
    sig = {k: sp.spectral_norm(W, iters, 0, WL.stream_id(0, 16 + i)) for i, (k, W) in enumerate(Ws.items())}
    alpha, beta = (torch.from_numpy(a).cuda() for a in WL.gen_norm(d))
    delta = {"ln": sp.sensitivity(sp.SPLITEE_BOUND_LN, alpha),
             "att": sp.sensitivity(sp.SPLITEE_BOUND_ATT, alpha, w_norm_a=sig["w_val"]),
             "act": sp.sensitivity(sp.SPLITEE_BOUND_ACT, alpha, beta, sig["w_up"], sig["w_gate"])}
    stream = torch.cuda.current_stream()

    def timed(W, n):
        nbytes = sp.splitee_spectral_norm_workspace_bytes(W.shape[0], W.shape[1], n)
        ws = torch.empty(nbytes + 256, dtype=torch.uint8, device="cuda")
        ws = ws[(-ws.data_ptr()) % 256:][:nbytes]
        best = float("inf")
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            sp.splitee_spectral_norm(W, sp.SPLITEE_BF16, W.shape[1], W.shape[0], W.shape[1], n, 0, 0, ws,
                                     nbytes, stream=stream)
            b.record(stream)
            b.synchronize()
            best = min(best, a.elapsed_time(b) * 1e3)
        return best

    round_us, gbs = {}, {}
    for k, W in Ws.items():
        timed(W, 5)
        t = (timed(W, 60) - timed(W, 10)) / 50.0
        round_us[k] = round(t, 2)
        gbs[k] = round(W.numel() * 2 / (t * 1e-6) / 1e9, 1)
    big = max(Ws, key=lambda k: Ws[k].numel())
    return {"model": model.name, "iters": iters, "sigma": {k: round(v, 6) for k, v in sig.items()},
            "delta": {k: float("%.6g" % v) for k, v in delta.items()},
            "round_us": round_us,
            "roofline": {"bound": "hbm", "kernel": "power-method round (pi_round + pi_reduce), %s %dx%d bf16"
                         % ((big,) + tuple(Ws[big].shape)),
                         "achieved": gbs[big], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(gbs[big] / HBM_PEAK_GBS, 4),
                         "bytes_per_round": {k: int(W.numel() * 2) for k, W in Ws.items()},
                         "achieved_per_matrix": gbs}}


def noise_bank_leg(torch, sp, WL, workload, rows=2048):
    """The noise bank of one layer of the workload's model (its projection groups, random-init
    bf16 weights, corrections in BF16X3): create the banks for `rows` positions in a
    temporary directory, then load them as decode steps (16 rows per group per step) and
    as one batch of all rows.  Times are host wall-clock around synchronising calls."""
    import shutil
    import tempfile
    model = WL.QWEN3_4B if workload.startswith("qwen") else WL.LLAMA_3B
    projs = model.projections()
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    Ws = [(torch.randn((p.N, p.K), generator=g, device="cuda") * 0.02).to(torch.bfloat16) for p in projs]
    d = tempfile.mkdtemp(prefix="splitee-bank-")
    try:
        paths = [sp.splitee_bank_path(d, p.K, p.N, WL.stream_id(0, p.group)) for p in projs]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for p, W, path in zip(projs, Ws, paths):
            sp.bank_create(path, W, p.K, sp.SPLITEE_MECH_GAUSSIAN, 1.0, 1.0, 0, WL.stream_id(0, p.group), 0, rows)
        t_create = time.perf_counter() - t0
        banks = [sp.splitee_bank_open(path) for path in paths]
        infos = [sp.splitee_bank_info(b) for b in banks]
        Cs = [torch.empty((rows, p.N), device="cuda") for p in projs]
        steps = rows // 2 // 16
        t0 = time.perf_counter()
        for s in range(steps):
            for b, C, p in zip(banks, Cs, projs):
                sp.splitee_bank_load(b, 16, C[16 * s:], p.N, True)
        t_steps = time.perf_counter() - t0
        rest = rows - 16 * steps
        t0 = time.perf_counter()
        for b, C, p in zip(banks, Cs, projs):
            sp.splitee_bank_load(b, rest, C[16 * steps:], p.N, True)
        t_batch = time.perf_counter() - t0
        for b in banks:
            sp.splitee_bank_close(b)
    finally:
        shutil.rmtree(d, ignore_errors=True)
    row_bytes = sum(4 * p.N for p in projs)
    flops = sum(2.0 * 3 * rows * p.N * p.K for p in projs)  # three MFMA passes of the exact split
    return {"model": model.name, "groups": [p.name for p in projs], "rows": rows,
            "bytes_stored": int(sum(i["bytes_stored"] for i in infos)),
            "bytes_with_masks": int(sum(i["bytes_with_masks"] for i in infos)),
            "create_s": round(t_create, 3), "create_GBps": round(rows * row_bytes / t_create / 1e9, 3),
            "create_correction_TFLOPs_issued": round(flops / t_create / 1e12, 2),
            "decode_load_us_per_step": round(t_steps / steps * 1e6, 1),
            "decode_load_GBps": round(steps * 16 * row_bytes / t_steps / 1e9, 3),
            "batch_load_GBps": round(rest * row_bytes / t_batch / 1e9, 3)}


F64_PEAK_TFS = 78.6


def down_f64_leg(torch, sp, WL, workload, M=128, delta=1.66e8, eps=1.0, reps=20):
    """The Down projection of the workload's model at 128 tokens with the noise scale of
    Theorem 3 (Delta about 1.66e8 for random-init Llama-shaped weights, eps = 1): the
    binary64 fused call against the binary32-accurate (bf16x3) one, time per call (HIP
    events on the stream the kernels run on, mean of `reps` calls) and the error of each
    against X W^T evaluated in binary64 on the GPU (a reference for this figure only)."""
    model = WL.QWEN3_4B if workload.startswith("qwen") else WL.LLAMA_3B
    K, N = model.ff, model.hidden
    g = torch.Generator(device="cuda")
    g.manual_seed(13)
    X = torch.randn((M, K), generator=g, device="cuda")
    W = (torch.randn((N, K), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    G = sp.SPLITEE_MECH_GAUSSIAN
    sid = WL.stream_id(0, 3)
    C64 = sp.correction_f64(W, M, G, delta, eps, 0, sid, 0)
    C32 = sp.correction(W, M, G, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3)
    ws64 = sp.workspace_f64(M, N, K)
    ws32 = sp.workspace(M, N, K, sp.SPLITEE_PREC_BF16X3)
    Y64 = torch.empty((M, N), device="cuda")
    Y32 = torch.empty((M, N), device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        b.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    t64 = timed(lambda: sp.masked_linear_fused_f64(X, W, C64, G, delta, eps, 0, sid, 0, ws=ws64, Y=Y64))
    t32 = timed(lambda: sp.masked_linear_fused(X, W, C32, G, delta, eps, 0, sid, 0, sp.SPLITEE_PREC_BF16X3,
                                               ws=ws32, Y=Y32))
    ref = X.double() @ W.double().t()
    den = ref.abs()
    rel64 = ((Y64.double() - ref).abs() / den)
    rel32 = ((Y32.double() - ref).abs() / den)
    flops = 2.0 * M * N * K
    tf = flops / (t64 * 1e-6) / 1e12
    return {"model": model.name, "projection": "down", "tokens": M, "K": K, "N": N, "delta": delta, "eps": eps,
            "f64_us": round(t64, 1), "bf16x3_us": round(t32, 1), "cost_ratio": round(t64 / t32, 2),
            "f64_rel_error_median": float("%.3g" % rel64.median().item()),
            "f64_rel_error_max": float("%.3g" % rel64.max().item()),
            "bf16x3_rel_error_median": float("%.3g" % rel32.median().item()),
            "roofline": {"bound": "mfma", "kernel": "mask (binary64) + gemm_f64_kernel + f64_sum_kernel",
                         "achieved": round(tf, 2), "peak": F64_PEAK_TFS, "unit": "TFLOP/s",
                         "frac": round(tf / F64_PEAK_TFS, 4)}}


def leg_summary(sp, path, ms, per_proj_us, mask_us, prec, workload):
    """value, ms per step, and the roofline object of one workload: the dominant launch
    (the projection group with the most algorithmic flops) against the MFMA or HBM peak
    by its algorithmic intensity, every GEMM launch, the noise + mask launches, and the
    whole step (algorithmic flops / bytes of the fused minimum over ms per step)."""
    projs, M, L = path.projs, path.M, path.layers_per_step
    flops = [2.0 * M * p.N * p.K for p in projs]
    gb = path.gemm_bytes()
    planes = 3 if prec == sp.SPLITEE_PREC_BF16X3 else 1
    f32 = prec == sp.SPLITEE_PREC_F32
    mfma_peak = FP32_PEAK_TFS if f32 else BF16_PEAK_TFS
    ridge = mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9)

    def frac_of(fl, by, us):
        if fl / by < ridge:
            a = by / (us * 1e-6) / 1e9
            return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(a / HBM_PEAK_GBS, 4)}
        a = fl / (us * 1e-6) / 1e12
        return {"bound": "mfma", "achieved": round(a, 1), "peak": mfma_peak, "unit": "TFLOP/s",
                "frac": round(a / mfma_peak, 4)}

    d = max(range(len(projs)), key=lambda i: flops[i])
    roof = frac_of(flops[d], gb[d], per_proj_us[d])
    pname = {v: k for k, v in sp.PRECS.items()}[prec]
    traffic = measured_traffic(workload, pname, path.layout, [p.name for p in projs])
    roof.update({"kernel": ("%s projection: mask + GEMM + unmask in one launch (masks drawn per step)"
                            if path.step_masks else "%s projection: GEMM + unmask launch") % projs[d].name,
                 "launch_us": round(per_proj_us[d], 2), "algorithmic_bytes": int(gb[d]),
                 "algorithmic_flops": int(flops[d]), "algorithmic_ai": round(flops[d] / gb[d], 1),
                 "traffic": None if traffic is None else int(traffic[projs[d].name]),
                 "traffic_per_launch": traffic and {k: int(v) for k, v in traffic.items()}})
    if not f32 and M > 16:
        issued = planes * flops[d] / (per_proj_us[d] * 1e-6) / 1e12
        roof.update({"mfma_issued_tflops": round(issued, 1), "mfma_issued_frac": round(issued / BF16_PEAK_TFS, 4),
                     "mfma_passes": planes})
    step_flops = L * sum(flops)
    step_bytes = L * sum(gb)
    step = frac_of(step_flops, step_bytes, ms * 1e3)
    mask_total_us = (mask_us[0] if path.step_masks else L * sum(mask_us))
    step.update({"what": "whole step: noise, mask, GEMM and unmask of every projection group of %d layer(s); "
                         "algorithmic flops and fused-minimum bytes over ms per step" % L,
                 "ms": round(ms, 4), "algorithmic_flops": int(step_flops), "algorithmic_bytes": int(step_bytes),
                 "noise_mask_us": round(mask_total_us, 1),
                 "noise_mask_share": round(mask_total_us / (ms * 1e3), 4)})
    roof["step"] = step
    roof["launches"] = {p.name: dict(frac_of(flops[i], gb[i], per_proj_us[i]), launch_us=round(per_proj_us[i], 2))
                        for i, p in enumerate(projs)}
    roof["noise_mask_launch_us"] = ({"all layers": round(mask_us[0], 2)} if path.step_masks else
                                    {p.name: round(u, 2) for p, u in zip(projs, mask_us)})
    value = step_flops / (ms * 1e-3) / 1e12
    return {"value": round(value, 3), "ms_per_step": round(ms, 4), "tokens": M, "layers_per_step": L,
            "projections": {p.name: [p.K, p.N] for p in projs}, "w_layout": path.layout,
            "w_tiled": [p.name for p, t in zip(projs, path.tiled) if t], "weight_sets": path.nsets,
            "row0": path.row0}, roof


LEGS = ["llama3b-28l-m512", "llama3b-layer-m128", "qwen3-4b-decode-m1", "qwen3-4b-decode-m4",
        "qwen3-4b-decode-m16", "qwen3-4b-decode-m64"]


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the masked linear layer runs on a single MI355X "
              "(sharding over several GPUs is not implemented); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return
    import torch
    import paper_2609_15039_amd as sp
    import workloads as WL
    sp.load()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    prec = sp.PRECS[args.prec]
    if args.workload == "single-fp32-m32":
        prec = sp.SPLITEE_PREC_F32
    if args.counter_launches:
        counter_launches(torch, sp, WL, args, prec)
        return
    if args.down_f64_only:
        print(json.dumps({"down_f64": down_f64_leg(torch, sp, WL, args.workload)}), flush=True)
        return
    if args.noise_bank_only:
        print(json.dumps({"noise_bank": noise_bank_leg(torch, sp, WL, args.workload)}), flush=True)
        return
    if args.noise_scale_only:
        print(json.dumps({"noise_scale": noise_scale_leg(torch, sp, WL, args.workload, args.power_iters)}),
              flush=True)
        return
    path, ms, per_proj_us, mask_us = run_mode(torch, sp, WL, args.workload, prec, args, args.steps, args.warmup)
    head, roofline = leg_summary(sp, path, ms, per_proj_us, mask_us, prec, args.workload)
    pname = {v: k for k, v in sp.PRECS.items()}[prec]
    correction_ms = path.correction_ms
    projs, M, w_dtype = path.projs, path.M, path.w_dtype
    del path
    torch.cuda.empty_cache()
    modes = {}
    if not args.no_modes and args.workload != "single-fp32-m32":
        for mname in ("bf16x3", "bf16", "f32"):
            if sp.PRECS[mname] == prec:
                continue
            mpath, m_ms, m_pp, _ = run_mode(torch, sp, WL, args.workload, sp.PRECS[mname], args,
                                            max(5, args.steps // 2), 2)
            modes[mname] = {"ms_per_step": round(m_ms, 4),
                            "tflops": round(mpath.flops() / (m_ms * 1e-3) / 1e12, 2),
                            "gemm_us": {p.name: round(u, 2) for p, u in zip(mpath.projs, m_pp)}}
            del mpath
            torch.cuda.empty_cache()
    legs = {}
    if not args.no_legs and args.workload == DEFAULT_WORKLOAD:
        for name in LEGS:
            lpath, l_ms, l_pp, l_mask = run_mode(torch, sp, WL, name, prec, args, args.steps, args.warmup)
            lhead, lroof = leg_summary(sp, lpath, l_ms, l_pp, l_mask, prec, name)
            lhead["roofline"] = lroof
            legs[name] = lhead
            del lpath
            torch.cuda.empty_cache()
            print("leg %s: %.3f TFLOP/s, %.4f ms per step" % (name, lhead["value"], lhead["ms_per_step"]),
                  file=sys.stderr, flush=True)
    out = {
        "metric": METRIC, "value": head["value"], "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": pname,
        "data": "synthetic (seeded random activations and random-init weights)",
        "config": dict({"workload": args.workload}, **{k: v for k, v in head.items()
                                                       if k not in ("value", "ms_per_step")},
                       mechanism=args.mech, delta=args.delta, eps=args.eps, precision=pname,
                       launch="eager" if args.no_graph else "hip-graph (the timed steps captured as one graph)"),
        "roofline": roofline,
        "correction_ms": round(correction_ms, 4),
        "modes": modes,
        "legs": legs,
    }
    if not args.no_down_f64:
        out["down_f64"] = down_f64_leg(torch, sp, WL, args.workload)
    if not args.no_noise_bank:
        out["noise_bank"] = noise_bank_leg(torch, sp, WL, args.workload)
    if not args.no_noise_scale:
        out["noise_scale"] = noise_scale_leg(torch, sp, WL, args.workload, args.power_iters)
    if not args.no_cpu_baseline:
        deltas = out["noise_scale"]["delta"] if "noise_scale" in out else None
        out["cpu_baseline"], out["fp_error"] = cpu_baseline_leg(torch, sp, WL, args.cpu_seconds, projs, M,
                                                                w_dtype, args.workload, deltas)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
