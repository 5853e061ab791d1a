#!/usr/bin/env python3
"""Throughput of the DP-masked linear path on one MI355X.

Default workload: one step = the whole hot path for one Llama-3.2-3B-shaped
layer at a 128-token prefill: for each projection group (QKV 3072->5120,
O 3072->3072, gate/up 3072->16384, down 8192->3072) noise + mask (one kernel)
and the GEMM with the fused unmask epilogue (one kernel).  Weights are bf16
~ N(0, 0.02^2), activations float32 ~ N(0, 1), Gaussian mechanism (Prop. 2)
with Delta = 1, eps = 1; the corrections eta W^T are precomputed outside the
timed region (the paper's offline step) and reported separately.  Steps cycle
through 8 distinct weight sets so the 201 MB per layer is streamed from HBM,
not the 256 MB MALL.  --workload selects the other shapes: the single float32
projection, the 28-layer Llama stack at 512 tokens, the 36-layer Qwen3-4B stack
at 1024 tokens, and Qwen3-4B decode steps (M tokens at position 1024 of a
2048-position correction bank).  At decode sizes (M <= 16, bfloat16 modes) a
layer's masks are drawn by one launch and each projection is one launch that
forms fl32(X + eta), multiplies and unmasks.  The timed steps are captured, in
order, as one HIP graph and replayed once (after an untimed replay), so the host
launches once for all of them.

Prints one JSON line.  Fields beyond the common contract: ``roofline`` (the
GEMM + unmask kernel: each projection group's launches for every layer or
weight set back to back in one HIP graph, bracketed by HIP events on the stream
they run on; ``traffic`` from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
summary of the workload when the kernel sources still match it, else null),
``cpu_baseline`` (the CPU oracle on a bounded sample of the same workload),
``modes`` (other precision modes), ``correction_ms`` (offline precompute),
``down_f64`` (the Down projection at Theorem 3's noise scale through the binary64
path against the bf16x3 one: time and error), ``noise_bank`` (one layer's correction
banks for 2048 positions: created from the
GPU corrections into files, then loaded as decode steps and as one batch),
``noise_scale`` (the offline noise-scale step of the same model: spectral norms
of W_val, W_up and W_gate by the power method, the sensitivity bounds of
Theorems 1-3 from them, and the time of one power-method round against the
HBM roofline of reading W once).
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
    ap.add_argument("--workload", default="llama3b-layer-m128", choices=WORKLOADS)
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
    ap.add_argument("--no-modes", action="store_true", help="skip the other precision modes")
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


WORKLOADS = ["llama3b-layer-m128", "single-fp32-m32", "llama3b-28l-m512", "qwen3-4b-36l-m1024",
             "qwen3-4b-decode-m1", "qwen3-4b-decode-m4", "qwen3-4b-decode-m16", "qwen3-4b-decode-m64",
             "llama3b-lmhead-m1", "llama3b-lmhead-m15", "llama3b-lmhead-m128",
             "qwen3-4b-lmhead-m1", "qwen3-4b-lmhead-m15"]
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
    the unmask epilogue.  Decode-sized M (the skinny kernel): per layer, one launch
    draws the masks of all projection groups, then one launch per projection forms
    fl32(X + eta), multiplies and unmasks."""

    def __init__(self, torch, sp, WL, name, prec, mech, delta, eps, weight_sets, layout="auto"):
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
        self.tiled = [can_tile and weight_tiled(layout, M, p.N) for p in self.projs]
        self.wt = [sp.SPLITEE_BF16_TILED if t else wt for t in self.tiled]
        self.layout = "tiled" if all(self.tiled) else ("row-major" if not any(self.tiled) else "mixed")
        self.X, self.Xt, self.Y, self.ws = [], [], [], []
        for p in self.projs:
            self.X.append(torch.randn((M, p.K), generator=g, device=dev, dtype=torch.float32))
            planes = 3 if prec == sp.SPLITEE_PREC_BF16X3 else 1
            dt = torch.float32 if prec == sp.SPLITEE_PREC_F32 else torch.int16
            self.Xt.append(torch.empty((planes, M, p.K), dtype=dt, device=dev))
            self.Y.append(torch.empty((M, p.N), dtype=torch.float32, device=dev))
        self.decode = M <= 16 and prec != sp.SPLITEE_PREC_F32
        for p in self.projs:
            self.ws.append(sp.workspace(M, p.N, p.K, prec, dev, gemm_only=not self.decode))
        # decode: the masks of every layer of a step, [layer][token][k] per projection group
        self.eta = [torch.empty((self.layers_per_step, M, p.K), dtype=torch.float32, device=dev)
                    for p in self.projs] if self.decode else None
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
        (decode: mask + GEMM + unmask, on the mask drawn for the layer)."""
        p, M = self.projs[i], self.M
        W, C = self.W[l][i], self.C[l][i]
        if self.decode:
            self.sp.splitee_masked_linear_fused(
                self.X[i], p.K, W, self.wt[i], p.K, C, C.stride(0), self.Y[i], p.N, M, p.N, p.K, self.mech,
                self.delta, self.eps, 0, self.sid[l][i], self.row0, self.eta[i][l % self.layers_per_step], self.prec,
                self.ws[i][0], self.ws[i][1])
        else:
            self.sp.splitee_masked_linear_unmask(self.Xt[i], self.prec, p.K, W, self.wt[i], p.K, C,
                                                 C.stride(0), self.Y[i], p.N, M, p.N, p.K,
                                                 self.ws[i][0], self.ws[i][1])

    def draw_masks(self, base):
        """Decode: one launch draws the masks of all layers and projection groups of a step."""
        Ks = [p.K for p in self.projs]
        self.sp.splitee_noise_gen_multi(self.eta, Ks, Ks, self.sid[base], self.M, self.mech, self.delta,
                                        self.eps, 0, self.row0, reps=self.layers_per_step,
                                        rep_strides=[self.M * K for K in Ks], rep_sid_step=self.sid_step)

    def launches(self, s):
        """All kernels of step s: noise, mask, GEMM and unmask of every projection."""
        sp, M = self.sp, self.M
        base = (s % self.nsets) * self.layers_per_step
        if self.decode:
            self.draw_masks(base)
        for l in range(base, base + self.layers_per_step):
            if self.decode:
                for i in range(len(self.projs)):
                    self.gemm(l, i)
                continue
            for i, p in enumerate(self.projs):
                sp.splitee_noise_mask(self.X[i], p.K, self.Xt[i], self.prec, p.K, M, p.K, self.mech,
                                      self.delta, self.eps, 0, self.sid[l][i], self.row0)
                self.gemm(l, i)

    def flops(self):
        return self.layers_per_step * sum(2.0 * self.M * p.N * p.K for p in self.projs)

    def gemm_bytes(self):
        """Algorithmic bytes of each GEMM + unmask launch: W, float32 X (and, in the
        decode launch that forms the masked input, float32 eta), C and Y."""
        wb = 4.0 if self.w_dtype == "f32" else 2.0
        xb = 8.0 if self.decode else 4.0
        return [wb * p.N * p.K + xb * self.M * p.K + 8.0 * self.M * p.N for p in self.projs]


def run_mode(torch, sp, WL, name, prec, args, steps, warmup):
    path = Path(torch, sp, WL, name, prec, sp.MECHS[args.mech], args.delta, args.eps,
                args.weight_sets, args.layout)
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

    # per-launch duration of the GEMM + unmask kernel of each projection group: its
    # launches for every layer / weight set of the run, back to back in one HIP
    # graph (eager launches when --no-graph), bracketed by HIP events recorded on
    # the stream the kernels run on; averaged over launches and repeats
    nproj = len(path.projs)
    per_proj_us = [0.0] * nproj
    reps = max(2, min(steps, 20))
    for i in range(nproj):
        def gemms(i=i):
            for s in range(path.nsets):
                base = s * path.layers_per_step
                for l in range(base, base + path.layers_per_step):
                    path.gemm(l, i)
        n_launch = path.nsets * path.layers_per_step
        if graphs is not None:
            gemms()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                gemms()
            go = g.replay
        else:
            go = gemms
        go()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            go()
        e1.record()
        torch.cuda.synchronize()
        per_proj_us[i] = e0.elapsed_time(e1) * 1e3 / (reps * n_launch)
    return path, ms, per_proj_us


def cpu_baseline(WL, target_s, projs, tokens, w_dtype):
    """The oracle (binary128 noise, mask, binary64 GEMM, correction GEMM, unmask) on
    a row sample of one layer of the same workload; throughput in TFLOP/s of the
    sample's algorithmic work (2 x rows x N x K per projection group)."""
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
    return {"value": flops / total / 1e12, "unit": "TFLOP/s",
            "cores": int(max(O.num_threads(), blas_threads)), "kind": "oracle",
            "sample": "%d x %d of %d tokens of one layer's %d projection group(s): noise, mask, GEMM, "
                      "correction GEMM, unmask; %.1f s" % (reps, rows, tokens, len(projs), total)}


GEMM_SOURCES = ["paper_2609_15039_amd/csrc/gemm.hip", "paper_2609_15039_amd/csrc/common.hpp"]


def gemm_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def weight_tiled(layout, M, N):
    """Whether a bfloat16 projection of N output rows at M tokens stores W tiled.  auto:
    one or two tokens run the vector-ALU GEMV, which reads whole rows of row-major W faster
    for the narrower projections and 32-row blocks of tiled W faster from 16384 rows up
    (gate/up, the LM heads); every other M runs the MFMA kernels on tiled W."""
    if layout == "auto":
        return not (M <= 2 and N < 16384)
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
    path = Path(torch, sp, WL, args.workload, prec, sp.MECHS[args.mech], args.delta, args.eps, 1, args.layout)
    if path.decode:
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
    path, ms, per_proj_us = run_mode(torch, sp, WL, args.workload, prec, args, args.steps, args.warmup)
    flops = path.flops()
    value = flops / (ms * 1e-3) / 1e12
    gb = path.gemm_bytes()
    gemm_us = sum(per_proj_us)
    gflops = [2.0 * path.M * p.N * p.K for p in path.projs]
    ai = sum(gflops) / sum(gb)
    if ai < 315.0 or path.w_dtype == "f32" and ai < 19.7:
        achieved = sum(gb) / (gemm_us * 1e-6) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        peak = FP32_PEAK_TFS if prec == sp.SPLITEE_PREC_F32 else BF16_PEAK_TFS
        achieved = sum(gflops) / (gemm_us * 1e-6) / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(achieved / peak, 4)}
    pname = {v: k for k, v in sp.PRECS.items()}[prec]
    names = [p.name for p in path.projs]
    layout = path.layout
    traffic = measured_traffic(args.workload, pname, layout, names)
    # bf16x3 issues three MFMA passes per algorithmic flop (the exact split of the masked input)
    planes = 3 if prec == sp.SPLITEE_PREC_BF16X3 else 1
    if prec != sp.SPLITEE_PREC_F32 and not path.decode:
        issued = planes * sum(gflops) / (gemm_us * 1e-6) / 1e12
        roofline.update({"mfma_issued_tflops": round(issued, 1),
                         "mfma_issued_frac": round(issued / BF16_PEAK_TFS, 4), "mfma_passes": planes})
    roofline.update({"traffic": None if traffic is None else int(sum(traffic.values())),
                     "traffic_per_launch": traffic and {k: int(v) for k, v in traffic.items()},
                     "kernel": ("mask + GEMM + unmask (one launch per projection group, on the masks "
                                "one launch per layer draws)") if path.decode
                               else "GEMM + unmask (one launch per projection group)",
                     "launch_us": {p.name: round(u, 2) for p, u in zip(path.projs, per_proj_us)},
                     "bytes_per_launch": {p.name: int(b) for p, b in zip(path.projs, gb)},
                     "flops_per_launch": {p.name: int(f) for p, f in zip(path.projs, gflops)},
                     "algorithmic_ai": round(ai, 1)})
    modes = {}
    if not args.no_modes and args.workload != "single-fp32-m32":
        for mname in ("bf16x3", "bf16", "f32"):
            if sp.PRECS[mname] == prec:
                continue
            _, m_ms, m_pp = run_mode(torch, sp, WL, args.workload, sp.PRECS[mname], args,
                                     max(10, args.steps // 2), 3)
            modes[mname] = {"ms_per_step": round(m_ms, 4),
                            "tflops": round(flops / (m_ms * 1e-3) / 1e12, 2),
                            "gemm_us": {p.name: round(u, 2) for p, u in zip(path.projs, m_pp)}}
    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": pname,
        "data": "synthetic (seeded random activations and random-init weights)",
        "config": {"workload": args.workload, "tokens": path.M, "layers_per_step": path.layers_per_step,
                   "projections": {p.name: [p.K, p.N] for p in path.projs},
                   "mechanism": args.mech, "delta": args.delta, "eps": args.eps,
                   "precision": pname, "w_layout": layout,
                   "w_tiled": [p.name for p, t in zip(path.projs, path.tiled) if t],
                   "weight_sets": path.nsets, "row0": path.row0,
                   "launch": "eager" if args.no_graph else "hip-graph (the timed steps captured as one graph)"},
        "roofline": roofline,
        "correction_ms": round(path.correction_ms, 4),
        "modes": modes,
    }
    if not args.no_down_f64:
        out["down_f64"] = down_f64_leg(torch, sp, WL, args.workload)
    if not args.no_noise_bank:
        out["noise_bank"] = noise_bank_leg(torch, sp, WL, args.workload)
    if not args.no_noise_scale:
        out["noise_scale"] = noise_scale_leg(torch, sp, WL, args.workload, args.power_iters)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(WL, args.cpu_seconds, path.projs, path.M, path.w_dtype)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
