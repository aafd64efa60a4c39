"""Benchmark of the lattice hot path on one MI355X.

One step = one pass of the whole path over one synthetic cloud: splat (build
the lattice and splat the point features), build the 1-ring neighbour table,
every lattice convolution the workload lists (chained: each one's output
feeds the next), and slice the last output back onto the points.  The inputs
(positions, features, batch ids, weights already rounded to bf16 where the
conv is bf16) are resident in HBM before the timed region; every step
rebuilds the lattice from scratch.

The default workload is the largest one: four LiDAR sweeps of a scene with
moving boxes, 421 398 points in a d = 4 space-time lattice, one 64 -> 64 bf16
conv with 11 taps.

Prints one JSON line.  `value` is points per second of whole steps; the
`roofline` object reports the step's slowest single-kernel stage (the
neighbour search, a conv or the slice) against its own roofline, timed with
HIP events recorded on the stream the kernels run on; `stages` gives every
stage, the multi-kernel splat included (mean, and p10 / median / p90 over the
steps); `stages_cold` repeats that with the caches evicted before every step;
`hbm_frac_splat_slice` is the splat and slice bytes over their time against
peak HBM; `cpu_baseline` is the CPU oracle timed on this host on a bounded
sample with all its BLAS threads, `cpu_baseline_1core` with one.
`other_configs` repeats the plain step on the indoor room and the LiDAR scan
(stages and rooflines), and `targets` sets the two performance goals against
what was measured: splat + slice at 50% of peak HBM (on every workload timed),
and the bf16 conv at C = 128 (the LiDAR scan's 128 -> 128) at 40% of peak bf16
MFMA.  `roofline.traffic_source` says where the HBM traffic figure comes from.

With --op deform the step ends in DeformSlice fused with the linear
classifier (per-point logits, the network's output layer) instead of the
plain slice, and the `roofline` object covers that kernel.

With --op train the step is the forward pass followed by its backward pass
from a fixed point gradient dL/df: the slice's gradient (a splat of dL/df),
each conv's input gradient and weight gradient in reverse order (two stages
each), and the splat's gradient with respect to the point features.

With --op unet the step also builds the coarse lattice (the same points at
twice the scale), downsamples the last conv's output onto it (a strided
conv), upsamples it back onto the fine vertices (a transposed conv) and
slices that: one level of the paper's U-Net.

With --op pointnet the network's input layer replaces the splat of the
features: the step builds the lattice, then Distribute + PointNet + per-vertex
max (fused) turns the raw point features into the 64-channel vertex values
the convs take (workloads whose first conv has 64 inputs); each PointNet block
starts with a group normalisation whose statistics are computed per cloud.

With --backward (after --op deform, unet or pointnet) the step adds the
backward pass of every stage from a fixed gradient at its output: DeformSlice
with the classifier (dL/d logits), or the slice, then the upsample's and the
downsample's, every conv's input and weight gradients, and last the splat's
(dL/d features) or Distribute + PointNet's (every block's parameters).

Usage: python bench.py [--steps K] [--warmup W] [--config N] [--op slice|deform|train|unet|pointnet]
       [--backward] [--no-cpu-baseline] [--no-other-configs] [--no-cold]
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

import numpy as np  # noqa: E402

DEFAULT_CONFIG = 5          # the largest workload: four LiDAR sweeps in a d = 4 space-time lattice
# Workloads whose stages are also timed in the default run (`other_configs`):
# the indoor room (the largest d = 3 cloud) and the LiDAR scan (128 -> 128
# bf16 conv, where the MFMA target is set).
EXTRA_CONFIGS = (3, 4)
TARGET_HBM_FRAC = 0.5       # splat + slice, algorithmic bytes over their time, of peak HBM
TARGET_MFMA_FRAC = 0.4      # the bf16 lattice conv at C = 128 (LiDAR scan, 128 -> 128), of peak bf16 MFMA
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
# fp32 vector units: 256 CUs x 4 SIMDs x 2.4 GHz x 64 lanes x 2 flops (FMA) at
# the published rate; without packed fp32 instructions one wave64 FMA issues
# every second cycle, so 78.6 TFLOP/s is the reachable ceiling here.
ALU_PEAK_TFLOPS = 157.3

WORKLOAD_NAMES = {
    1: "tiny-spheres-4096pts-d3",
    2: "partseg-16x2500pts-d3-sigma0.04-C64-conv64x64-f32+bf16",
    3: "indoor-room-200kpts-d3-sigma0.04-C64-conv64x64+64x128-bf16",
    4: "lidar-scan-64beam-d3-sigma0.3-C128-conv128x128-bf16",
    5: "spatiotemporal-4scans-d4-sigma0.3-C64-conv64x64-bf16",
}


class Pipeline:
    """Device-resident inputs and buffers of one workload, and one step over them.

    Everything runs on one side stream (default priority): a caller that reads
    the outputs on another stream synchronises with `stream` first.  Every
    buffer is allocated up front and the step never synchronises with the host
    (V stays on the device), so the step can be captured once as a HIP graph
    and replayed."""

    def __init__(self, w, stream=None, tail="slice", backward=False):
        import torch

        from paper_2108_03917_amd import Lattice

        self.w = w
        self.tail = tail
        # --op train is the slice step with its backward pass; --backward adds
        # the backward pass to the deform, unet and pointnet steps
        self.backward = backward or tail == "train"
        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        self.stream = stream if stream is not None else torch.cuda.Stream(device=dev)
        self.graph = None
        self.L = Lattice(w.d, w.sigma, max_points=w.m, stream=self.stream)
        self.pos = torch.from_numpy(w.pos).to(dev)
        self.feat = torch.from_numpy(w.feat).to(dev)
        self.batch = None if w.batch is None else torch.from_numpy(w.batch).to(dev)
        mv = self.L.max_vertices(w.m)
        self.convs = list(w.convs)
        # A stage stores its vertex rows as bf16 exactly when the next stage is
        # a bf16 conv (which would round them to bf16 on load anyway); the
        # rows the slice reads stay fp32.
        def storage(i):
            return torch.bfloat16 if i < len(self.convs) and self.convs[i].dtype == "bf16" else torch.float32
        self.values = torch.empty((mv, w.C), dtype=storage(0), device=dev)
        self.weights, self.outs = [], []
        for i, cv in enumerate(self.convs):
            wd = torch.from_numpy(cv.weight).to(dev)
            if cv.dtype == "bf16":
                wd = self.L.weights_to_bf16(wd)   # parameters: rounded once, outside the step
            self.weights.append(wd)
            self.outs.append(torch.empty((mv, cv.c_out), dtype=storage(i + 1), device=dev))
        c_last = self.convs[-1].c_out if self.convs else w.C
        if tail == "deform":
            from datagen.clouds import N_CLASSES, deform_weights

            self.dw = deform_weights(c_last, N_CLASSES.get(w.config, 20), seed=100 + w.config)
            self.w_delta = torch.from_numpy(self.dw.w_delta).to(dev)
            self.w_cls = torch.from_numpy(self.dw.w_cls).to(dev)
            self.b_cls = torch.from_numpy(self.dw.b_cls).to(dev)
            self.sliced = torch.empty((w.m, self.w_cls.shape[0]), dtype=torch.float32, device=dev)
        else:
            self.sliced = torch.empty((w.m, c_last), dtype=torch.float32, device=dev)
        if tail == "pointnet":
            from datagen.clouds import pointnet_gn_weights, raw_point_features

            if not self.convs or self.convs[0].c_in != 64:
                raise SystemExit("--op pointnet needs a workload whose first conv takes the PointNet's 64 channels "
                                 "(workloads 2, 3, 5)")
            raw = raw_point_features(w)
            self.raw = torch.from_numpy(raw).to(dev)
            k0 = w.d + raw.shape[1]
            # group normalisation before each block, min(32, K) groups, per cloud
            self.pn_layers = pointnet_gn_weights(k0, seed=800 + w.config)
            self.pn_groups = [min(32, k) for k in (k0, 16, 32)]
            self.pn_params = Lattice.pack_pointnet(self.pn_layers).to(dev)
            self.values = torch.empty((mv, 64), dtype=storage(0), device=dev)
        if tail == "unet":
            from datagen.clouds import conv_weight

            sig = np.asarray(w.sigma, dtype=np.float32)
            self.Lc = Lattice(w.d, 2 * sig, max_points=w.m, stream=self.stream)
            mvc = self.Lc.max_vertices(w.m)
            last = self.convs[-1]
            st = torch.bfloat16 if last.dtype == "bf16" else torch.float32
            self.rs_dtype = last.dtype
            wd = torch.from_numpy(conv_weight(c_last, c_last, w.d, seed=600 + w.config)).to(dev)
            wu = torch.from_numpy(conv_weight(c_last, c_last, w.d, seed=700 + w.config)).to(dev)
            if last.dtype == "bf16":
                wd, wu = self.L.weights_to_bf16(wd), self.L.weights_to_bf16(wu)
            self.w_down, self.w_up = wd, wu
            # the coarse rows feed a conv of the conv's dtype; the fine rows feed the slice
            self.coarse_vals = torch.empty((mvc, c_last), dtype=st, device=dev)
            self.up_vals = torch.empty((mv, c_last), dtype=torch.float32, device=dev)
            # the last forward conv's output feeds the downsample: store it as its input dtype
            self.outs[-1] = torch.empty((mv, c_last), dtype=st, device=dev)
        if self.backward:
            from datagen.clouds import random_rows

            # the loss gradient at the points (dL/d logits after DeformSlice
            # with the classifier, else dL/df): an input of the step
            n_out = self.w_cls.shape[0] if tail == "deform" else c_last
            self.gout = torch.from_numpy(random_rows(w.m, n_out, seed=500 + w.config)).to(dev)
            # a gradient row is stored as bf16 where the conv that reads it
            # computes in bf16 (it would round it on load anyway)
            def gstore(i):
                return torch.bfloat16 if i >= 0 and self.convs[i].dtype == "bf16" else torch.float32
            n = len(self.convs)
            # dL/dy of the last conv (the slice's gradient), then dL/dx of each conv
            self.gtop = torch.empty((mv, c_last), dtype=gstore(n - 1), device=dev)
            self.gin = [torch.empty((mv, cv.c_in), dtype=gstore(i - 1), device=dev) for i, cv in enumerate(self.convs)]
            self.gw = [torch.empty((cv.c_out, w.taps, cv.c_in), dtype=torch.float32, device=dev) for cv in self.convs]
            self.gfeat = torch.empty((w.m, w.C), dtype=torch.float32, device=dev)
            if tail == "unet":
                self.g_up = torch.empty((mv, c_last), dtype=torch.float32, device=dev)
            if tail == "pointnet":
                self.gparams = torch.empty_like(self.pn_params)
            assert n > 0
        torch.cuda.synchronize()

    @property
    def conv_spec(self):
        return self.convs[-1]

    def run(self, ev=None):
        """One step, enqueued on the pipeline's stream.  With `ev` (a list of
        torch events) an event is recorded on that stream before every stage
        and one after the last."""
        import torch

        with torch.cuda.stream(self.stream):
            return self._run(ev)

    def capture(self):
        """Capture one step as a graph (after at least one eager step, which
        sets up every kernel's launch attributes)."""
        import torch

        self.stream.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=self.stream):
            self._run(None)
        self.stream.synchronize()
        self.graph = g
        return g

    def replay(self):
        import torch

        with torch.cuda.stream(self.stream):
            self.graph.replay()
        return self.sliced

    def _run(self, ev):
        L = self.L
        k = 0

        def mark():
            nonlocal k
            if ev is not None:
                ev[k].record(self.stream)
                k += 1

        mark()
        if self.tail == "pointnet":
            L.splat(self.pos, None, self.batch, want_weight=False)
            mark()
            L.distribute_pointnet(self.pos, self.raw, self.pn_params, out=self.values, groups=self.pn_groups)
        else:
            L.splat(self.pos, self.feat, self.batch, values=self.values, want_weight=False)
        if self.tail == "unet":
            mark()
            self.Lc.splat(self.pos, None, self.batch, want_weight=False)
        mark()
        L.build_neighbors()
        x = self.values
        for cv, wd, out in zip(self.convs, self.weights, self.outs):
            mark()
            L.conv(x, wd, dtype=cv.dtype, out=out)
            x = out
        if self.tail == "unet":
            mark()
            L.downsample(self.Lc, x, self.w_down, dtype=self.rs_dtype, out=self.coarse_vals)
            mark()
            self.Lc.upsample(L, self.coarse_vals, self.w_up, dtype=self.rs_dtype, out=self.up_vals)
            x = self.up_vals
        mark()
        if self.tail == "deform":
            L.deform_slice(x, self.w_delta, self.dw.b_delta, self.w_cls, self.b_cls, out=self.sliced)
        else:
            L.slice(x, out=self.sliced)
        if self.backward:
            n = len(self.convs)
            gdt = "bf16" if self.convs[-1].dtype == "bf16" else "f32"
            mark()
            if self.tail == "deform":
                gy = L.deform_slice_backward(x, self.w_delta, self.dw.b_delta, self.gout, w_cls=self.w_cls,
                                             grad_dtype=gdt)[0]
            elif self.tail == "unet":
                L.slice_backward(self.gout, out=self.g_up)
                mark()
                g_coarse = self.Lc.upsample_backward(L, self.g_up, self.w_up, x=self.coarse_vals,
                                                     dtype=self.rs_dtype, grad_in_dtype=self.rs_dtype)[0]
                mark()
                gy = L.downsample_backward(self.Lc, g_coarse, self.w_down, x=self.outs[-1], dtype=self.rs_dtype,
                                           grad_in_dtype=gdt)[0]
            else:
                L.slice_backward(self.gout, out=self.gtop)
                gy = self.gtop
            for i in reversed(range(n)):
                cv = self.convs[i]
                xin = self.values if i == 0 else self.outs[i - 1]
                g = gy if i == n - 1 else self.gin[i + 1]
                mark()
                L.conv_backward(g, self.weights[i], dtype=cv.dtype, want_weight=False, grad_in=self.gin[i])
                mark()
                L.conv_backward(g, self.weights[i], xin, dtype=cv.dtype, want_input=False, grad_w=self.gw[i])
            mark()
            if self.tail == "pointnet":
                L.distribute_pointnet_backward(self.pos, self.raw, self.pn_params, self.gin[0], groups=self.pn_groups,
                                               grad_params=self.gparams)
            else:
                L.splat_backward(self.gin[0], out=self.gfeat)
        mark()
        return self.sliced

    def stage_names(self):
        fwd = ["splat", "neighbors"] + [f"conv{i}_{c.c_in}x{c.c_out}_{c.dtype}" for i, c in enumerate(self.convs)]
        if self.tail == "unet":
            names = ["splat", "coarse_lattice"] + fwd[1:] + ["downsample", "upsample", "slice"]
        elif self.tail == "pointnet":
            names = ["lattice", "distribute"] + fwd[1:] + ["slice"]
        elif self.tail == "deform":
            names = fwd + ["deform"]
        else:
            names = fwd + ["slice"]
        if not self.backward:
            return names
        bwd = {"deform": ["deform_bwd"], "unet": ["slice_bwd", "upsample_bwd", "downsample_bwd"]}.get(self.tail,
                                                                                                     ["slice_bwd"])
        for i in reversed(range(len(self.convs))):
            c = self.convs[i]
            bwd += [f"conv{i}_{c.c_in}x{c.c_out}_{c.dtype}_bwd_in", f"conv{i}_{c.c_in}x{c.c_out}_{c.dtype}_bwd_w"]
        return names + bwd + ["distribute_bwd" if self.tail == "pointnet" else "splat_bwd"]


def algorithmic_work(w, V, n_cls=0, Vc=0, f_raw=-1):
    """Compulsory HBM bytes (and MFMA flops) of each stage of one step.

    splat:     read positions (4d B), batch id (4 B), features (4C B) and write
               the simplex record (vertex index + weight, 8(d+1) B) per point;
               write the value row (2C or 4C B) and packed key (8 B) per vertex.
    neighbors: read the key (8 B), write T indices (4T B) per vertex.
    conv:      read the input row (s C_in), neighbour row (4T), write the output
               row (s' C_out) per vertex, plus the weights once; 2 T C_in C_out
               flops per vertex (s, s' = 2 for bf16-stored rows, else 4).
    slice:     read the record (8(d+1)) and write the output row (4C) per point,
               read each vertex row once (4C per vertex).
    deform:    DeformSlice + classifier: read the record (8(d+1)) and write
               the logits (4 n_cls) per point, read each vertex row once (4C
               per vertex), plus the weights (4(C + n_cls C + n_cls)) once."""
    d, m, C = w.d, w.m, w.C
    T = 2 * (d + 1) + 1
    work = {}
    s0 = 2 if w.convs and w.convs[0].dtype == "bf16" else 4
    work["splat"] = {"bytes": m * (4 * d + 4 * C + 8 * (d + 1) + (4 if w.batch is not None else 0))
                     + V * (s0 * C + 8)}
    work["neighbors"] = {"bytes": V * (8 + 4 * T)}
    for i, cv in enumerate(w.convs):
        s = 2 if cv.dtype == "bf16" else 4
        s_out = 2 if i + 1 < len(w.convs) and w.convs[i + 1].dtype == "bf16" else 4
        work[f"conv{i}_{cv.c_in}x{cv.c_out}_{cv.dtype}"] = {
            "bytes": V * (s * cv.c_in + 4 * T + s_out * cv.c_out) + T * cv.c_in * cv.c_out * s,
            "flops": 2 * V * T * cv.c_in * cv.c_out, "dtype": cv.dtype}
    c_last = w.convs[-1].c_out if w.convs else C
    work["slice"] = {"bytes": m * (8 * (d + 1) + 4 * c_last) + V * 4 * c_last}
    work["deform"] = {"bytes": m * (8 * (d + 1) + 4 * n_cls) + V * 4 * c_last + 4 * (c_last + n_cls * c_last + n_cls)}
    # backward (--op train): a gradient row is bf16 where a bf16 conv reads it
    def sg(i):
        return 2 if i >= 0 and w.convs[i].dtype == "bf16" else 4
    n = len(w.convs)
    if n:
        # slice backward: read dL/df (4 c_last) and the pair (8 B) per point-vertex pair, write the row
        work["slice_bwd"] = {"bytes": m * (4 * c_last + 8 * (d + 1)) + V * sg(n - 1) * c_last}
        for i, cv in enumerate(w.convs):
            name = f"conv{i}_{cv.c_in}x{cv.c_out}_{cv.dtype}"
            s_x = 2 if cv.dtype == "bf16" else 4
            # input gradient: a forward conv C_out -> C_in with flipped weights
            work[name + "_bwd_in"] = {
                "bytes": V * (sg(i) * cv.c_out + 4 * T + sg(i - 1) * cv.c_in) + T * cv.c_in * cv.c_out * s_x,
                "flops": 2 * V * T * cv.c_in * cv.c_out, "dtype": cv.dtype}
            # weight gradient: read g, x and the neighbour row per vertex, write
            # the fp32 weights; on the MFMA of the conv's dtype
            work[name + "_bwd_w"] = {
                "bytes": V * (sg(i) * cv.c_out + s_x * cv.c_in + 4 * T) + T * cv.c_in * cv.c_out * 4,
                "flops": 2 * V * T * cv.c_in * cv.c_out, "dtype": cv.dtype}
        # splat backward: the slice of the vertex gradient onto the points
        work["splat_bwd"] = {"bytes": m * (8 * (d + 1) + 4 * C) + V * sg(-1) * C}
    if f_raw >= 0:
        E = m * (d + 1)
        k0 = d + f_raw
        # lattice only: read the positions (and batch id), write the record per
        # point and the key per vertex
        work["lattice"] = {"bytes": m * (4 * d + 8 * (d + 1) + (4 if w.batch is not None else 0)) + V * 8}
        # distribute + PointNet: read each point's position and raw features,
        # each pair-list entry (8 B) and each vertex's list header (8 B), write
        # the 64-channel row (bf16 when the first conv is bf16); 2 (k0 16 +
        # 16 32 + 32 64) flops per pair on fp32 MFMA (the group
        # normalisation's statistics passes recompute blocks 1 and 2: not
        # counted)
        work["distribute"] = {"bytes": m * 4 * (d + f_raw) + E * 8 + V * (8 + s0 * 64),
                              "flops": 2 * E * (k0 * 16 + 16 * 32 + 32 * 64), "dtype": "f32"}
        # its backward (every block's parameter gradients): the same reads plus
        # dL/dx (4 x 64 B per vertex); the forward's products once more and
        # the backward's two per layer (input and weight gradients), on the
        # fp32 vector units (the fp32 per-pair records it stores and rereads
        # are not counted)
        work["distribute_bwd"] = {"bytes": m * 4 * (d + f_raw) + E * 8 + V * (8 + 4 * 64),
                                  "flops": 3 * 2 * E * (k0 * 16 + 16 * 32 + 32 * 64), "dtype": "alu"}
    if n and Vc:
        last = w.convs[-1]
        s = 2 if last.dtype == "bf16" else 4
        # coarse lattice: read the positions (and batch id), write the simplex
        # record per point and the key per coarse vertex
        work["coarse_lattice"] = {"bytes": m * (4 * d + 8 * (d + 1) + (4 if w.batch is not None else 0)) + Vc * 8}
        # downsample: per coarse vertex its T indices and its output row, each
        # fine row read once, the weights once; 2 T C C flops per coarse vertex
        work["downsample"] = {"bytes": Vc * (4 * T + s * c_last) + V * s * c_last + T * c_last * c_last * s,
                              "flops": 2 * Vc * T * c_last * c_last, "dtype": last.dtype}
        # upsample: per fine vertex its T indices and its fp32 output row, each
        # coarse row read once; every tap is multiplied (absent ones as zeros)
        work["upsample"] = {"bytes": V * (4 * T + 4 * c_last) + Vc * s * c_last + T * c_last * c_last * s,
                            "flops": 2 * V * T * c_last * c_last, "dtype": last.dtype}
        # their backward passes (input and weight gradients in one call): the
        # output gradient, the forward input and the input gradient once per
        # row, the taps, the weights read and their gradient written (fp32);
        # the flops of the forward twice
        work["upsample_bwd"] = {"bytes": V * (4 * c_last + 4 * T) + Vc * 2 * s * c_last
                                + T * c_last * c_last * (s + 4),
                                "flops": 4 * V * T * c_last * c_last, "dtype": last.dtype}
        work["downsample_bwd"] = {"bytes": Vc * (s * c_last + 4 * T) + V * 2 * s * c_last
                                  + T * c_last * c_last * (s + 4),
                                  "flops": 4 * Vc * T * c_last * c_last, "dtype": last.dtype}
    if n and n_cls:
        # DeformSlice + classifier backward: per point the record and dL/d
        # logits, per vertex its row read and its gradient row written, the
        # weights read and their gradients written
        work["deform_bwd"] = {"bytes": m * (8 * (d + 1) + 4 * n_cls) + V * (sg(n - 1) + sg(n - 1)) * c_last
                              + 8 * (c_last + n_cls * c_last + n_cls)}
    return work


def roofline_entry(name, ms, wk):
    """achieved vs peak for one stage: MFMA-bound convs where their arithmetic
    intensity exceeds the ridge, vector-ALU-bound work (dtype "alu") against the
    fp32 vector peak, HBM otherwise."""
    if wk.get("dtype") == "alu":
        ridge = ALU_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
        if wk["flops"] / wk["bytes"] >= ridge:
            a = wk["flops"] / (ms * 1e-3) / 1e12
            return {"bound": "alu", "achieved": a, "peak": ALU_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": a / ALU_PEAK_TFLOPS}
    elif "flops" in wk:
        peak_t = MFMA_PEAK_TFLOPS[wk["dtype"]]
        ridge = peak_t * 1e12 / (HBM_PEAK_GBS * 1e9)
        if wk["flops"] / wk["bytes"] >= ridge:
            a = wk["flops"] / (ms * 1e-3) / 1e12
            return {"bound": "mfma", "achieved": a, "peak": peak_t, "unit": "TFLOP/s", "frac": a / peak_t}
    a = wk["bytes"] / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": a, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": a / HBM_PEAK_GBS}


def cpu_baseline(w, budget_s=20.0, dw=None, train=False, unet=False, pointnet=None):
    """The CPU oracle, as it stands, over the same workload: whole steps
    (lattice build, splat, neighbours, every conv, slice -- or DeformSlice
    with the classifier when `dw` holds its weights; with `unet` the coarse
    lattice, the downsample and the upsample before the slice; with
    `pointnet` (its layers and group counts) Distribute + PointNet instead of
    the features' splat; with `train` also the backward pass of every stage,
    down to the features or the PointNet's parameters) repeated until about
    `budget_s` seconds, reported as points/s."""
    from threadpoolctl import threadpool_info

    from oracle import lattice_oracle as O

    if train:
        from datagen.clouds import random_rows

        c_last = w.convs[-1].c_out if w.convs else w.C
        gout = random_rows(w.m, dw.w_cls.shape[0] if dw is not None else c_last, seed=500 + w.config)

    if pointnet is not None:
        from datagen.clouds import raw_point_features

        raw = raw_point_features(w)

    def one():
        lat = O.build(w.pos, w.sigma, batch=w.batch)
        if pointnet is not None:
            layers, groups = pointnet
            x, _, _ = O.distribute_pointnet(lat, w.pos, raw, layers, groups=groups)
        else:
            x, _, _ = O.splat(lat, w.feat)
        nbr = O.neighbors(lat)
        ins = []
        for cv in w.convs:
            ins.append(x)
            xi = x
            Wt = cv.weight
            if cv.dtype == "bf16":
                xi = O.round_bf16(x.astype(np.float32))
                Wt = O.round_bf16(Wt)
            x, _ = O.conv(xi, nbr, Wt)
        x_last = x
        if unet:
            from datagen.clouds import conv_weight

            c = x.shape[1]
            coarse = O.coarsen(w.pos, w.sigma, batch=w.batch)
            wd = conv_weight(c, c, w.d, seed=600 + w.config)
            wu = conv_weight(c, c, w.d, seed=700 + w.config)
            xc, _ = O.downsample(lat, coarse, x, wd)
            x, _ = O.upsample(coarse, lat, xc, wu)
        if dw is None:
            O.slice_(lat, x)
        else:
            O.deform_slice(lat.idx, lat.bary, x, dw.w_delta, dw.b_delta, dw.w_cls, dw.b_cls)
        if train:
            if dw is not None:
                g = O.deform_slice_backward(lat.idx, lat.bary, x, dw.w_delta, dw.b_delta, gout, lat.V, dw.w_cls,
                                            dw.b_cls)[0][0]
            else:
                g, _ = O.slice_backward(lat, gout)
            if unet:
                g = O.upsample_backward(coarse, lat, xc, wu, g)[0]
                g = O.downsample_backward(lat, coarse, x_last, wd, g)[0]
            for cv, xi in zip(reversed(w.convs), reversed(ins)):
                g, _, _, _, _, _ = O.conv_backward(xi, nbr, cv.weight, g)
            if pointnet is not None:
                O.distribute_pointnet_backward(lat, w.pos, raw, pointnet[0], g, groups=pointnet[1])
            else:
                O.splat_backward(lat, g)

    t0 = time.perf_counter()
    n = 0
    while True:
        one()
        n += 1
        if time.perf_counter() - t0 >= budget_s or n >= 50:
            break
    dt = time.perf_counter() - t0
    threads = 1
    for info in threadpool_info():
        threads = max(threads, int(info.get("num_threads", 1)))
    return {"value": n * w.m / dt, "unit": "points/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} whole step(s) of the {w.name} workload ({w.m} points), {dt:.1f} s"}


# Source files that define each stage's kernels; a stored traffic measurement
# is used only while their contents are unchanged.
STAGE_SOURCES = {
    "splat": ["splat.hip", "keys.h", "internal.h"],
    "neighbors": ["neighbors.hip", "keys.h", "internal.h"],
    "conv": ["conv.hip", "internal.h"],
    "slice": ["slice.hip", "internal.h"],
    "deform": ["deform.hip", "internal.h"],
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_hash(stage: str) -> str:
    import hashlib

    h = hashlib.sha1()
    kind = "conv" if stage.startswith("conv") else stage
    for f in STAGE_SOURCES[kind]:
        with open(os.path.join(ROOT, "paper_2108_03917_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str, stage: str):
    """HBM bytes per launch of a stage from committed rocprofv3 counter runs
    (FETCH_SIZE and WRITE_SIZE, each scaled by its copy-kernel calibration),
    with a note of where they come from; (None, reason) when there is no
    measurement or the kernel source has changed since it was taken."""
    rel = os.path.relpath(TRAFFIC_FILE, ROOT)
    if not os.path.exists(TRAFFIC_FILE):
        return None, f"no counter table ({rel})"
    with open(TRAFFIC_FILE) as fh:
        table = json.load(fh)
    key = f"{workload}/{stage}"
    e = table.get("entries", {}).get(key)
    if not e:
        return None, f"no counter run of this kernel in {rel}"
    if e.get("source_sha1") != source_hash(stage):
        return None, (f"{rel} entry {key} was measured on kernel source {e.get('source_sha1', '?')[:12]}, "
                      f"the current source is {source_hash(stage)[:12]}")
    cal = table["calibration"]
    bytes_ = (e["fetch_kib"] * cal["fetch_scale"] + e["write_kib"] * cal["write_scale"]) * 1024.0
    return bytes_, (f"{rel} entry {key}: a stored rocprofv3 --pmc run (FETCH_SIZE x {cal['fetch_scale']}, "
                    f"WRITE_SIZE x {cal['write_scale']}, per dispatch) of the same command on kernel source "
                    f"{e['source_sha1'][:12]}, not measured in this run")


def calibrate_copy(mib: int):
    """A plain device copy of `mib` MiB (three times), the reference kernel for
    scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch

    x = torch.ones(mib * 1024 * 1024 // 4, dtype=torch.float32, device="cuda:0")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_mib": mib}))


def time_pipeline(pipe, steps, warmup, cold=True, graph=False):
    """Warm up, then time `steps` whole steps (region 1), the same number
    again with HIP events around every stage (region 2) and, with `cold`, up
    to 50 steps with the caches evicted before each (region 3).  Returns the
    seconds of region 1, V, and the per-stage millisecond samples of regions 2
    and 3 (None without `cold`)."""
    import torch

    for _ in range(warmup):
        pipe.run()
    pipe.stream.synchronize()
    V = pipe.L.num_vertices()

    # Timed region 1: whole steps (eager, or graph replays with --graph).
    step = pipe.run
    if graph:
        pipe.capture()
        for _ in range(3):
            pipe.replay()
        step = pipe.replay
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0

    # Timed region 2: the same steps run eagerly with HIP events recorded on
    # the pipeline's stream around every stage (each conv and the slice are
    # one kernel launch), for the per-stage times and the roofline.
    names = pipe.stage_names()
    nev = len(names) + 1
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(steps)]
    torch.cuda.synchronize()
    for s_ in range(steps):
        pipe.run(evs[s_])
    torch.cuda.synchronize()
    samples = {n: [evs[s_][i].elapsed_time(evs[s_][i + 1]) for s_ in range(steps)] for i, n in enumerate(names)}

    # Timed region 3 (cold): before every step a 512 MiB buffer is written
    # (outside the events), which evicts the 256 MiB Infinity Cache and the
    # L2s, so each stage starts from HBM as the first touch of a new cloud would.
    cold_samples = None
    if cold:
        flush = torch.empty(512 * 1024 * 1024 // 4, dtype=torch.float32, device="cuda:0")
        n_cold = min(steps, 50)
        cev = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(n_cold)]
        torch.cuda.synchronize()
        for s_ in range(n_cold):
            with torch.cuda.stream(pipe.stream):
                flush.fill_(float(s_))
            pipe.run(cev[s_])
        torch.cuda.synchronize()
        cold_samples = {n: [cev[s_][i].elapsed_time(cev[s_][i + 1]) for s_ in range(n_cold)]
                        for i, n in enumerate(names)}
        del flush
    return sec, V, samples, cold_samples


def kernel_time(pipe, stage, steps):
    """Mean milliseconds of the one kernel of `stage` ("slice" or "deform")
    over `steps` eager steps, from the events its launch records at the
    kernel's start and end (library stage timing, on the pipeline's stream)."""
    import torch

    L = pipe.L
    torch.cuda.synchronize()
    L.set_timing(2)  # reset the sums
    L.set_timing(1)
    for _ in range(steps):
        pipe.run()
    torch.cuda.synchronize()
    ms, n = L.timing()[stage]
    L.set_timing(0)
    if n != steps:
        raise RuntimeError(f"kernel timing: {n} launches of {stage} recorded for {steps} steps")
    return ms / n


def pct(v):
    return {"p10": float(np.percentile(v, 10)), "median": float(np.median(v)), "p90": float(np.percentile(v, 90))}


def splat_slice_frac(work, stage_ms):
    """Splat + slice algorithmic bytes over their summed time, of peak HBM."""
    return ((work["splat"]["bytes"] + work["slice"]["bytes"]) / ((stage_ms["splat"] + stage_ms["slice"]) * 1e-3)
            / (HBM_PEAK_GBS * 1e9))


def other_config(config, steps, warmup):
    """The plain step (splat, neighbours, convs, slice) of another workload:
    whole-step rate and every stage against its roofline (HIP events, mean and
    percentiles over the steps; no cache eviction)."""
    from datagen.clouds import make_workload

    w = make_workload(config)
    pipe = Pipeline(w, tail="slice")
    sec, V, samples, _ = time_pipeline(pipe, steps, warmup, cold=False)
    work = algorithmic_work(w, V)
    stage_ms = {n: float(np.mean(v)) for n, v in samples.items()}
    res = {"workload": WORKLOAD_NAMES[config], "points": w.m, "d": w.d, "vertices": V,
           "value": w.m * steps / sec, "unit": "points/s", "ms_per_step": sec * 1e3 / steps,
           "stages": {n: dict(ms=stage_ms[n], ms_pct=pct(samples[n]), **roofline_entry(n, stage_ms[n], work[n]))
                      for n in samples},
           "hbm_frac_splat_slice": splat_slice_frac(work, stage_ms)}
    pipe.L.close()
    del pipe
    return res


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=DEFAULT_CONFIG)
    ap.add_argument("--op", choices=("slice", "deform", "train", "unet", "pointnet"), default="slice",
                    help="end the step with the plain slice, with DeformSlice + classifier, run the "
                         "forward and backward passes (train), add a coarse level (unet), or start with "
                         "Distribute + PointNet (pointnet)")
    ap.add_argument("--backward", action="store_true",
                    help="with --op deform, unet or pointnet: add the backward pass of every stage (--op train "
                         "is the slice step with its backward pass)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cache-flushed stage timings")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the indoor and LiDAR steps timed after the main workload (and the targets)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB")
    ap.add_argument("--graph", action="store_true", help="time graph replays of the step instead of eager steps")
    ap.add_argument("--conv-path", choices=("auto", "tiled", "ws", "rs"), default="auto",
                    help="force one conv kernel family (the library picks per shape by default)")
    args = ap.parse_args(argv)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested): the lattice path has no "
              "multi-GPU mode", file=sys.stderr)
        return 2

    import torch

    from datagen.clouds import make_workload

    w = make_workload(args.config)
    if args.backward and args.op not in ("deform", "unet", "pointnet"):
        raise SystemExit("--backward goes with --op deform, unet or pointnet (--op train is the slice step's)")
    pipe = Pipeline(w, tail=args.op, backward=args.backward)
    pipe.L.set_conv_path(args.conv_path)
    sec, V, samples, cold = time_pipeline(pipe, args.steps, args.warmup, not args.no_cold, args.graph)
    names = pipe.stage_names()
    stage_ms = {n: float(np.mean(v)) for n, v in samples.items()}

    n_cls = pipe.w_cls.shape[0] if args.op == "deform" else 0
    Vc = pipe.Lc.num_vertices() if args.op == "unet" else 0
    f_raw = pipe.raw.shape[1] if args.op == "pointnet" else -1
    work = algorithmic_work(w, V, n_cls, Vc, f_raw)
    stages = {n: dict(ms=stage_ms[n], ms_pct=pct(samples[n]), **roofline_entry(n, stage_ms[n], work[n]))
              for n in names}
    if cold is not None:
        stages_cold = {n: dict(ms_pct=pct(cold[n]), **roofline_entry(n, float(np.median(cold[n])), work[n]))
                       for n in names}
    # the roofline object covers one kernel: the slowest stage that is a
    # single launch (neighbours, each conv, slice); the splat stage (seven
    # kernels) is reported in `stages` with its own HBM roofline
    # (with --op deform: the DeformSlice + classifier kernel itself)
    single = [n for n in names if n not in ("splat", "slice_bwd", "coarse_lattice", "downsample", "upsample",
                                            "lattice", "distribute", "deform_bwd", "upsample_bwd", "downsample_bwd",
                                            "distribute_bwd")]
    dominant = "deform" if args.op == "deform" else max(single, key=lambda n: stage_ms[n])
    rf = dict(stages[dominant])
    rf["ms_stage"] = rf.pop("ms")
    # The slice and the deform slice are one kernel each, whose launch can
    # record HIP events at the kernel's own start and end (the library's stage
    # timing): their roofline takes the kernel's duration from those, over as
    # many more eager steps, without the gap before the launch that the
    # events around the stage include.
    if dominant in ("slice", "deform") and not args.graph:
        kms = kernel_time(pipe, dominant, args.steps)
        rf.update(roofline_entry(dominant, kms, work[dominant]))
        rf["ms_kernel"] = kms
        rf["timing"] = ("HIP events recorded by the kernel's launch at its start and end (library stage timing), "
                        f"mean over {args.steps} eager steps")
    else:
        rf["timing"] = "HIP events around the stage (stages)"
    rf["kernel"] = dominant
    rf["traffic"], rf["traffic_source"] = measured_traffic(WORKLOAD_NAMES.get(args.config, w.name), dominant)
    rf["algorithmic_bytes"] = work[dominant]["bytes"]
    if "flops" in work[dominant]:
        rf["algorithmic_flops"] = work[dominant]["flops"]

    out = {
        "metric": {"slice": "points/s for splat+conv+slice",
                   "deform": "points/s for splat+conv+deformslice+classifier",
                   "train": "points/s for splat+conv+slice forward and backward",
                   "unet": "points/s for splat+conv+downsample+upsample+slice",
                   "pointnet": "points/s for lattice+distribute/pointnet+conv+slice"}[args.op]
                  + (" forward and backward" if args.backward else ""),
        "value": w.m * args.steps / sec,
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 splat/slice, " + "+".join(f"{c.dtype} conv" for c in w.convs),
        "data": "synthetic",
        "config": {"workload": WORKLOAD_NAMES.get(args.config, w.name), "points": w.m, "d": w.d,
                   "sigma": float(w.sigma[0]), "channels": w.C, "vertices": V,
                   "convs": [f"{c.c_in}->{c.c_out} {c.dtype}" for c in w.convs]}
                  | ({"classes": n_cls, "tail": "deformslice+classifier"} if args.op == "deform" else {})
                  | ({"tail": "slice, then the backward pass of every stage"} if args.op == "train" else {})
                  | ({"backward": "the backward pass of every stage, down to the "
                                  + ("PointNet's parameters" if args.op == "pointnet" else "point features")}
                     if args.backward else {})
                  | ({"coarse_vertices": Vc, "tail": "downsample+upsample+slice"} if args.op == "unet" else {})
                  | ({"head": f"distribute+pointnet ({w.d}+{f_raw} -> 16 -> 32 -> 64, group norm "
                              f"{pipe.pn_groups} per cloud)"} if args.op == "pointnet" else {}),
        "roofline": rf,
        "stages": stages,
        "vertices_per_s": V / (sum(v for n, v in stage_ms.items() if n.startswith("conv")) * 1e-3),
        "hbm_frac_splat_slice": None if args.op in ("deform", "pointnet") else splat_slice_frac(work, stage_ms),
        "timing": ("value: " + ("graph replays" if args.graph else "eager steps") + " of the whole step, no "
                   "events inside; stages: HIP events around each stage of eager steps on the same stream; "
                   "roofline: see its own timing field; stages_cold: the same after evicting the caches "
                   "before every step (512 MiB write, outside the events), roofline of the median"),
    }
    if cold is not None:
        out["stages_cold"] = stages_cold
    if args.op == "slice" and not args.no_other_configs:
        # the two performance targets, each on the workload it is set on
        others = {str(c): other_config(c, min(args.steps, 20), min(args.warmup, 5))
                  for c in EXTRA_CONFIGS if c != args.config}
        out["other_configs"] = others
        mine = {"workload": out["config"]["workload"], "stages": stages,
                "hbm_frac_splat_slice": out["hbm_frac_splat_slice"]}
        by_cfg = {str(args.config): mine, **others}
        hb = {k: v["hbm_frac_splat_slice"] for k, v in by_cfg.items()}
        tg = {"splat_slice_hbm_frac": {"target": TARGET_HBM_FRAC, "value": out["hbm_frac_splat_slice"],
                                       "workload": out["config"]["workload"],
                                       "met": out["hbm_frac_splat_slice"] >= TARGET_HBM_FRAC,
                                       "by_workload": {by_cfg[k]["workload"]: v for k, v in hb.items()}}}
        lidar = by_cfg.get("4")
        if lidar is not None:
            st = lidar["stages"]["conv0_128x128_bf16"]
            tg["bf16_conv_c128_mfma_frac"] = {
                "target": TARGET_MFMA_FRAC, "value": st["frac"], "bound": st["bound"],
                "achieved_tflops": st["achieved"], "peak_tflops": st["peak"], "ms": st["ms"],
                "kernel": "conv0_128x128_bf16", "workload": lidar["workload"],
                "met": st["bound"] == "mfma" and st["frac"] >= TARGET_MFMA_FRAC}
        out["targets"] = tg
    if not args.no_cpu_baseline and (args.op in ("train", "unet", "pointnet") or args.backward):
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget, pipe.dw if args.op == "deform" else None,
                                           train=pipe.backward, unet=args.op == "unet",
                                           pointnet=(pipe.pn_layers, pipe.pn_groups) if args.op == "pointnet" else None)
    elif not args.no_cpu_baseline:
        dw = pipe.dw if args.op == "deform" else None
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget, dw)
        from threadpoolctl import threadpool_limits

        with threadpool_limits(limits=1):
            out["cpu_baseline_1core"] = cpu_baseline(w, args.cpu_budget / 2, dw)
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
