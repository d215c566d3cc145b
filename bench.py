#!/usr/bin/env python3
"""Benchmark of the Approximate Random Dropout hot path on one MI355X.

Default workload: the wide MLP 8192-8192-8192-8192 (bf16 with fp32
accumulation, batch 2048, ReLU) with row-based dropout on both hidden layers
at p = 0.7. Each step samples a fresh pattern per hidden layer from the
distribution K searched for p, plans it, gathers the compact weights of the
layers whose inputs are dropped on the device, and runs fwd, bwd_data and
bwd_weight of all three layers (bwd_data of the first layer is not needed).
The headline value is TFLOP/s counted on the work actually kept; the same
steps at p = 0.3 and 0.5 and at p = 0 (period 1: the same kernels with
nothing dropped) give the speedups. Other workloads (--workload): the single
FC layer, the 3-layer MLP 784-2048-2048-10, the tile-pattern layer, the LSTM
layers.

The roofline entry covers the layer GEMM calls: a second pass of the same
steps brackets every call with HIP events on the step's stream, and
achieved = sum of their kept FLOPs / sum of their durations.

Prints one JSON line. Inputs are synthetic and resident in HBM before timing.
"""

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fwd+bwd layer TFLOP/s (kept work) & speedup vs p=0 at p=0.3/0.5/0.7"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}   # MI355X dense matrix peaks
PEAK_HBM_GBS = 8000.0
PATTERN_SEED = 8939


class Mlp:
    """An MLP whose hidden layers take row-based dropout patterns sampled per
    step from K(p). Layers are FC: Xt[K][B] -> Yt[N][B]. With
    last_input_major the last layer, whose outputs carry no pattern, stores its
    weights (and their gradient and momentum) input-major, W^T[K][N]: its kept
    inputs are then whole rows, read in place, and no step compacts it."""

    def __init__(self, name, dims, batch, dtype, init, seed, relu_last=False, dropped="skip", streams=1,
                 last_input_major=False):
        import torch
        from paper_1805_08939_amd import api, synth
        self.api, self.torch = api, torch
        self.name, self.dims, self.B, self.dtype = name, dims, batch, dtype
        self.ard_dtype = api.ARD_F32 if dtype == "f32" else api.ARD_BF16
        dev = torch.device("cuda:0")
        g = synth.generator(seed)
        sdt = synth.storage_dtype(dtype)
        L = len(dims) - 1
        self.L = L
        self.X0 = synth.to_storage(synth.normal(g, (dims[0], batch)), dtype).to(dev)
        self.input_major = [last_input_major and l == L - 1 for l in range(L)]
        self.W = []
        for l in range(L):
            w = synth.xavier(g, dims[l + 1], dims[l]) if init == "xavier" else synth.he(g, dims[l + 1], dims[l])
            w = synth.to_storage(w, dtype).to(dev)
            self.W.append(w.t().contiguous() if self.input_major[l] else w)
        self.bias = [torch.zeros(dims[l + 1], device=dev) for l in range(L)]
        self.Y = [torch.zeros(dims[l + 1], batch, dtype=sdt, device=dev) for l in range(L)]
        self.dY = [torch.zeros(dims[l + 1], batch, dtype=sdt, device=dev) for l in range(L)]
        self.dY[-1].copy_(synth.to_storage(synth.normal(g, (dims[-1], batch)), dtype).to(dev))
        self.dW = [torch.zeros(*((dims[l], dims[l + 1]) if self.input_major[l] else (dims[l + 1], dims[l])),
                               device=dev) for l in range(L)]
        self.db = [torch.zeros(dims[l + 1], device=dev) for l in range(L)]
        self.plans = [api.ard_row_plan() for _ in range(L - 1)]
        # compact weights of the layers whose inputs are dropped (built once per
        # step, shared by fwd and bwd_data) and one workspace for split-K sums:
        # at most two rounds of 256 output tiles of 256 x 256 fp32
        self.comp_layers = [l for l in range(1, L) if not self.input_major[l]]
        self.Wc = [torch.zeros(dims[l + 1] * ((dims[l] + 7) // 8 * 8), dtype=sdt, device=dev)
                   if l in self.comp_layers else None for l in range(L)]
        self.ws = torch.empty(2 * 256 * 256 * 256, dtype=torch.float32, device=dev)
        # streams == 2: the step runs the compaction and the weight-gradient
        # products of the hidden layers on a second stream (same priority),
        # with its own split-K workspace, beside the chain fwd -> bwd_data
        self.streams = streams
        if streams == 2:
            self.side = torch.cuda.Stream(device=dev)
            self.ws_side = torch.empty_like(self.ws)
            self.ev = [torch.cuda.Event() for _ in range(5)]
        self.K = None
        self.config = {"workload": name, "global_batch": batch, "layers": dims,
                       "patterns": "row-based, sampled per step from K(p), n_max 16", "dropped": dropped,
                       "streams": streams}
        self.dropped = api.ARD_DROPPED_ZERO if dropped == "zero" else api.ARD_DROPPED_SKIP
        # raw device addresses and the stream handle, resolved once: the step
        # then costs one C call per launch with no per-call tensor lookups
        self.stream = torch.cuda.current_stream().cuda_stream
        self.ptr = {
            "X0": self.X0.data_ptr(), "W": [w.data_ptr() for w in self.W],
            "Wc": [w.data_ptr() if w is not None else None for w in self.Wc],
            "bias": [b.data_ptr() for b in self.bias],
            "Y": [y.data_ptr() for y in self.Y], "dY": [d.data_ptr() for d in self.dY],
            "dW": [w.data_ptr() for w in self.dW], "db": [b.data_ptr() for b in self.db]}

    def set_rate(self, p):
        api = self.api
        self.p = p
        self.K, _ = api.ard_search_distribution(p)
        # descriptors point at the plan structs, which each step refills
        self.descs, self.cdescs = [], []
        for l in range(self.L):
            in_plan = self.plans[l - 1] if l > 0 else None
            out_plan = self.plans[l] if l < self.L - 1 else None
            act = api.ARD_ACT_RELU if l < self.L - 1 else api.ARD_ACT_NONE
            args = (self.ard_dtype, self.B, self.dims[l], self.dims[l + 1], in_plan, out_plan, 1.0, act,
                    self.dropped)
            if self.input_major[l]:
                self.descs.append(api.fc_desc(*args, api.ARD_WEIGHTS_INPUT_MAJOR))
                self.cdescs.append(self.descs[-1])
                continue
            self.descs.append(api.fc_desc(*args))
            # a layer whose inputs are dropped reads the compact weights and
            # writes the compact weight gradient dWc[kept_out][ldc] into dW
            self.cdescs.append(api.fc_desc(*args, api.ARD_WEIGHTS_COMPACT_GRAD) if l > 0 else self.descs[-1])
        # the calls of one step, in order, with their arguments resolved once.
        # A layer whose inputs are all kept in a step (period 1) needs no
        # compact weight copy: it reads W itself through the full-layout
        # descriptor; so every layer has two call sets, picked per step.
        P, st = self.ptr, self.stream
        acts = [P["X0"]] + P["Y"]
        ws = (self.ws.data_ptr(), self.ws.numel() * 4)

        def layer_calls(l, compact):
            desc = self.cdescs[l] if compact else self.descs[l]
            w = P["Wc"][l] if compact else P["W"][l]
            calls = {("fwd", l): (api.ard_fc_fwd, (desc, acts[l], w, P["bias"][l], P["Y"][l], ws, st), {})}
            if l > 0:
                # the layer's backward in one call: bwd_data (which also applies the
                # ReLU derivative of the layer below, Xgate = that layer's output, so
                # every dY[l] below the top is already gated and is passed with
                # Yt = None) and bwd_weight, one launch where both are small
                calls[("bwd", l)] = (api.ard_fc_bwd, (desc, acts[l], P["dY"][l], None, w, P["dY"][l - 1],
                                                      P["dW"][l], P["db"][l], ws, st), {"Xgate": acts[l]})
            else:  # the network input needs no gradient
                calls[("bwd_weight", l)] = (api.ard_fc_bwd_weight, (desc, acts[l], P["dY"][l], None, P["dW"][l],
                                                                    P["db"][l], ws, st), {})
            return calls

        self.layer_calls = [{False: layer_calls(l, False), True: layer_calls(l, True) if l in self.comp_layers
                             else None} for l in range(self.L)]

        def split_calls(l, compact):
            """The layer's products as separate calls: fwd and bwd_data on the
            step stream, bwd_weight of a hidden layer on the second stream."""
            desc = self.cdescs[l] if compact else self.descs[l]
            w = P["Wc"][l] if compact else P["W"][l]
            calls = {("fwd", l): (api.ard_fc_fwd, (desc, acts[l], w, P["bias"][l], P["Y"][l], ws, st), {})}
            if l > 0:
                calls[("bwd_data", l)] = (api.ard_fc_bwd_data, (desc, P["dY"][l], None, w, P["dY"][l - 1], ws, st),
                                          {"Xgate": acts[l]})
                side = (self.ws_side.data_ptr(), self.ws_side.numel() * 4), self.side.cuda_stream
            else:
                side = ws, st
            calls[("bwd_weight", l)] = (api.ard_fc_bwd_weight, (desc, acts[l], P["dY"][l], None, P["dW"][l],
                                                                P["db"][l]) + side, {})
            return calls

        if self.streams == 2:
            self.split_calls = [{False: split_calls(l, False), True: split_calls(l, True) if l in self.comp_layers
                                 else None} for l in range(self.L)]
        # one compaction launch per step for the layers whose inputs are
        # dropped: the marshalled arguments of every subset, built once
        import itertools
        self.compact_batches = {}
        for r in range(1, len(self.comp_layers) + 1):
            for sub in itertools.combinations(self.comp_layers, r):
                self.compact_batches[sub] = api.CompactBatch([self.cdescs[l] for l in sub],
                                                             [P["W"][l] for l in sub], [P["Wc"][l] for l in sub])
        self.order = [("fwd", l) for l in range(self.L)]
        self.order += [("bwd", l) for l in reversed(range(1, self.L))] + [("bwd_weight", 0)]

    def patterns(self, it):
        return [self.api.ard_sample_row_pattern(self.K, PATTERN_SEED, l + 1, it) for l in range(self.L - 1)]

    # ------------------------------------------------------- conventional dropout
    def set_conventional(self, p):
        """The same network under conventional dropout (Sec. II-C), the paper's
        baseline: dense layer GEMMs (the p = 0 calls) and a Bernoulli(1 - p)
        element mask, drawn per step on the device, on each hidden layer's
        output (forward) and output derivative (backward)."""
        import torch
        api = self.api
        self.conv_p = p
        if not hasattr(self, "masks"):
            self.masks = [torch.zeros((self.dims[l + 1] * self.B + 31) // 32, dtype=torch.int32, device="cuda")
                          for l in range(self.L - 1)]
            self.ptr["mask"] = [m.data_ptr() for m in self.masks]
        self.dense = []
        for l in range(self.L):
            act = api.ARD_ACT_RELU if l < self.L - 1 else api.ARD_ACT_NONE
            layout = api.ARD_WEIGHTS_INPUT_MAJOR if self.input_major[l] else api.ARD_WEIGHTS_FULL
            self.dense.append(api.fc_desc(self.ard_dtype, self.B, self.dims[l], self.dims[l + 1], None, None, 1.0, act,
                                          api.ARD_DROPPED_SKIP, layout))

    def sgd_step(self, dense):
        """Momentum SGD on every layer (lr 1e-6, momentum 0.9; the cost does not
        depend on the values): on the approximate path restricted to the
        step's kept weights, on the conventional one dense."""
        import torch
        api, P, st = self.api, self.ptr, self.stream
        if not hasattr(self, "V"):
            self.V = [torch.zeros_like(w) for w in self.dW]
            self.Vb = [torch.zeros_like(b) for b in self.db]
            P["V"], P["Vb"] = [v.data_ptr() for v in self.V], [v.data_ptr() for v in self.Vb]
        for l in range(self.L):
            desc = self.dense[l] if dense else (self.cdescs[l] if l in self.step_compact else self.descs[l])
            api.ard_fc_sgd_momentum(desc, P["W"][l], P["V"][l], P["dW"][l], P["bias"][l], P["Vb"][l], P["db"][l],
                                    1e-6, 0.9, st)

    def conventional_step(self, it):
        api, P, st, L, B = self.api, self.ptr, self.stream, self.L, self.B
        acts = [P["X0"]] + P["Y"]
        ws = (self.ws.data_ptr(), self.ws.numel() * 4)
        d, dt, p = self.dense, self.ard_dtype, self.conv_p
        for l in range(L):
            api.ard_fc_fwd(d[l], acts[l], P["W"][l], P["bias"][l], P["Y"][l], ws, st)
            if l < L - 1:
                api.ard_dropout_fwd(dt, self.dims[l + 1], B, p, 1.0, PATTERN_SEED, l + 1, it, P["Y"][l],
                                    P["mask"][l], st)
        for l in reversed(range(1, L)):
            if l < L - 1:
                api.ard_dropout_bwd(dt, self.dims[l + 1], B, 1.0, P["mask"][l], P["dY"][l], st)
            api.ard_fc_bwd(d[l], acts[l], P["dY"][l], None, P["W"][l], P["dY"][l - 1], P["dW"][l], P["db"][l], ws, st,
                           Xgate=acts[l])
        api.ard_dropout_bwd(dt, self.dims[1], B, 1.0, P["mask"][0], P["dY"][0], st)
        api.ard_fc_bwd_weight(d[0], acts[0], P["dY"][0], None, P["dW"][0], P["db"][0], ws, st)

    def kept(self, pats):
        api = self.api
        n = [self.dims[0]]
        for l, (per, off) in enumerate(pats):
            n.append(api.ard_row_kept(self.dims[l + 1], per, off))
        n.append(self.dims[-1])
        return n

    def kept_flops(self, pats):
        """(total, per-call dict): 2*B*K_kept*N_kept per GEMM (fwd, bwd_data,
        bwd_weight); no bwd_data for layer 0. A ("bwd", l) call holds two GEMMs."""
        n = self.kept(pats)
        per = {}
        for l in range(self.L):
            f = 2.0 * self.B * n[l] * n[l + 1]
            per[("fwd", l)] = f
            if l > 0:
                per[("bwd", l)] = 2.0 * f
            else:
                per[("bwd_weight", l)] = f
        return sum(per.values()), per

    def kept_bytes(self, pats):
        """Per-call algorithmic HBM bytes: the kept operands read once and the
        kept outputs written once (weights and activations in the storage
        dtype, weight and bias gradients fp32); bwd_data also reads the ReLU
        gate of the layer below."""
        n, B = self.kept(pats), self.B
        es = 2 if self.dtype == "bf16" else 4
        per = {}
        for l in range(self.L):
            w, x, y = n[l + 1] * n[l] * es, n[l] * B * es, n[l + 1] * B * es
            per[("fwd", l)] = w + x + y
            dw = y + x + n[l + 1] * n[l] * 4 + 4 * n[l + 1]
            per[("bwd", l) if l > 0 else ("bwd_weight", l)] = dw + (w + y + 2 * x if l > 0 else 0)
        return per

    def prepare(self, it):
        """Samples this step's patterns, plans them and gathers the compact
        weights of the layers whose inputs are dropped. Returns the patterns and
        the step's calls {key: (fn, args, kwargs)}. The FC kernels read a row
        pattern's kept set (offset + period * i) as strided views, so the plans
        are list-free: no device index list is built, none is read."""
        api, P, st = self.api, self.ptr, self.stream
        pats = self.patterns(it)
        for l, (per, off) in enumerate(pats):
            api.ard_plan_rows(self.dims[l + 1], per, off, None, st, plan=self.plans[l])
        calls = dict(self.layer_calls[0][False])
        sub = tuple(l for l in self.comp_layers if pats[l - 1][0] > 1)
        self.step_compact = sub  # layers whose dW holds the compact gradient this step
        if sub:
            api.ard_fc_compact_weights_batch(self.compact_batches[sub], st)
        for l in range(1, self.L):
            calls.update(self.layer_calls[l][l in sub])
        return pats, calls

    def step_overlapped(self, it):
        """One step on two streams. The step stream runs the dependent chain
        fwd 0 .. L-1, bwd_data L-1 .. 1, bwd_weight 0; the second stream runs
        the compaction (joined before the first layer that reads compact
        weights) and the weight-gradient products of the layers above the
        first (each after the step stream has produced its operands), and is
        joined at the end of the step, so the next step (or anything after
        it on the step stream) sees every result."""
        api, P, st = self.api, self.ptr, self.stream
        torch = self.torch
        main, side, ev = torch.cuda.current_stream(), self.side, self.ev
        pats = self.patterns(it)
        for l, (per, off) in enumerate(pats):
            api.ard_plan_rows(self.dims[l + 1], per, off, None, st, plan=self.plans[l])
        sub = tuple(l for l in self.comp_layers if pats[l - 1][0] > 1)
        self.step_compact = sub
        calls = [self.split_calls[l][l in sub] for l in range(self.L)]

        def run(key):
            fn, args, kw = calls[key[1]][key]
            fn(*args, **kw)

        if sub:
            ev[0].record(main)
            side.wait_event(ev[0])  # the previous step's readers of the compact weights are done
            api.ard_fc_compact_weights_batch(self.compact_batches[sub], side.cuda_stream)
            ev[1].record(side)
        for l in range(self.L):
            if l == 1 and sub:
                main.wait_event(ev[1])
            run(("fwd", l))
            if l == self.L - 2:  # the input of the top layer is ready: its weight gradient can start
                ev[2].record(main)
        side.wait_event(ev[2])
        run(("bwd_weight", self.L - 1))
        for l in reversed(range(1, self.L)):
            run(("bwd_data", l))
            if l > 1:
                ev[3].record(main)
                side.wait_event(ev[3])
                run(("bwd_weight", l - 1))
        run(("bwd_weight", 0))
        ev[4].record(side)
        main.wait_event(ev[4])
        return pats, []

    def step(self, it, events=None):
        """One step of iteration it. With events (a list of (start, end) event
        pairs, consumed from the front), every call is bracketed by a pair
        recorded on the current stream, and the calls run one after the other
        on the step stream; returns the patterns and the list of (call key,
        start, end) used. Without events, a two-stream workload runs the
        overlapped schedule."""
        if events is None and getattr(self, "streams", 1) == 2:
            return self.step_overlapped(it)
        pats, calls = self.prepare(it)
        used = []
        for key in self.order:
            fn, args, kw = calls[key]
            if events is not None:
                e0, e1 = events.pop()
                e0.record()
                fn(*args, **kw)
                e1.record()
                used.append((key, e0, e1))
            else:
                fn(*args, **kw)
        return pats, used

    # ------------------------------------------------------------------ oracle
    def oracle_step(self, pats):
        """The same step through the fp64 oracle (masked dense layers)."""
        import numpy as np
        from oracle import fc as ofc
        from oracle import patterns as opat
        masks = [opat.row_mask(self.dims[0], 1, 0)]
        for l, (per, off) in enumerate(pats):
            masks.append(opat.row_mask(self.dims[l + 1], per, off))
        masks.append(opat.row_mask(self.dims[-1], 1, 0))
        X = self._host["X0"]
        Ys = []
        for l in range(self.L):
            act = "relu" if l < self.L - 1 else "none"
            X = ofc.fc_forward(X, self._host["W"][l], None, masks[l], masks[l + 1], 1.0, act)
            Ys.append(X)
        dY = self._host["dY"]
        for l in reversed(range(self.L)):
            act = "relu" if l < self.L - 1 else "none"
            Xin = Ys[l - 1] if l > 0 else self._host["X0"]
            dX, dW, db = ofc.fc_backward(Xin, self._host["W"][l], Ys[l], dY, masks[l], masks[l + 1], 1.0, act)
            dY = dX
        return np.abs(dW).sum()

    def full_weight(self, l):
        """Layer l's weights as W[N][K] (a view of the stored tensor)."""
        return self.W[l].t() if self.input_major[l] else self.W[l]

    def host_copies(self):
        self._host = {"X0": self.X0.double().cpu().numpy().T.copy(),
                      "W": [self.full_weight(l).double().cpu().numpy() for l in range(self.L)],
                      "dY": self.dY[-1].double().cpu().numpy().T.copy()}


class FcLayer:
    """One fully connected layer whose output neurons take a row-based pattern
    per step (Sec. III-A): fwd, then bwd_data and bwd_weight (one call). At
    p = 0.5 the pattern keeps every second neuron (K = e_2, the offset drawn
    per step); at other rates (dp, offset) come from the K searched for p."""

    def __init__(self, name, n_in, n_out, batch, dtype, w_std, seed):
        import torch
        from paper_1805_08939_amd import api, synth
        self.api, self.torch = api, torch
        self.name, self.K, self.N, self.B, self.dtype = name, n_in, n_out, batch, dtype
        self.ard_dtype = api.ARD_F32 if dtype == "f32" else api.ARD_BF16
        dev = torch.device("cuda:0")
        g = synth.generator(seed)
        sdt = synth.storage_dtype(dtype)
        X = synth.to_storage(synth.normal(g, (batch, n_in)), dtype)
        W = synth.to_storage(synth.normal(g, (n_out, n_in), w_std), dtype)
        dY = synth.to_storage(synth.normal(g, (batch, n_out)), dtype)
        self._host_src = (X, W, dY)
        self.Xt, self.W, self.dYt = X.T.contiguous().to(dev), W.to(dev), dY.T.contiguous().to(dev)
        self.bias = torch.zeros(n_out, device=dev)
        self.Yt = torch.zeros(n_out, batch, dtype=sdt, device=dev)
        self.dXt = torch.zeros(n_in, batch, dtype=sdt, device=dev)
        self.dW = torch.zeros(n_out, n_in, device=dev)
        self.db = torch.zeros(n_out, device=dev)
        self.plan = api.ard_row_plan()
        self.desc = api.fc_desc(self.ard_dtype, batch, n_in, n_out, None, self.plan, 1.0, api.ARD_ACT_NONE,
                                api.ARD_DROPPED_SKIP)
        self.ws = torch.empty(max(api.ard_fc_workspace_bytes(
            api.fc_desc(self.ard_dtype, batch, n_in, n_out)), 16) // 4, device=dev)
        self.stream = torch.cuda.current_stream().cuda_stream
        self.order = [("fwd", 0), ("bwd", 0)]
        self.config = {"workload": name, "global_batch": batch, "layer": [n_in, n_out],
                       "patterns": "row-based on the outputs: K = e_2 at p = 0.5 (every second neuron kept, offset "
                                   "drawn per step), else sampled per step from K(p), n_max 16",
                       "dropped": "skip"}

    def set_rate(self, p):
        import numpy as np
        self.p = p
        if p == 0.5:
            self.Kdist = np.zeros(16)
            self.Kdist[1] = 1.0
        else:
            self.Kdist, _ = self.api.ard_search_distribution(p)

    def patterns(self, it):
        return [self.api.ard_sample_row_pattern(self.Kdist, PATTERN_SEED, 1, it)]

    def kept_flops(self, pats):
        f = 2.0 * self.B * self.K * self.api.ard_row_kept(self.N, *pats[0])
        per = {("fwd", 0): f, ("bwd", 0): 2.0 * f}
        return 3.0 * f, per

    def kept_bytes(self, pats):
        """Algorithmic HBM bytes per call (see Mlp.kept_bytes)."""
        es = 2 if self.dtype == "bf16" else 4
        n = self.api.ard_row_kept(self.N, *pats[0])
        w, x, y = n * self.K * es, self.K * self.B * es, n * self.B * es
        return {("fwd", 0): w + x + y, ("bwd", 0): (w + y + x) + (y + x + 4 * n * self.K + 4 * n)}

    def prepare(self, it):
        api, st = self.api, self.stream
        pats = self.patterns(it)
        api.ard_plan_rows(self.N, *pats[0], None, st, plan=self.plan)
        d, ws = self.desc, (self.ws.data_ptr(), self.ws.numel() * 4)
        calls = {("fwd", 0): (api.ard_fc_fwd, (d, self.Xt, self.W, self.bias, self.Yt, ws, st), {}),
                 ("bwd", 0): (api.ard_fc_bwd, (d, self.Xt, self.dYt, None, self.W, self.dXt, self.dW, self.db, ws,
                                               st), {})}
        return pats, calls

    step = Mlp.step

    def oracle_step(self, pats):
        from oracle import fc as ofc
        from oracle import patterns as opat
        X, W, dY = self._host
        m_in, m_out = opat.row_mask(self.K, 1, 0), opat.row_mask(self.N, *pats[0])
        Y = ofc.fc_forward(X, W, None, m_in, m_out)
        return ofc.fc_backward(X, W, Y, dY, m_in, m_out)

    def host_copies(self):
        from paper_1805_08939_amd import synth
        self._host = tuple(synth.as_f64(t).numpy() for t in self._host_src)


class TileLayer:
    """One layer under a tile-based pattern: each step draws a Bernoulli(1 - p)
    keep bitmap over the 64 x 64 tiles of W[N][K] on the device together with
    the kept-tile lists (one kernel; the same draws as the host sampler, which
    the FLOP count and the oracle use), then runs the forward and the backward
    (bwd_data and bwd_weight in one launch), reading and writing only kept
    tiles."""

    def __init__(self, name, n, k, batch, tile, dtype, seed, w_std, fused_bwd=True):
        import torch
        from paper_1805_08939_amd import api, synth
        self.api, self.torch = api, torch
        self.name, self.N, self.K, self.B, self.tile, self.dtype = name, n, k, batch, tile, dtype
        self.tn, self.tk = n // tile, k // tile
        dev = torch.device("cuda:0")
        g = synth.generator(seed)
        sdt = synth.storage_dtype(dtype)
        X = synth.to_storage(synth.normal(g, (batch, k)), dtype)
        W = synth.to_storage(synth.normal(g, (n, k), w_std), dtype)
        dY = synth.to_storage(synth.normal(g, (batch, n)), dtype)
        self._host_src = (X, W, dY)
        self.Xt, self.W, self.dYt = X.T.contiguous().to(dev), W.to(dev), dY.T.contiguous().to(dev)
        self.Yt = torch.empty(n, batch, dtype=sdt, device=dev)
        self.dXt = torch.empty(k, batch, dtype=sdt, device=dev)
        self.dW = torch.empty(n, k, dtype=torch.float32, device=dev)
        self.words = (self.tn * self.tk + 31) // 32
        # two plan buffers: the plan of step i + 1 is built on a second stream
        # (same priority) while step i's products run (see step_pipelined)
        self.bits_bufs = [torch.empty(self.words, dtype=torch.int32, device=dev) for _ in range(2)]
        self.ws_bufs = [torch.empty(max(api.ard_tile_plan_workspace_bytes(self.tn, self.tk), 16) // 4,
                                    dtype=torch.int32, device=dev) for _ in range(2)]
        self.bits_dev, self.plan_ws = self.bits_bufs[0], self.ws_bufs[0]
        self.side = torch.cuda.Stream(device=dev)
        self.ev_plan = [torch.cuda.Event() for _ in range(2)]
        self.ev_done = [torch.cuda.Event() for _ in range(2)]
        self.planned = {}  # buffer -> (step, plan) built into it
        self.desc = api.tile_desc(api.ARD_BF16 if dtype == "bf16" else api.ARD_F32, batch, k, n, 1.0,
                                  api.ARD_DROPPED_SKIP)
        self.stream = torch.cuda.current_stream().cuda_stream
        # the backward as one call (bwd_data and bwd_weight in one launch), or
        # the two calls one after the other
        self.fused_bwd = fused_bwd
        self.order = [("fwd", 0), ("bwd", 0)] if fused_bwd else [("fwd", 0), ("bwd_data", 0), ("bwd_weight", 0)]
        self.config = {"workload": name, "global_batch": batch, "layer": [k, n], "tile": tile,
                       "patterns": "Bernoulli tile bitmap per step, keep probability 1 - p", "dropped": "skip"}

    def set_rate(self, p):
        self.p = p
        self.planned = {}

    def patterns(self, it):
        bits = self.api.ard_tile_bitmap_bernoulli(self.tn, self.tk, self.p, PATTERN_SEED, 0, it)
        return bits, self.api.ard_bitmap_popcount(bits, self.tn * self.tk)

    def plan_into(self, it, buf, stream):
        """Draws step it's bitmap and plans it on the device, into plan buffer buf."""
        return self.api.ard_plan_tiles_bernoulli(self.N, self.K, self.tile, self.p, PATTERN_SEED, 0, it,
                                                 self.bits_bufs[buf], self.ws_bufs[buf], stream)

    def layer_calls(self, plan):
        api, d, st = self.api, self.desc, self.stream
        return {("fwd", 0): (api.ard_tile_fwd, (d, plan, self.Xt, self.W, self.Yt, st), {}),
                ("bwd", 0): (api.ard_tile_bwd, (d, plan, self.Xt, self.dYt, self.W, self.dXt, self.dW, st), {}),
                ("bwd_data", 0): (api.ard_tile_bwd_data, (d, plan, self.dYt, self.W, self.dXt, st), {}),
                ("bwd_weight", 0): (api.ard_tile_bwd_weight, (d, plan, self.Xt, self.dYt, self.dW, st), {})}

    def step_pipelined(self, it):
        """Step it with the plan built one step ahead: the second stream plans
        step it + 1 into the other buffer (once step it - 1, its last reader,
        is done) while the step stream runs step it's products on the plan
        built during step it - 1 (or now, at the start of a run of steps)."""
        torch = self.torch
        main, side = torch.cuda.current_stream(), self.side
        b, nb = it % 2, (it + 1) % 2
        if self.planned.get(b, (None,))[0] != it:  # first step of a run: plan it now
            side.wait_stream(main)
            self.planned[b] = (it, self.plan_into(it, b, side.cuda_stream))
            self.ev_plan[b].record(side)
        side.wait_event(self.ev_done[nb])
        self.planned[nb] = (it + 1, self.plan_into(it + 1, nb, side.cuda_stream))
        self.ev_plan[nb].record(side)
        main.wait_event(self.ev_plan[b])
        for fn, args, kw in (self.layer_calls(self.planned[b][1])[k] for k in self.order):
            fn(*args, **kw)
        self.ev_done[b].record(main)
        return it, []

    def kept_flops(self, pats):
        if isinstance(pats, int):  # a step number: its pattern from the host sampler
            pats = self.patterns(pats)
        f = 2.0 * self.B * self.tile * self.tile * pats[1]
        per = {key: (2 * f if key[0] == "bwd" else f) for key in self.order}
        return sum(per.values()), per

    def kept_bytes(self, pats):
        """Algorithmic HBM bytes per call: the kept tiles of W (read) or dW
        (fp32, written), the activations and outputs of every row once."""
        if isinstance(pats, int):
            pats = self.patterns(pats)
        es = 2 if self.dtype == "bf16" else 4
        wt = pats[1] * self.tile * self.tile
        x, y = self.K * self.B * es, self.N * self.B * es
        per = {("fwd", 0): wt * es + x + y, ("bwd_data", 0): wt * es + y + x, ("bwd_weight", 0): y + x + 4 * wt}
        per[("bwd", 0)] = per[("bwd_data", 0)] + per[("bwd_weight", 0)]
        return {key: per[key] for key in self.order}

    def prepare(self, it):
        self.planned = {}
        return it, self.layer_calls(self.plan_into(it, 0, self.stream))

    def step(self, it, events=None):
        """Without events the pipelined step; with events (the roofline pass)
        the plan and the products one after the other on the step stream."""
        if events is None:
            return self.step_pipelined(it)
        return Mlp.step(self, it, events)

    def oracle_step(self, pats):
        import numpy as np
        from oracle import patterns as opat
        from oracle import tdp as otdp
        grid = opat.bitmap_to_grid(list(pats[0]), self.tn, self.tk).astype(np.float64)
        M = np.kron(grid, np.ones((self.tile, self.tile)))
        X, W, dY = self._host
        otdp.tdp_forward(X, W, M)
        return otdp.tdp_backward(X, W, dY, M)

    def host_copies(self):
        from paper_1805_08939_amd import synth
        self._host = tuple(synth.as_f64(t).numpy() for t in self._host_src)


class TileLayerTdp(TileLayer):
    """The same layer under the paper's tile-based pattern (Sec. III-B): each
    step draws (dp, offset) from K(p) and keeps the tiles t = tn * tiles_k + tk
    with t mod dp == offset. The bitmaps of every (dp, offset) are built once on
    the device; a step plans the drawn one there."""

    def __init__(self, **kw):
        super().__init__(**kw)
        self.config["patterns"] = "tile-based (dp, offset) per step from K(p), n_max 16"
        self.tdp_bits = {}

    def set_rate(self, p):
        api, torch = self.api, self.torch
        self.p = p
        self.planned = {}
        self.Kdist, _ = api.ard_search_distribution(p)
        for per in range(1, len(self.Kdist) + 1):
            for off in range(per):
                if (per, off) not in self.tdp_bits:
                    bits = api.ard_tile_bitmap_tdp(self.tn, self.tk, per, off)
                    dev = torch.from_numpy(bits.view("int32").copy()).to("cuda")
                    self.tdp_bits[(per, off)] = (dev, api.ard_bitmap_popcount(bits, self.tn * self.tk), bits)

    def patterns(self, it):
        per, off = self.api.ard_sample_row_pattern(self.Kdist, PATTERN_SEED, 0, it)
        _, nnz, bits = self.tdp_bits[(per, off)]
        return bits, nnz, (per, off)

    def plan_into(self, it, buf, stream):
        """Plans step it's (dp, offset) bitmap (resident on the device) into plan buffer buf."""
        _, nnz, pat = self.patterns(it)
        return self.api.ard_plan_tiles(self.N, self.K, self.tile, self.tdp_bits[pat][0], nnz, self.ws_bufs[buf],
                                       stream)


class Lstm:
    """One LSTM layer whose hidden units take a row-based pattern sampled per
    sequence from K(p): the gate GEMMs run on the kept hidden set (forward, then
    BPTT backward)."""

    def __init__(self, name, T, batch, inputs, hidden, dtype, seed):
        import torch
        from paper_1805_08939_amd import api, synth
        self.api, self.torch = api, torch
        self.name, self.T, self.B, self.I, self.H, self.dtype = name, T, batch, inputs, hidden, dtype
        dev = torch.device("cuda:0")
        g = synth.generator(seed)
        X = synth.uniform(g, (T, batch, inputs), 0.1)
        W = synth.uniform(g, (4 * hidden, inputs + hidden), 0.1)
        b = synth.uniform(g, (4 * hidden,), 0.1)
        dHs = synth.normal(g, (T, batch, hidden))
        self._host_src = (X, W, b, dHs)
        self.X = X.permute(0, 2, 1).contiguous().to(dev)
        self.W, self.b = W.to(dev), b.to(dev)
        self.dHs = dHs.permute(0, 2, 1).contiguous().to(dev)
        self.Hs = torch.empty(T, hidden, batch, device=dev)
        self.hT = torch.empty(hidden, batch, device=dev)
        self.cT = torch.empty(hidden, batch, device=dev)
        self.dX = torch.empty(T, inputs, batch, device=dev)
        self.dW = torch.empty(4 * hidden, inputs + hidden, device=dev)
        self.db = torch.empty(4 * hidden, device=dev)
        self.dh0 = torch.empty(hidden, batch, device=dev)
        self.dc0 = torch.empty(hidden, batch, device=dev)
        self.idx = torch.empty(hidden, dtype=torch.int32, device=dev)
        self.plan = api.ard_row_plan()
        self.desc = api.lstm_desc(api.ARD_F32, T, batch, inputs, hidden, self.plan)
        full = api.ard_plan_rows(hidden, 1, 0, self.idx)  # the workspace of the largest kept set
        nbytes = api.ard_lstm_workspace_bytes(api.lstm_desc(api.ARD_F32, T, batch, inputs, hidden, full))
        self.ws = torch.empty(max(nbytes, 16) // 4 + 1, device=dev)
        self.stream = torch.cuda.current_stream().cuda_stream
        self.order = [("fwd", 0), ("bwd", 0)]
        self.config = {"workload": name, "global_batch": batch, "seq_len": T, "input": inputs, "hidden": hidden,
                       "patterns": "row-based on hidden units, sampled per sequence from K(p), n_max 16"}

    def set_rate(self, p):
        self.p = p
        self.K, _ = self.api.ard_search_distribution(p)

    def patterns(self, it):
        return [self.api.ard_sample_row_pattern(self.K, PATTERN_SEED, 1, it)]

    def kept_flops(self, pats):
        S = self.api.ard_row_kept(self.H, *pats[0])
        f = 2.0 * self.T * self.B * (self.I + S) * 4 * S  # input projection + recurrence
        per = {("fwd", 0): f, ("bwd", 0): 2.0 * f}
        return 3.0 * f, per

    def prepare(self, it):
        api, st = self.api, self.stream
        pats = self.patterns(it)
        api.ard_plan_rows(self.H, *pats[0], self.idx, st, plan=self.plan)
        d = self.desc
        calls = {("fwd", 0): (api.ard_lstm_fwd, (d, self.X, self.W, self.b, None, None, self.Hs, self.hT,
                                                  self.cT, self.ws, st), {}),
                 ("bwd", 0): (api.ard_lstm_bwd, (d, self.X, self.dHs, None, None, self.ws, self.dX, self.dW,
                                                  self.db, self.dh0, self.dc0, st), {})}
        return pats, calls

    step = Mlp.step

    def oracle_step(self, pats):
        from oracle import lstm as olstm
        from oracle import patterns as opat
        X, W, b, dHs = self._host
        m = opat.row_mask(self.H, *pats[0])
        Hs, hT, cT, cache = olstm.lstm_forward(X, W, b, m)
        return olstm.lstm_backward(X, W, m, cache, dHs)

    def host_copies(self):
        from paper_1805_08939_amd import synth
        self._host = tuple(synth.as_f64(t).numpy() for t in self._host_src)


class LstmStack:
    """Stacked LSTM layers (Sec. IV-C's language model shape), each with a
    hidden-unit pattern sampled per sequence from K(p); a layer's input rows
    are the layer below's hidden units, so its input plan is that layer's
    pattern and its input products shrink with it (K-side compaction).
    Forward through the stack, then BPTT backward from the top, the top
    layer's dX being the layer below's dHs."""

    def __init__(self, name, T, batch, inputs, hidden, layers, dtype, seed):
        import torch
        from paper_1805_08939_amd import api, synth
        self.api, self.torch = api, torch
        self.name, self.T, self.B, self.I, self.H, self.NL, self.dtype = name, T, batch, inputs, hidden, layers, dtype
        dev = torch.device("cuda:0")
        g = synth.generator(seed)
        X = synth.uniform(g, (T, batch, inputs), 0.1)
        self.X = X.permute(0, 2, 1).contiguous().to(dev)
        self.Ws, self.bs, self.Hs, self.dX, self.dW, self.db, self.ws, self.idx = [], [], [], [], [], [], [], []
        self.plans = [api.ard_row_plan() for _ in range(layers)]
        for l in range(layers):
            i = inputs if l == 0 else hidden
            self.Ws.append(synth.uniform(g, (4 * hidden, i + hidden), 0.1).to(dev))
            self.bs.append(synth.uniform(g, (4 * hidden,), 0.1).to(dev))
            self.Hs.append(torch.empty(T, hidden, batch, device=dev))
            self.dX.append(torch.empty(T, i, batch, device=dev))
            self.dW.append(torch.empty(4 * hidden, i + hidden, device=dev))
            self.db.append(torch.empty(4 * hidden, device=dev))
            self.idx.append(torch.empty(hidden, dtype=torch.int32, device=dev))
            full = api.ard_plan_rows(hidden, 1, 0, self.idx[l])  # the largest kept set bounds the workspace
            nbytes = api.ard_lstm_workspace_bytes(api.lstm_desc(api.ARD_F32, T, batch, i, hidden, full))
            self.ws.append(torch.empty(max(nbytes, 16) // 4 + 1, device=dev))
        self.dHs = synth.normal(g, (T, batch, hidden)).permute(0, 2, 1).contiguous().to(dev)
        self.descs = [api.lstm_desc(api.ARD_F32, T, batch, inputs if l == 0 else hidden, hidden, self.plans[l],
                                    self.plans[l - 1] if l > 0 else None) for l in range(layers)]
        self.stream = torch.cuda.current_stream().cuda_stream
        self.order = [("fwd", 0), ("bwd", 0)]
        self.config = {"workload": name, "global_batch": batch, "seq_len": T, "input": inputs, "hidden": hidden,
                       "layers": layers,
                       "patterns": "row-based on each layer's hidden units, sampled per sequence from K(p), n_max 16; "
                                   "each layer's input plan is the pattern of the layer below"}

    def set_rate(self, p):
        self.p = p
        self.K, _ = self.api.ard_search_distribution(p)

    def patterns(self, it):
        return [self.api.ard_sample_row_pattern(self.K, PATTERN_SEED, l + 1, it) for l in range(self.NL)]

    def kept(self, pats):
        return [self.api.ard_row_kept(self.H, *pt) for pt in pats]

    def kept_flops(self, pats):
        S = self.kept(pats)
        f = 0.0
        for l in range(self.NL):
            ic = self.I if l == 0 else S[l - 1]
            f += 2.0 * self.T * self.B * (ic + S[l]) * 4 * S[l]
        per = {("fwd", 0): f, ("bwd", 0): 2.0 * f}
        return 3.0 * f, per

    def prepare(self, it):
        api, st = self.api, self.stream
        pats = self.patterns(it)
        for l, pt in enumerate(pats):
            api.ard_plan_rows(self.H, *pt, self.idx[l], st, plan=self.plans[l])

        def fwd():
            for l in range(self.NL):
                x = self.X if l == 0 else self.Hs[l - 1]
                api.ard_lstm_fwd(self.descs[l], x, self.Ws[l], self.bs[l], None, None, self.Hs[l], None, None,
                                 self.ws[l], st)

        def bwd():
            for l in reversed(range(self.NL)):
                x = self.X if l == 0 else self.Hs[l - 1]
                dh = self.dHs if l == self.NL - 1 else self.dX[l + 1]
                api.ard_lstm_bwd(self.descs[l], x, dh, None, None, self.ws[l], self.dX[l] if l > 0 else None,
                                 self.dW[l], self.db[l], None, None, st)
        return pats, {("fwd", 0): (fwd, (), {}), ("bwd", 0): (bwd, (), {})}

    step = Mlp.step

    def host_copies(self):
        self._host = {"X": self.X.double().cpu().numpy().transpose(0, 2, 1),
                      "W": [w.double().cpu().numpy() for w in self.Ws],
                      "b": [b.double().cpu().numpy() for b in self.bs],
                      "dHs": self.dHs.double().cpu().numpy().transpose(0, 2, 1)}

    def oracle_step(self, pats):
        """The stack through the fp64 oracle (one sequence)."""
        from oracle import lstm as olstm
        from oracle import patterns as opat
        X = self._host["X"]
        masks = [opat.row_mask(self.H, *pt) for pt in pats]
        caches = []
        for l in range(self.NL):
            W, b = self._host["W"][l], self._host["b"][l]
            m_in = masks[l - 1] if l > 0 else None
            Hs, _, _, cache = olstm.lstm_forward(X, W, b, masks[l], m_in=m_in)
            caches.append((X, W, cache, m_in))
            X = Hs
        dH = self._host["dHs"]
        for l in reversed(range(self.NL)):
            Xl, W, cache, m_in = caches[l]
            dH = olstm.lstm_backward(Xl, W, masks[l], cache, dH, m_in=m_in)[0]
        return dH


class LstmTile:
    """One LSTM layer whose weight matrix W[4H][I+H] takes the paper's tile
    pattern, (dp, offset) drawn from K(p) per sequence over its 64 x 64 tiles:
    the gate products read only kept tiles, the weight gradient is computed on
    kept tiles only; every hidden unit is kept."""

    def __init__(self, name, T, batch, inputs, hidden, tile, dtype, seed):
        import torch
        from paper_1805_08939_amd import api, synth
        self.api, self.torch = api, torch
        self.name, self.T, self.B, self.I, self.H, self.tile, self.dtype = name, T, batch, inputs, hidden, tile, dtype
        dev = torch.device("cuda:0")
        g = synth.generator(seed)
        self.X = synth.uniform(g, (T, batch, inputs), 0.1).permute(0, 2, 1).contiguous().to(dev)
        self.W = synth.uniform(g, (4 * hidden, inputs + hidden), 0.1).to(dev)
        self.b = synth.uniform(g, (4 * hidden,), 0.1).to(dev)
        self.dHs = synth.normal(g, (T, batch, hidden)).permute(0, 2, 1).contiguous().to(dev)
        self.Hs = torch.empty(T, hidden, batch, device=dev)
        self.dX = torch.empty(T, inputs, batch, device=dev)
        self.dW = torch.empty(4 * hidden, inputs + hidden, device=dev)
        self.db = torch.empty(4 * hidden, device=dev)
        self.tn, self.tk = 4 * hidden // tile, (inputs + hidden) // tile
        self.plan_ws = torch.empty(max(api.ard_tile_plan_workspace_bytes(self.tn, self.tk), 16) // 4,
                                   dtype=torch.int32, device=dev)
        self.tdp_bits = {}
        self.ws = None
        self.stream = torch.cuda.current_stream().cuda_stream
        self.order = [("fwd", 0), ("bwd", 0)]
        self.config = {"workload": name, "global_batch": batch, "seq_len": T, "input": inputs, "hidden": hidden,
                       "tile": tile, "patterns": "tile-based (dp, offset) on W per sequence from K(p), n_max 16"}

    def set_rate(self, p):
        api, torch = self.api, self.torch
        self.p = p
        self.Kdist, _ = api.ard_search_distribution(p)
        for per in range(1, len(self.Kdist) + 1):
            for off in range(per):
                if (per, off) not in self.tdp_bits:
                    bits = api.ard_tile_bitmap_tdp(self.tn, self.tk, per, off)
                    dev = torch.from_numpy(bits.view("int32").copy()).to("cuda")
                    self.tdp_bits[(per, off)] = (dev, api.ard_bitmap_popcount(bits, self.tn * self.tk))

    def patterns(self, it):
        return [self.api.ard_sample_row_pattern(self.Kdist, PATTERN_SEED, 1, it)]

    def kept_flops(self, pats):
        nnz = self.tdp_bits[tuple(pats[0])][1]
        f = 2.0 * self.T * self.B * nnz * self.tile * self.tile
        per = {("fwd", 0): f, ("bwd", 0): 2.0 * f}
        return 3.0 * f, per

    def prepare(self, it):
        api, st = self.api, self.stream
        pats = self.patterns(it)
        dbits, nnz = self.tdp_bits[tuple(pats[0])]
        plan = api.ard_plan_tiles(4 * self.H, self.I + self.H, self.tile, dbits, nnz, self.plan_ws, st)
        d = api.lstm_tile_desc(api.ARD_F32, self.T, self.B, self.I, self.H, plan)
        if self.ws is None:
            self.ws = self.torch.empty(api.ard_lstm_tile_workspace_bytes(d) // 4 + 1, device="cuda")
        calls = {("fwd", 0): (api.ard_lstm_tile_fwd, (d, self.X, self.W, self.b, None, None, self.Hs, None, None,
                                                       self.ws, st), {}),
                 ("bwd", 0): (api.ard_lstm_tile_bwd, (d, self.W, self.dHs, None, None, self.ws, self.dX, self.dW,
                                                       self.db, None, None, st), {})}
        return pats, calls

    step = Mlp.step

    def host_copies(self):
        self._host = (self.X.double().cpu().numpy().transpose(0, 2, 1), self.W.double().cpu().numpy(),
                      self.b.double().cpu().numpy(), self.dHs.double().cpu().numpy().transpose(0, 2, 1))

    def oracle_step(self, pats):
        import numpy as np
        from oracle import lstm as olstm
        from oracle import patterns as opat
        from oracle import prng as oprng
        X, W, b, dHs = self._host
        words = oprng.tile_bitmap_tdp(self.tn, self.tk, *pats[0])
        Wm = W * opat.tile_mask(words, self.tn, self.tk, self.tile)
        ones = np.ones(self.H)
        _, _, _, cache = olstm.lstm_forward(X, Wm, b, ones)
        return olstm.lstm_backward(X, Wm, ones, cache, dHs)


WORKLOADS = {
    "fc784": dict(cls="FcLayer", name="fc-784x512-fp32-b64", n_in=784, n_out=512, batch=64, dtype="f32",
                  w_std=0.05, seed=1805 + 0),
    "mlp784": dict(cls="Mlp", name="mlp-784-2048-2048-10-fp32-b128", dims=[784, 2048, 2048, 10], batch=128,
                   dtype="f32", init="xavier", seed=1805 + 1),
    "tile4096": dict(cls="TileLayer", name="tile-4096x4096-bf16-b512-t64", n=4096, k=4096, batch=512, tile=64,
                     dtype="bf16", seed=1805 + 2, w_std=0.02),
    "tile4096tdp": dict(cls="TileLayerTdp", name="tile-4096x4096-bf16-b512-t64-tdp", n=4096, k=4096, batch=512,
                        tile=64, dtype="bf16", seed=1805 + 2, w_std=0.02),
    "lstm1024": dict(cls="Lstm", name="lstm-t35-b64-i1024-h1024-fp32", T=35, batch=64, inputs=1024, hidden=1024,
                     dtype="f32", seed=1805 + 3),
    "lstm2x1500": dict(cls="LstmStack", name="lstm-2x1500-t35-b20-fp32", T=35, batch=20, inputs=1500, hidden=1500,
                       layers=2, dtype="f32", seed=1805 + 5),
    "lstm2x1500b40": dict(cls="LstmStack", name="lstm-2x1500-t35-b40-fp32", T=35, batch=40, inputs=1500,
                          hidden=1500, layers=2, dtype="f32", seed=1805 + 5),
    "lstm1024tile": dict(cls="LstmTile", name="lstm-t35-b64-i1024-h1024-fp32-tile64", T=35, batch=64, inputs=1024,
                         hidden=1024, tile=64, dtype="f32", seed=1805 + 3),
    "mlp8192": dict(cls="Mlp", name="mlp-8192x4-bf16-b2048", dims=[8192, 8192, 8192, 8192], batch=2048,
                    dtype="bf16", init="he", seed=1805 + 4, streams=2, last_input_major=True),
}


class NoGC:
    """Python's cyclic garbage collector off for a timed region: a collection
    pass stalls the host (and so a host-fed GPU queue) for milliseconds."""

    def __enter__(self):
        import gc
        self.was = gc.isenabled()
        gc.collect()
        gc.disable()

    def __exit__(self, *exc):
        import gc
        if self.was:
            gc.enable()


def time_steps(wl, steps, warmup, it0):
    """GPU time of `steps` steps after `warmup` untimed ones: one HIP event
    pair on the step stream around the whole run; FLOPs counted afterwards
    from the host sampler's patterns."""
    with NoGC():
        return _time_steps(wl, steps, warmup, it0)


def _time_steps(wl, steps, warmup, it0):
    import torch
    for i in range(warmup):
        wl.step(it0 + i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    all_pats = [wl.step(it0 + warmup + i)[0] for i in range(steps)]
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_flops = sum(wl.kept_flops(pats)[0] for pats in all_pats)  # FLOP accounting off the timed path
    return {"ms": start.elapsed_time(end), "wall_s": wall, "flops": total_flops}


def roofline_pass(wl, steps, warmup, it0):
    with NoGC():
        return _roofline_pass(wl, steps, warmup, it0)


def _roofline_pass(wl, steps, warmup, it0):
    """The same steps once more with every layer call bracketed by a HIP event
    pair on the step stream. Returns, per call key and in total, the number of
    calls, the summed event time, the summed kept FLOPs and the algorithmic
    bytes of the calls. A one-element int16 fill before and after the timed steps
    marks their kernels in a rocprofv3 trace or counter run of this command
    (--summarize-pass)."""
    import torch
    for i in range(warmup):
        wl.step(it0 + i)
    torch.cuda.synchronize()
    lead = spin_cycles(LEAD_MS)
    marker = torch.empty(1, dtype=torch.int16, device="cuda:0")
    marker.fill_(1)
    n = steps * len(wl.order)
    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    runs = []
    for i in range(steps):
        # a bounded spin ahead of each step keeps the GPU busy while the host
        # enqueues the step, so an event pair brackets the call's kernels and
        # not the host's launch latency
        torch.cuda._sleep(lead)
        runs.append(wl.step(it0 + warmup + i, events))
    marker.fill_(2)
    torch.cuda.synchronize()
    per = {}
    nbytes = 0.0
    for pats, used in runs:
        _, fl = wl.kept_flops(pats)
        by = wl.kept_bytes(pats) if hasattr(wl, "kept_bytes") else {}
        for key, e0, e1 in used:
            rec = per.setdefault(key, [0, 0.0, 0.0])
            rec[0] += 1
            rec[1] += e0.elapsed_time(e1)
            rec[2] += fl[key]
            nbytes += by.get(key, 0.0)
    calls = sum(r[0] for r in per.values())
    ms = sum(r[1] for r in per.values())
    flops = sum(r[2] for r in per.values())
    return {"calls": calls, "ms": ms, "flops": flops, "per": per, "bytes": nbytes}


LEAD_MS = 2.0  # GPU spin ahead of each step of the roofline pass


def spin_cycles(ms):
    """Cycles of torch's spin kernel that take about ms milliseconds on this
    GPU (measured once with a HIP event pair)."""
    import torch
    global _SPIN_PER_MS
    if _SPIN_PER_MS is None:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)
        e0.record()
        torch.cuda._sleep(1_000_000)
        e1.record()
        torch.cuda.synchronize()
        _SPIN_PER_MS = 1_000_000 / max(e0.elapsed_time(e1), 1e-3)
    return int(ms * _SPIN_PER_MS)


_SPIN_PER_MS = None


def time_conventional(wl, steps, warmup, it0):
    """GPU ms of `steps` conventional-dropout steps after `warmup` untimed ones
    (the same timing as the approximate-dropout steps)."""
    with NoGC():
        return _time_conventional(wl, steps, warmup, it0)


def _time_conventional(wl, steps, warmup, it0):
    import torch
    for i in range(warmup):
        wl.conventional_step(it0 + i)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        wl.conventional_step(it0 + warmup + i)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end)


def time_training(wl, steps, warmup, it0, conventional):
    """GPU ms of `steps` training steps (a step of the path, or of the
    conventional network, followed by the momentum-SGD update of every layer)."""
    with NoGC():
        return _time_training(wl, steps, warmup, it0, conventional)


def _time_training(wl, steps, warmup, it0, conventional):
    import torch

    def one(it):
        if conventional:
            wl.conventional_step(it)
        else:
            wl.step(it)
        wl.sgd_step(conventional)
    for i in range(warmup):
        one(it0 + i)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        one(it0 + warmup + i)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end)


def cpu_baseline(wl, p, budget_s):
    """The oracle on the host cores: as many steps as fit in ~budget_s."""
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    wl.set_rate(p)
    n, flops, t = 0, 0.0, 0.0
    while t < budget_s and n < 1000:
        pats = wl.patterns(10_000 + n)
        t0 = time.perf_counter()
        wl.oracle_step(pats)
        t += time.perf_counter() - t0
        flops += wl.kept_flops(pats)[0]
        n += 1
    return {"value": flops / t / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} steps of the same workload at p={p} (fp64 masked dense layers, numpy), {t:.1f} s"}


def code_text(src):
    """C/C++/HIP source text without its comments, with every run of blanks
    within a line made one space and blank lines dropped (string and character
    literals kept as they are): what the compiler sees of the code, up to
    layout."""
    out, i, n = [], 0, len(src)
    while i < n:
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif src[i] in "\"'":
            q, j = src[i], i + 1
            while j < n and src[j] != q:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(src[i])
            i += 1
    lines = (" ".join(line.split()) for line in "".join(out).split("\n"))
    return "\n".join(line for line in lines if line)


def source_digest():
    """sha256 over the code of the kernel sources and the header (comments and
    layout left out): a stored counter reading holds only for the code it was
    taken on."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1805_08939_amd", "csrc")
    files = sorted(os.path.join(csrc, f) for f in os.listdir(csrc))
    files.append(os.path.join(ROOT, "include", "ard.h"))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, encoding="utf-8") as fh:
            h.update(code_text(fh.read()).encode())
    return h.hexdigest()


def traffic_record(workload, p, steps):
    """HBM bytes per layer call of the roofline pass, from the committed
    rocprofv3 counter summaries (FETCH_SIZE and WRITE_SIZE passes over the same
    command, each scaled by what the counter reads for a plain copy of known
    size). None when no summary covers this workload, rate and step count, or
    when the kernel sources changed since."""
    pdir = os.path.join(ROOT, "profiles")
    if not os.path.isdir(pdir):
        return None
    digest = source_digest()
    for f in sorted(os.listdir(pdir)):
        if not f.endswith((".txt", ".md")):
            continue
        with open(os.path.join(pdir, f)) as fh:
            for line in fh:
                if not line.startswith("traffic-record: "):
                    continue
                rec = json.loads(line[len("traffic-record: "):])
                if (rec.get("workload") == workload and rec.get("p") == p and rec.get("steps") == steps
                        and rec.get("source_digest") == digest):
                    return rec["bytes_per_call"]
    return None


def _demangle(name):
    if not name.startswith("_Z"):
        return name
    import shutil
    import subprocess
    tool = shutil.which("c++filt")
    if tool:  # GNU c++filt does not know the bf16 mangling DF16b: spell it as a vendor type
        out = subprocess.run([tool, name.replace("DF16b", "u6__bf16")], capture_output=True, text=True).stdout
        return out.strip() or name
    return name


def _short_kernel(name):
    name = _demangle(name).replace("void ", "").replace("ard::", "").replace("(anonymous namespace)::", "")
    depth, out = 0, []
    for ch in name:  # drop the argument list, keep template arguments
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).strip()[:150]


def _col(row, *names):
    low = {k.lower(): v for k, v in row.items()}
    for n in names:
        if n.lower() in low and low[n.lower()] not in (None, ""):
            return low[n.lower()]
    raise KeyError(names[0])


def summarize_trace(path, top, last=0, tail=0):
    """Per (kernel, grid) table of a rocprofv3 kernel trace (CSV); with
    last > 0 only each kernel's last dispatches, with tail > 0 only the run's
    last tail dispatches (a replayed call)."""
    import csv
    with open(path) as fh:
        recs = sorted(((int(_col(r, "Start_Timestamp")), r) for r in csv.DictReader(fh)), key=lambda t: t[0])
    if tail > 0:
        recs = recs[-tail:]
    agg = {}
    for start, r in recs:
        name = _short_kernel(_col(r, "Kernel_Name"))
        wg = [max(int(_col(r, f"Workgroup_Size_{d}")), 1) for d in "XYZ"]
        grid = tuple(int(_col(r, f"Grid_Size_{d}")) // w for d, w in zip("XYZ", wg))
        end = int(_col(r, "End_Timestamp"))
        agg.setdefault((name, grid), []).append((start, (end - start) / 1000.0))
    rows = {}
    for key, v in agg.items():
        v.sort()
        if last > 0:
            v = v[-last:]
        rows[key] = (len(v), sum(us for _, us in v))
    tot = sum(us for _, us in rows.values()) or 1.0
    print("| calls | total us | avg us | % | workgroups | kernel |")
    print("|---:|---:|---:|---:|---|---|")
    for (name, grid), (n, us) in sorted(rows.items(), key=lambda kv: -kv[1][1])[:top]:
        print(f"| {n} | {us:.1f} | {us / n:.2f} | {100 * us / tot:.2f} | {grid[0]}x{grid[1]}x{grid[2]} | `{name}` |")


MARKER = "FillFunctor<short>"
# per-step work outside the layer calls, and the pass's spin kernel
EXCLUDE = ("compact_weights_kernel", "plan_tiles_kernel", "plan_tiles_wide_kernel", "plan_rows_kernel", "spin_kernel")


def summarize_pass(path, top, calls, kind):
    """The kernels of bench.py's roofline pass, between the two marker fills,
    from a rocprofv3 kernel trace (kind "trace": time per kernel) or counter
    collection (kind "counters": counter sums per kernel), per layer call of
    the pass (`calls` of them)."""
    import csv
    with open(path) as fh:
        rows = list(csv.DictReader(fh))
    if kind == "trace":
        recs = sorted(((int(_col(r, "Start_Timestamp")), r) for r in rows), key=lambda t: t[0])
        marks = [i for i, (_, r) in enumerate(recs) if MARKER in _col(r, "Kernel_Name")]
        assert len(marks) >= 2, "marker fills not found"
        inside = [r for _, r in recs[marks[0] + 1:marks[1]] if not any(x in _col(r, "Kernel_Name") for x in EXCLUDE)]
        per = {}
        for r in inside:
            name = _short_kernel(_col(r, "Kernel_Name"))
            us = (int(_col(r, "End_Timestamp")) - int(_col(r, "Start_Timestamp"))) / 1000.0
            a = per.setdefault(name, [0, 0.0])
            a[0] += 1
            a[1] += us
        tot = sum(v[1] for v in per.values())
        print(f"roofline pass: {len(inside)} kernels, {tot:.1f} us of kernel time, {tot / calls:.2f} us per layer "
              f"call ({calls} calls)")
        print("| dispatches | total us | avg us | us per layer call | % | kernel |")
        print("|---:|---:|---:|---:|---:|---|")
        for name, (n, us) in sorted(per.items(), key=lambda kv: -kv[1][1])[:top]:
            print(f"| {n} | {us:.1f} | {us / n:.2f} | {us / calls:.2f} | {100 * us / tot:.2f} | `{name}` |")
        return
    disp = {}
    for r in rows:
        d = int(_col(r, "Dispatch_Id"))
        e = disp.setdefault(d, {"name": _col(r, "Kernel_Name"), "v": {}})
        c = _col(r, "Counter_Name")
        e["v"][c] = e["v"].get(c, 0.0) + float(_col(r, "Counter_Value"))
    ids = sorted(disp)
    marks = [d for d in ids if MARKER in disp[d]["name"]]
    assert len(marks) >= 2, "marker fills not found"
    # the step's compaction runs between the calls, outside their event brackets
    inside = [disp[d] for d in ids if marks[0] < d < marks[1] and not any(x in disp[d]["name"] for x in EXCLUDE)]
    per, tot = {}, {}
    for e in inside:
        name = _short_kernel(e["name"])
        for c, v in e["v"].items():
            a = per.setdefault((name, c), [0, 0.0])
            a[0] += 1
            a[1] += v
            tot[c] = tot.get(c, 0.0) + v
    for c, v in sorted(tot.items()):
        print(f"roofline pass: {c} sum {v:.1f} over {len(inside)} dispatches, {v / calls:.1f} per layer call")
    print("| dispatches | sum | per layer call | counter | kernel |")
    print("|---:|---:|---:|---|---|")
    for (name, c), (n, v) in sorted(per.items(), key=lambda kv: -kv[1][1])[:top]:
        print(f"| {n} | {v:.1f} | {v / calls:.1f} | {c} | `{name}` |")


def summarize_counters(path, top, last=0, tail=0):
    """Per (kernel, grid size, counter) mean value per dispatch of a rocprofv3
    counter collection (CSV); with last > 0 only each kernel's last
    dispatches, with tail > 0 only the run's last tail dispatches."""
    import csv
    agg = {}
    with open(path) as fh:
        rows = list(csv.DictReader(fh))
    keep = None
    if tail > 0:
        keep = set(sorted({int(_col(r, "Dispatch_Id")) for r in rows})[-tail:])
    for r in rows:
        disp = int(_col(r, "Dispatch_Id"))
        if keep is not None and disp not in keep:
            continue
        key = (_short_kernel(_col(r, "Kernel_Name")), _col(r, "Grid_Size"), _col(r, "Counter_Name"), disp)
        agg[key] = agg.get(key, 0.0) + float(_col(r, "Counter_Value"))
    by = {}
    for (name, grid, counter, disp), v in agg.items():
        by.setdefault((name, grid, counter), []).append((disp, v))
    per = {}
    for key, vals in by.items():
        vals.sort()
        if last > 0:
            vals = vals[-last:]
        per[key] = (len(vals), sum(v for _, v in vals))
    print("| dispatches | mean per dispatch | counter | grid size (work-items) | kernel |")
    print("|---:|---:|---|---:|---|")
    for (name, grid, counter), (n, v) in sorted(per.items(), key=lambda kv: -kv[1][1])[:top]:
        print(f"| {n} | {v / n:.1f} | {counter} | {grid} | `{name}` |")


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mlp8192", choices=sorted(WORKLOADS))
    ap.add_argument("--p", type=float, default=0.7, help="dropout rate of the headline value")
    ap.add_argument("--dropped", default="skip", choices=["skip", "zero"],
                    help="MLP workloads: dropped outputs and gradients left untouched (skip) or written 0 (zero)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--streams", type=int, choices=[1, 2], default=None,
                    help="MLP workloads: one stream, or two (compaction and weight gradients beside the chain)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-baselines", action="store_true",
                    help="skip the conventional-dropout and training-step comparisons")
    ap.add_argument("--summarize-trace", metavar="CSV", help="print a per-kernel table of a rocprofv3 kernel trace")
    ap.add_argument("--summarize-counters", metavar="CSV", help="print per-kernel means of a rocprofv3 counter run")
    ap.add_argument("--top", type=int, default=25)
    ap.add_argument("--last", type=int, default=0, help="--summarize-trace / --summarize-counters: only the last N dispatches per kernel")
    ap.add_argument("--tail", type=int, default=0,
                    help="--summarize-trace / --summarize-counters: only the run's last N dispatches")
    ap.add_argument("--summarize-pass", metavar="CSV",
                    help="per-kernel table of the roofline pass from a rocprofv3 trace or counter CSV of this command")
    ap.add_argument("--pass-kind", default="trace", choices=["trace", "counters"])
    ap.add_argument("--digest", action="store_true", help="print the kernel source digest")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of 1 GiB (3 times), the reference for HBM counters")
    args = ap.parse_args()
    if args.summarize_trace:
        return summarize_trace(args.summarize_trace, args.top, args.last, args.tail)
    if args.summarize_counters:
        return summarize_counters(args.summarize_counters, args.top, args.last, args.tail)
    if args.summarize_pass:
        spec = WORKLOADS[args.workload]
        per_step = {"Mlp": 2 * (len(spec.get("dims", ())) - 1)}.get(spec["cls"], 2)  # fwd and bwd per layer
        return summarize_pass(args.summarize_pass, args.top, args.steps * per_step, args.pass_kind)
    if args.digest:
        return print(source_digest())
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": src.numel() * 4, "copies": 3}), flush=True)
        return
    from paper_1805_08939_amd import _ffi
    _ffi.lib()
    spec = dict(WORKLOADS[args.workload])
    cls = {"Mlp": Mlp, "FcLayer": FcLayer, "TileLayer": TileLayer, "TileLayerTdp": TileLayerTdp, "Lstm": Lstm,
           "LstmStack": LstmStack, "LstmTile": LstmTile}[spec.pop("cls")]
    if args.dropped != "skip":
        if cls is not Mlp:
            sys.exit("--dropped zero applies to the MLP workloads")
        spec["dropped"] = args.dropped
    if args.streams is not None:
        if cls is not Mlp:
            sys.exit("--streams applies to the MLP workloads")
        spec["streams"] = args.streams
    wl = cls(**spec)
    dtype = spec["dtype"]
    if not args.no_cpu_baseline:
        wl.host_copies()  # the oracle's inputs, taken before any GPU timing

    rates = sorted({0.0, 0.3, 0.5, 0.7, args.p})
    # Alg. 1 on the host, once per rate (a one-time cost, outside the timed steps)
    from paper_1805_08939_amd import api
    k_search = {}
    for p in rates:
        t_s = time.perf_counter()
        _, info = api.ard_search_distribution(p)
        k_search[f"{p}"] = {"ms": (time.perf_counter() - t_s) * 1e3, "iters": int(info.iters),
                            "loss": float(info.loss), "p_global": float(info.p_global),
                            "converged": bool(info.converged)}
    results = {}
    for i, p in enumerate(rates):
        wl.set_rate(p)
        r = time_steps(wl, args.steps, args.warmup, 1_000_000 * (i + 1))
        results[p] = r
        print(f"# p={p}: {r['ms'] / args.steps:.4f} ms/step, kept {r['flops'] / args.steps / 1e9:.3f} GFLOP/step, "
              f"{r['flops'] / (r['ms'] * 1e-3) / 1e12:.3f} TFLOP/s", file=sys.stderr, flush=True)

    # the roofline: the headline steps again (same iterations, so the same
    # patterns), every layer call bracketed by HIP events on the step stream
    wl.set_rate(args.p)
    head_it0 = 1_000_000 * (rates.index(args.p) + 1)
    rp = roofline_pass(wl, args.steps, args.warmup, head_it0)
    print(f"# roofline pass p={args.p}: {rp['calls']} layer calls, {rp['ms'] / rp['calls'] * 1e3:.2f} us per call, "
          f"{rp['flops'] / (rp['ms'] * 1e-3) / 1e12:.3f} TFLOP/s over the calls", file=sys.stderr, flush=True)

    # the paper's own baseline (Sec. II-C, Sec. IV): conventional dropout on the
    # same network, dense GEMMs plus element masks, at the same rates
    conventional = None
    if hasattr(wl, "conventional_step") and not args.no_baselines:
        conventional = {"ms_per_step": {}, "speedup_vs_conventional": {}, "training_time_reduction": {}}
        for i, p in enumerate(rates):
            if p == 0.0:
                continue
            wl.set_conventional(p)
            ms = time_conventional(wl, args.steps, args.warmup, 5_000_000 * (i + 1)) / args.steps
            ard_ms = results[p]["ms"] / args.steps
            conventional["ms_per_step"][f"{p}"] = ms
            conventional["speedup_vs_conventional"][f"{p}"] = ms / ard_ms
            conventional["training_time_reduction"][f"{p}"] = 1.0 - ard_ms / ms
            print(f"# conventional dropout p={p}: {ms:.4f} ms/step ({ms / ard_ms:.3f}x the approximate step)",
                  file=sys.stderr, flush=True)

    # whole training steps: the same comparison with the optimizer update of
    # every layer after each step (the weights are restored afterwards)
    training = None
    if hasattr(wl, "sgd_step") and not args.no_baselines:
        saved = [w.clone() for w in wl.W]
        training = {"approximate_ms": {}, "conventional_ms": {}, "training_time_reduction": {}}
        for i, p in enumerate(rates):
            if p == 0.0:
                continue
            wl.set_rate(p)
            a_ms = time_training(wl, args.steps, args.warmup, 7_000_000 * (i + 1), False) / args.steps
            wl.set_conventional(p)
            c_ms = time_training(wl, args.steps, args.warmup, 8_000_000 * (i + 1), True) / args.steps
            training["approximate_ms"][f"{p}"] = a_ms
            training["conventional_ms"][f"{p}"] = c_ms
            training["training_time_reduction"][f"{p}"] = 1.0 - a_ms / c_ms
            print(f"# training step p={p}: approximate {a_ms:.4f} ms, conventional {c_ms:.4f} ms",
                  file=sys.stderr, flush=True)
        for w, s0 in zip(wl.W, saved):
            w.copy_(s0)
        del saved

    head = results[args.p]
    value = head["flops"] / (head["ms"] * 1e-3) / 1e12
    t0 = results[0.0]["ms"]
    speedup = {f"{p}": t0 / results[p]["ms"] for p in rates if p > 0}
    kept_frac = {f"{p}": (results[p]["flops"] / results[0.0]["flops"]) for p in rates if p > 0}
    achieved = rp["flops"] / (rp["ms"] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_TFLOPS[dtype], "unit": "TFLOP/s",
                "frac": achieved / PEAK_TFLOPS[dtype],
                "traffic": traffic_record(spec["name"], args.p, args.steps),
                "kernel": "every layer GEMM call of the timed steps at p=%g (%s), kept FLOPs only" % (
                    args.p, ", ".join("%s %d" % k for k in wl.order)),
                "avg_launch_us": rp["ms"] / rp["calls"] * 1e3, "launches": rp["calls"],
                "flops_per_launch": rp["flops"] / rp["calls"],
                "algorithmic_bytes_per_launch": rp["bytes"] / rp["calls"] if rp["bytes"] else None,
                "per_call": {"%s %d" % k: {"calls": r[0], "avg_us": r[1] / r[0] * 1e3,
                                           "tflops": r[2] / (r[1] * 1e-3) / 1e12 if r[1] > 0 else 0.0}
                             for k, r in rp["per"].items()},
                "call_ms_per_step": rp["ms"] / args.steps}
    out = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": head["ms"] / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": dict(wl.config, p=args.p),
        "speedup_vs_p0": speedup,
        "kept_flop_fraction": kept_frac,
        "time_fraction_vs_p0": {f"{p}": results[p]["ms"] / t0 for p in rates if p > 0},
        "per_p": {f"{p}": {"ms_per_step": results[p]["ms"] / args.steps,
                           "host_ms_per_step": results[p]["wall_s"] * 1e3 / args.steps,
                           "tflops_kept": results[p]["flops"] / (results[p]["ms"] * 1e-3) / 1e12}
                  for p in rates},
        "roofline": roofline,
        "k_search": k_search,
    }
    if training is not None:
        out["training_step"] = dict(training, definition="a step as above followed by momentum SGD (lr 1e-6, "
                                    "momentum 0.9) on every layer: restricted to the step's kept weights on the "
                                    "approximate path, dense under conventional dropout")
    if conventional is not None:
        out["conventional_dropout"] = dict(
            conventional, definition="dense layer GEMMs (the p = 0 kernels) plus a Bernoulli(1 - p) element mask "
                                     "kernel on each hidden output and its derivative; speedup = its step time / "
                                     "the approximate-dropout step time at the same p")
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.p, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
