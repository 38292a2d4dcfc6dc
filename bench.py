#!/usr/bin/env python3
"""CompAct layer benchmark: fwd + bwd + Adam step over every linear layer of a
synthetic model-shaped workload, on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload llama-350m]

One step = the forward of every linear layer, its backward (reverse order) and
the Adam step of every layer, on synthetic inputs resident in HBM.  Layers that
read the same input (q, k, v; gate, up) run as one group: compact_fwd_group and
compact_bwd_group (dL/dx over the concatenated weight, the sum a shared input
needs, and every G^ of the group in one split-K launch).  --no-group runs every
layer on its own (compact_fwd / compact_bwd per layer, dL/dx not summed).
Prints ONE JSON line: tokens/s, the MFMA roofline fraction of the dominant
kernel (the fused forward GEMM), per-phase timings, activation bytes saved and
the CPU oracle's throughput on the host cores.
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

from synthetic import input_groups  # noqa: E402  (layers that share an input)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fwd_traffic.json")


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama-350m")
    ap.add_argument("--fwd-mode", choices=["panel", "lds"], default="panel",
                    help="panel: P^T panel in workspace; lds: P tiles regenerated in LDS")
    ap.add_argument("--no-group", action="store_true",
                    help="run every linear layer on its own instead of grouping layers that share an input")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=1 << 30,
                    help="token slice for the oracle timing (default: the full step)")
    ap.add_argument("--reseed-period", type=int, default=50)
    ap.add_argument("--no-phases", action="store_true",
                    help="skip the per-phase timing pass (for counter collection runs)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one plain copy kernel over 256 MiB first (HBM counter calibration)")
    ap.add_argument("--proj", default="gaussian",
                    help="projection: gaussian (the paper's method), or sparse-jl[:s][:gather] (the ablation's "
                         "sparse JL, s draws per row, default 8; :gather computes z by gather-add)")
    ap.add_argument("--model-sweep", action="store_true",
                    help="instead of the benchmark: whole-model training steps of a LLaMA-350M-shaped model "
                         "(baseline, CompAct r=n/4, r=n/8) over batch sizes; one JSON line per point with the "
                         "peak allocated memory and the step time")
    ap.add_argument("--compare-blas", action="store_true",
                    help="instead of the benchmark: the dL/dx GEMM of compact_bwd (with its staging launch) "
                         "against torch.matmul (hipBLASLt) at 65536 tokens, n = 1024 and several K; one JSON "
                         "line per K")
    ap.add_argument("--sweep-batches", default="32,64,128,256,512",
                    help="batch sizes (sequences of 256 tokens) for --model-sweep")
    return ap.parse_args()


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2410_15352_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


class Model:
    """Device buffers of every CompAct linear layer of a workload."""

    def __init__(self, wl, fwd_mode, grouped=True, proj="gaussian"):
        import torch
        import paper_2410_15352_amd as cp
        from synthetic import bf16_bits, bf16_round
        self.wl, self.cp, self.torch = wl, cp, torch
        self.proj = proj
        dev = torch.device("cuda:0")
        T = wl.tokens
        assert wl.dtype == "bf16", "the benchmark workloads are bf16"

        def ld8(c):
            return (c + 7) // 8 * 8

        def dev_bf16(a, ld):
            rows, cols = a.shape
            buf = np.zeros((rows, ld), np.uint16)
            buf[:, :cols] = bf16_bits(a)
            return torch.from_numpy(buf.view(np.int16)).view(torch.bfloat16).to(dev)[:, :cols]

        def rng(seed):
            return np.random.Generator(np.random.PCG64(seed))

        # Every input group has its own activation, output and gradient
        # buffers (x, y, dL/do, dL/dx), as the layers of a model do, so no
        # launch finds its operands left in the caches by another group's.
        # When the workload's buffers would not fit in 85% of the device
        # memory, blocks share `act_sets` sets of them round-robin (reported).
        # Their values (x ~ N(0,1), dL/do ~ N(0, 1e-4)) come from a seeded
        # device generator; weights, z, G^ and the Adam moments are per layer.
        # A group's weights are column slices of one [n x sum m] tensor, its z
        # column slices of one [T x sum r] tensor.
        self.groups = input_groups(wl, grouped)
        per_block = {}
        for g in self.groups:
            Ls = [wl.layers[i] for i in g]
            n, M = Ls[0].n, sum(L.m for L in Ls)
            per_block[Ls[0].block] = per_block.get(Ls[0].block, 0) + 2 * T * 2 * (ld8(n) + ld8(M))
        need = max(per_block.values()) * len(per_block)
        budget = int(0.85 * torch.cuda.get_device_properties(dev).total_memory) - 16 * 2**30
        self.act_sets = max(1, min(len(per_block), budget // max(1, max(per_block.values()))))
        gen = torch.Generator(device=dev)
        act = {}  # (set, position of the group in its block) -> buffers

        def act_buffers(gi, n, M):
            Ls = [wl.layers[i] for i in self.groups[gi]]
            key = (Ls[0].block % self.act_sets, Ls[0].k)
            if key not in act:
                gen.manual_seed(1234 + 97 * key[0] + key[1])
                x = torch.empty(T, ld8(n), dtype=torch.bfloat16, device=dev)
                x.normal_(0.0, 1.0, generator=gen)
                dy = torch.empty(T, ld8(M), dtype=torch.bfloat16, device=dev)
                dy.normal_(0.0, 0.01, generator=gen)
                act[key] = (x[:, :n], torch.empty(T, ld8(M), dtype=torch.bfloat16, device=dev)[:, :M],
                            dy[:, :M], torch.empty(T, ld8(n), dtype=torch.bfloat16, device=dev)[:, :n])
            return act[key]

        self.x, self.y, self.dy, self.dx = [], [], [], []
        self.W, self.z = [None] * len(wl.layers), [None] * len(wl.layers)
        self.Wg, self.zg, self.msum = [], [], []
        for gi, g in enumerate(self.groups):
            Ls = [wl.layers[i] for i in g]
            n, M, R = Ls[0].n, sum(L.m for L in Ls), sum(L.r for L in Ls)
            xb, yb, dyb, dxb = act_buffers(gi, n, M)
            self.x.append(xb)
            self.y.append(yb)
            self.dy.append(dyb)
            self.dx.append(dxb)
            Wall = np.concatenate([bf16_round(0.02 * rng(1234 + L.layer_id).standard_normal((L.n, L.m), np.float32))
                                   for L in Ls], axis=1)
            Wg = dev_bf16(Wall, ld8(M))
            zg = torch.empty(T, ld8(R), dtype=torch.bfloat16, device=dev)[:, :R]
            mo = ro = 0
            for i, L in zip(g, Ls):
                self.W[i] = Wg[:, mo:mo + L.m]
                self.z[i] = zg[:, ro:ro + L.r]
                mo += L.m
                ro += L.r
            self.Wg.append(Wg)
            self.zg.append(zg)
            self.msum.append(M)
        self.act_bytes = need if self.act_sets == len(per_block) else None
        self.G, self.M, self.V = [], [], []
        for L in wl.layers:
            self.G.append(torch.empty(L.r, L.m, dtype=torch.float32, device=dev))
            self.M.append(torch.zeros(L.r, L.m, dtype=torch.float32, device=dev))
            self.V.append(torch.zeros(L.r, L.m, dtype=torch.float32, device=dev))
        if fwd_mode == "panel":
            wf = max(cp.fwd_group_workspace_bytes(wl.layers[g[0]].n, [wl.layers[i].m for i in g],
                                                  [wl.layers[i].r for i in g]) for g in self.groups)
        else:
            wf = 0
        wb = max(cp.bwd_group_workspace_bytes(T, wl.layers[g[0]].n, [wl.layers[i].m for i in g],
                                              [wl.layers[i].r for i in g]) for g in self.groups)
        wsz = max(cp.step_workspace_bytes(L.n, L.m, L.r) for L in wl.layers)
        self.batch = cp.prepare_layers([dict(W=self.W[i], G=self.G[i], M=self.M[i], V=self.V[i], seed=L.seed,
                                             alpha=wl.alpha) for i, L in enumerate(wl.layers)])
        wsz = max(wsz, cp.step_batched_workspace_bytes(self.batch))
        self.ws_f = torch.zeros(wf, dtype=torch.uint8, device=dev) if wf else None
        self.ws_b = torch.zeros(wb, dtype=torch.uint8, device=dev)
        self.ws_s = torch.zeros(wsz, dtype=torch.uint8, device=dev)
        self.seeds = [L.seed for L in wl.layers]
        self.t = 0

    def fwd(self, gi):
        g = self.groups[gi]
        Ls = [self.wl.layers[i] for i in g]
        x, y = self.x[gi], self.y[gi]
        if len(g) == 1:
            self.cp.compact_fwd(x, self.Wg[gi], y, self.zg[gi], self.seeds[g[0]], proj=self.proj, ws=self.ws_f)
        else:
            self.cp.compact_fwd_group(x, self.Wg[gi], y, self.zg[gi], [L.m for L in Ls], [L.r for L in Ls],
                                      [self.seeds[i] for i in g], proj=self.proj, ws=self.ws_f)

    def _bwd(self, gi, dx, ghat):
        g = self.groups[gi]
        Ls = [self.wl.layers[i] for i in g]
        dy = self.dy[gi]
        if len(g) == 1:
            self.cp.compact_bwd(dy, self.Wg[gi] if dx else None, self.zg[gi] if ghat else None,
                                self.dx[gi] if dx else None, self.G[g[0]] if ghat else None, ws=self.ws_b)
        else:
            self.cp.compact_bwd_group(dy, self.Wg[gi] if dx else None, self.zg[gi] if ghat else None,
                                      self.dx[gi] if dx else None, [self.G[i] for i in g] if ghat else None,
                                      [L.m for L in Ls], [L.r for L in Ls], ws=self.ws_b)

    def bwd_dx(self, gi):
        """dL/dx of a group: one GEMM over its concatenated weight."""
        self._bwd(gi, True, False)

    def bwd_ghat(self, gi):
        """G^ of every layer of a group: one split-K launch over the column slices of dL/do and z."""
        self._bwd(gi, False, True)

    def bwd(self, gi):
        """Alg. 2 for a group: compact_bwd(_group) computes dL/dx and every G^ in one call."""
        self._bwd(gi, True, True)

    def upd(self, i, t):
        wl = self.wl
        self.cp.compact_step(self.W[i], self.G[i], self.M[i], self.V[i], self.seeds[i], t, wl.lr,
                             wl.beta1, wl.beta2, wl.eps, wl.alpha, proj=self.proj, ws=self.ws_s)

    def upd_all(self, t):
        """Alg. 3 for every layer: batched Adam and decompression launches."""
        wl = self.wl
        self.batch.set_seeds(self.seeds)
        self.cp.compact_step_batched(self.batch, t, wl.lr, wl.beta1, wl.beta2, wl.eps, proj=self.proj,
                                     ws=self.ws_s)

    def step(self, reseed_period):
        self.t += 1
        ng = len(self.groups)
        for gi in range(ng):
            self.fwd(gi)
        for gi in reversed(range(ng)):
            self.bwd(gi)
        self.upd_all(self.t)
        for i in range(len(self.wl.layers)):
            self.seeds[i] = self.cp.compact_next_seed(self.seeds[i], self.t, reseed_period)


def algorithmic(wl, groups):
    """Per-step algorithmic work (sums over launches), per the kernel inventory:
    a group's forward and dL/dx read x (or write dL/dx) once."""
    T = wl.tokens
    f = dict(fwd=0.0, dx=0.0, ghat=0.0, dec=0.0)
    b = dict(fwd=0.0, dx=0.0, ghat=0.0, adam=0.0, dec=0.0)
    for g in groups:
        Ls = [wl.layers[i] for i in g]
        n, M, R = Ls[0].n, sum(L.m for L in Ls), sum(L.r for L in Ls)
        f["fwd"] += 2.0 * T * n * (M + R)
        f["dx"] += 2.0 * T * n * M
        b["fwd"] += 2.0 * (T * n + n * M + T * M + T * R)
        b["dx"] += 2.0 * (T * M + n * M + T * n)
    for L in wl.layers:
        n, m, r = L.n, L.m, L.r
        f["ghat"] += 2.0 * T * r * m
        f["dec"] += 2.0 * n * r * m
        b["ghat"] += 2.0 * (T * r + T * m) + 4.0 * r * m
        b["adam"] += 22.0 * r * m
        b["dec"] += 4.0 * n * m + 2.0 * r * m
    return f, b


def time_phases(model, torch, reps=2, step_reps=10):
    """Per-phase GPU time (ms per step) with HIP events on the launch stream.
    The step phase is short (under a millisecond), so it is repeated more."""
    ng = len(model.groups)
    stream = torch.cuda.current_stream()
    out = {}
    phases = {
        "fwd": lambda: [model.fwd(gi) for gi in range(ng)],
        "bwd_dx": lambda: [model.bwd_dx(gi) for gi in range(ng)],
        "bwd_ghat": lambda: [model.bwd_ghat(gi) for gi in range(ng)],
        "step": lambda: model.upd_all(max(model.t, 1)),
    }
    for name, fn in phases.items():
        fn()  # warm
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        k = step_reps if name == "step" else reps
        e0.record(stream)
        for _ in range(k):
            fn()
        e1.record(stream)
        e1.synchronize()
        out[name] = e0.elapsed_time(e1) / k
    return out


def host_info():
    """The CPU model and the cores this process may use (for the CPU baseline)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0))}


def cpu_baseline(wl, t_slice, min_secs=10.0, sparse_s=0):
    """The oracle (numpy fp64) timed on this host's cores on a bounded sample:
    fwd + bwd + step of each distinct layer shape on t_slice tokens (the full
    step when t_slice >= tokens), repeated until min_secs of CPU work, then
    weighted by how many layers have each shape (GEMM cost is linear in tokens,
    the step is token-free)."""
    from oracle import compact as oc
    from synthetic import bwd_inputs, fwd_inputs
    cores = len(os.sched_getaffinity(0))
    host = host_info()
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threadpool_limits(cores)  # the BLAS uses every core this process may run on
        blas = [d for d in threadpool_info() if d.get("user_api") == "blas"]
        threads = max([d.get("num_threads", 1) for d in blas] or [1])
        host["blas"] = ", ".join(f"{d.get('internal_api')} {d.get('version')} ({d.get('architecture')})" for d in blas)
    except Exception:  # pragma: no cover
        threads = cores
        host["blas"] = "unknown"
    host["blas_threads"] = int(threads)
    counts = {}
    for L in wl.layers:
        counts[(L.n, L.m, L.r)] = counts.get((L.n, L.m, L.r), 0) + 1
    Ts = min(t_slice, wl.tokens)
    inputs = {}
    for (n, m, r) in counts:
        x, W = fwd_inputs(Ts, n, m, wl.dtype, data_seed=1)
        dy, _, _ = bwd_inputs(Ts, n, m, r, wl.dtype, data_seed=1)
        inputs[(n, m, r)] = (x, W, dy)
    t_tok = {k: 0.0 for k in counts}
    t_step = {k: 0.0 for k in counts}
    reps, spent = 0, 0.0
    while reps == 0 or spent < min_secs:
        for (n, m, r), (x, W, dy) in inputs.items():
            t0 = time.perf_counter()
            _, z = oc.ref_fwd(x, W, 1 << 32, r, sparse_s=sparse_s)
            _, G = oc.ref_bwd(dy, z, W)
            t1 = time.perf_counter()
            oc.ref_step(W, G, np.zeros_like(G), np.zeros_like(G), 1 << 32, r, 1, wl.lr, wl.beta1,
                        wl.beta2, wl.eps, wl.alpha, sparse_s=sparse_s)
            t2 = time.perf_counter()
            t_tok[(n, m, r)] += t1 - t0
            t_step[(n, m, r)] += t2 - t1
            spent += t2 - t0
        reps += 1
    total = sum(cnt * (t_tok[k] / reps * wl.tokens / Ts + t_step[k] / reps) for k, cnt in counts.items())
    scaled = "" if Ts == wl.tokens else f", extrapolated linearly in tokens to {wl.tokens}"
    return {
        "value": wl.tokens / total,
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "host": host,
        "sample": (f"numpy fp64 oracle: fwd+bwd+step of each of the {len(counts)} distinct layer "
                   f"shapes at {Ts} tokens, {reps} repetition(s) ({spent:.1f} s){scaled}, "
                   f"weighted by the layer count of each shape ({len(wl.layers)} layers)"),
    }


def model_sweep(args):
    """Peak allocated memory and step time of whole training steps (forward,
    backward, CompActAdam and torch's Adam) of a LLaMA-350M-shaped model in the
    paper's pretraining setup (every block linear layer but o compressed, bf16,
    flash attention, sequences of 256 tokens, vocabulary 32000) against the
    same model uncompressed, over batch sizes: the measurement behind the
    paper's peak-memory-vs-batch figure and its throughput/memory figure, on
    synthetic tokens and random weights."""
    import gc
    import torch
    import paper_2410_15352_amd as cp
    from paper_2410_15352_amd.block import LlamaModel, block_saved_bytes, make_optimizers

    cp.library()
    vocab, d, heads, ffn, layers, seq, alpha = 32000, 1024, 16, 2736, 24, 256, 0.25
    batches = [int(b) for b in args.sweep_batches.split(",")]
    gen = torch.Generator(device="cuda:0").manual_seed(1234)
    for rank in (None, d // 4, d // 8):
        for b in batches:
            rec = {"sweep": "llama-350m-train-step", "rank": rank, "batch": b, "seq": seq, "tokens": b * seq,
                   "data": "synthetic", "dtype": "bf16",
                   "allocated_before_gib": round(torch.cuda.memory_allocated() / 2**30, 3)}
            model = opts = tokens = loss = None
            try:
                model = LlamaModel(vocab, d, heads, ffn, layers, rank=rank, alpha=alpha)
                opts = make_optimizers(model, lr=1e-3, reseed_period=args.reseed_period)
                tokens = torch.randint(0, vocab, (b, seq + 1), device="cuda:0", generator=gen)

                def step():
                    for o in opts:
                        o.zero_grad()
                    loss = model(tokens[:, :-1], tokens[:, 1:])
                    loss.backward()
                    for o in opts:
                        o.step()
                    return loss

                for _ in range(max(1, args.warmup)):
                    step()
                torch.cuda.synchronize()
                torch.cuda.reset_peak_memory_stats()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(args.steps):
                    loss = step()
                e1.record()
                torch.cuda.synchronize()
                ms = e0.elapsed_time(e1) / args.steps
                rec.update(peak_gib=round(torch.cuda.max_memory_allocated() / 2**30, 3), ms_per_step=round(ms, 2),
                           tokens_per_s=round(b * seq / ms * 1e3), loss=round(loss.item(), 4),
                           saved_per_block_gib=round(block_saved_bytes(b, seq, d, heads, ffn, rank=rank) / 2**30, 4))
            except torch.cuda.OutOfMemoryError:
                rec["oom"] = True
            # the last loss holds the autograd graph, whose nodes hold the model
            del model, opts, tokens, loss
            gc.collect()
            torch.cuda.empty_cache()
            print(json.dumps(rec), flush=True)


def compare_blas():
    """dL/dx = dL/do W^T through compact_bwd (the K-tiled staging of W and the
    persistent GEMM) against torch.matmul on the same bf16 operands: T = 65536
    tokens, n = 1024 outputs, K = m from 1024 to 8192 (the dx shapes of the
    LLaMA workloads and beyond).  Event-timed, 10 calls after one warm-up."""
    import torch
    import paper_2410_15352_amd as cp
    cp.library()
    dev = torch.device("cuda:0")
    T, n = 65536, 1024

    def timed(fn, reps=10):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) / reps

    for K in (1024, 2048, 2736, 3072, 4096, 5472, 8192):
        g = torch.Generator(device=dev)
        g.manual_seed(K)
        dy = torch.empty(T, K, device=dev).normal_(0.0, 0.01, generator=g).to(torch.bfloat16)
        W = torch.empty(n, K, device=dev).normal_(0.0, 0.02, generator=g).to(torch.bfloat16)
        Wt = W.t().contiguous()
        dx = torch.empty(T, n, dtype=torch.bfloat16, device=dev)
        ws = torch.zeros(cp.bwd_workspace_bytes(T, n, K, 128), dtype=torch.uint8, device=dev)
        ours = timed(lambda: cp.compact_bwd(dy, W, None, dx, None, ws=ws))
        lib = timed(lambda: torch.matmul(dy, Wt))
        fl = 2.0 * T * n * K
        print(json.dumps({"K": K, "tokens": T, "n": n, "compact_bwd_dx_us": round(ours * 1e3, 1),
                          "compact_bwd_dx_tflops": round(fl / ours / 1e9, 1),
                          "torch_matmul_us": round(lib * 1e3, 1), "torch_matmul_tflops": round(fl / lib / 1e9, 1)}),
              flush=True)
        del dy, W, Wt, dx, ws


def main():
    args = parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU (the library has no "
                                   "collectives; multi-GPU sharding is a design note only); rerun with --gpus 1"}),
              flush=True)
        sys.exit(2)
    if args.model_sweep:
        return model_sweep(args)
    if args.compare_blas:
        return compare_blas()
    import torch
    import paper_2410_15352_amd as cp
    from synthetic import workload

    cp.library()  # fails loudly when the HIP library is missing
    if args.calibrate_copy:
        a = torch.ones(64 << 20, dtype=torch.float32, device="cuda:0")
        b = torch.empty_like(a)
        torch.neg(a, out=b)  # reads 256 MiB, writes 256 MiB
        torch.cuda.synchronize()
        del a, b
    wl = workload(args.workload)
    T = wl.tokens
    print(f"[bench] workload {wl.name}: {len(wl.layers)} layers, {T} tokens; allocating", file=sys.stderr, flush=True)
    model = Model(wl, args.fwd_mode, grouped=not args.no_group, proj=args.proj)
    torch.cuda.synchronize()
    print(f"[bench] warmup {args.warmup} steps", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        model.step(args.reseed_period)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        model.step(args.reseed_period)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    if args.no_phases:
        print(json.dumps({"ms_per_step": ms_per_step, "tokens_per_s": T / (ms_per_step * 1e-3)}), flush=True)
        return
    phases = time_phases(model, torch)
    flops, bytes_ = algorithmic(wl, model.groups)
    fwd_tflops = flops["fwd"] / (phases["fwd"] * 1e-3) / 1e12
    gemm_ms = phases["fwd"] + phases["bwd_dx"] + phases["bwd_ghat"]
    gemm_frac = (flops["fwd"] + flops["dx"] + flops["ghat"]) / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
    upd_gbs = (bytes_["adam"] + bytes_["dec"]) / (phases["step"] * 1e-3) / 1e9

    def phase(bound, work, ms):
        rate = work / (ms * 1e-3)
        if bound == "mfma":
            return {"bound": bound, "achieved": round(rate / 1e12, 1), "unit": "TFLOP/s",
                    "frac": round(rate / 1e12 / PEAK_BF16_TFLOPS, 4)}
        return {"bound": bound, "achieved": round(rate / 1e9, 1), "unit": "GB/s",
                "frac": round(rate / 1e9 / PEAK_HBM_GBS, 4)}

    # each phase against its own bound: the GEMMs against the bf16 MFMA peak,
    # G^ (HBM-bound at r = n/8) and Alg. 3 against the HBM peak
    phase_roofline = {
        "fwd": phase("mfma", flops["fwd"], phases["fwd"]),
        "bwd_dx": phase("mfma", flops["dx"], phases["bwd_dx"]),
        "bwd_ghat": phase("hbm", bytes_["ghat"], phases["bwd_ghat"]),
        "step": phase("hbm", bytes_["adam"] + bytes_["dec"], phases["step"]),
    }

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        rec = json.load(open(TRAFFIC_FILE))
        if rec.get("src_hash") == kernel_source_hash() and rec.get("workload") == wl.name:
            traffic = rec.get("bytes_per_launch")
    nl = len(wl.layers)
    nf = len(model.groups)  # forward launches per step
    roofline = {
        "bound": "mfma", "kernel": "compact_fwd(_group): k_gemm_w4<0> ([y|z] = x [W^T; P^T]^T) with its W^T + P^T staging launch",
        "achieved": round(fwd_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
        "frac": round(fwd_tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
        "flops_per_launch": flops["fwd"] / nf,
        "avg_launch_ms": phases["fwd"] / nf,
    }
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        code = cp.proj_code(args.proj)
        sparse_s = (((code >> 8) & 0xFF) or cp.SPARSE_JL_DEFAULT_S) if (code & 0xFF) == cp.PROJ["sparse-jl"] else 0
        cpu = cpu_baseline(wl, args.cpu_tokens, sparse_s=sparse_s)
    act = [{"layer": L.name, "n": L.n, "r": L.r, "saved_bytes": 2 * T * L.r, "uncompressed_bytes": 2 * T * L.n}
           for L in wl.distinct_shapes()]
    line = {
        "metric": "CompAct linear fwd+bwd+step tokens/s, % bf16 MFMA peak, LLaMA-350M shapes",
        "value": round(T / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.description, "tokens_per_step": T, "layers": nl,
                   "input_groups": ("q,k,v and gate,up share their input (gate,up only when their width is a "
                                    "multiple of 8)") if not args.no_group else "none",
                   "fwd_mode": args.fwd_mode, "projection": args.proj, "parallelism": "single GPU",
                   "activation_buffers": ("one x, y, dL/do, dL/dx per input group" if model.act_bytes else
                                          f"{model.act_sets} sets shared round-robin by the blocks")},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "phases_ms": {k: round(v, 4) for k, v in phases.items()},
        "gemm_phases_mfma_frac": round(gemm_frac, 4),
        "update_phase_hbm_GBs": round(upd_gbs, 1),
        "update_phase_hbm_frac": round(upd_gbs / PEAK_HBM_GBS, 4),
        "phase_roofline": phase_roofline,
        "activation_bytes_per_layer": act,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
