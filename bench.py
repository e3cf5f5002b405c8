#!/usr/bin/env python3
"""Benchmark of slice-wise causal linear attention, forward + backward, on one GPU.

One step = slim_fwd + slim_bwd over one batch of the L = 32768 workload
(B=4, H=8, d=64, M=256, bf16 inputs, FAVOR+), inputs resident in device
memory; the backward gets the forward's outputs Y, logD (row normalisers),
key shift and context.  Prints one JSON line with throughput (tokens/s = B*L / step time),
a roofline entry for the dominant kernel, the fp64 CPU oracle timed on the
whole batch, and, unless switched off:

* sweep: every slice length C of the headline workload, with the in-slice
  block the kernels ran, the executed-work roofline fraction of the reverse
  walk, peak device memory beyond inputs and outputs, the lower bound "L/B"
  (the same measured on an input of length C) and the L2-relative gradient
  error against the oracle; then the same slice lengths with each slice
  evaluated as one masked quadratic form (the within-slice quadratic mode),
  and, up to C = 4096, with every row's state written out (the explicit
  prefix-sum mode, "PS");
* configs: the other workloads (tiny fp32 exactness check, B8 H8 L4096,
  L=262144 long context, the six-layer ReLU stack run forward r=1..6 then
  backward r=6..1), each with time, roofline and parity on sampled heads,
  and the headline shape in float32 (explicit prefix-sum mode);
* peak memory versus L at fixed C;
* the paper's own feature map (element-wise square, M = d = 64, W = I) at
  its per-layer shapes.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--C 64] [--quick]
"""

from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "causal FAVOR+ fwd+bwd tokens/sec at L=32k, d=64, M=256; peak mem vs slice C"
PEAK_BF16_FLOPS = 2.5e15  # MI355X dense bf16 matrix-core peak
PEAK_FP32_FLOPS = 157.3e12  # fp32 matrix / vector peak
TILE_ROWS = 32  # rows per tile of the kernels: the block of the in-slice evaluation
KIND_LABEL = {"favor+": "causal FAVOR+", "relu": "causal ReLU-feature", "square": "causal square-feature"}


def flops_per_token_head(d: int, M: int, c: int):
    """Flops (2 per multiply-add) per token and head, for an in-slice block
    of c rows evaluated as a causal quadratic form (c + 1 per row, the
    causal half), the state carried between blocks:
      fwd: 4dM (Q, K logits) + 4M(d+1) (state read + update) + (M+d+1)(c+1)
      bwd: 24dM + 10M + (3M+3d+1)(c+1) (recompute, downdate, gradients, chain
           rule through the feature map, dW)
    With c = C this is the algorithmic count of the method with the whole
    slice as one quadratic form; with c = min(C, 32) it is the work the
    kernels execute (their in-slice block is a 32-row tile)."""
    fwd = 4 * d * M + 4 * M * (d + 1) + (M + d + 1) * (c + 1)
    bwd = 24 * d * M + 10 * M + (3 * M + 3 * d + 1) * (c + 1)
    return fwd, bwd


def walk_takes_forward_outputs(dtype: str, M: int, kind: str) -> bool:
    """Whether the reverse walk, given the forward's Y and logD (as the
    benchmark's backward is), recomputes neither N nor D: the 8-wave walk
    (bf16, M in {128, 256}, FAVOR+ or ReLU)."""
    return dtype == "bf16" and M in (128, 256) and kind in ("favor+", "relu")


def executed_bwd_flops(d: int, M: int, c: int, given: bool) -> int:
    """The reverse walk's executed flops per token-head with its c-row block;
    given the forward's Y and logD it skips the numerators and denominators
    N = Q~[S|z] + A[V|1] of the recomputed block: 2M(d+1) + (d+1)(c+1)."""
    b = flops_per_token_head(d, M, c)[1]
    return b - (2 * M * (d + 1) + (d + 1) * (c + 1)) if given else b


def kernel_sources_sha() -> str:
    """Hash of the sources the attention kernels are compiled from (every
    file under csrc/ but the model step's own translation unit, which they
    do not include): traffic counters taken on other sources are not used."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2012_11346_amd", "csrc", "*"))):
        if os.path.basename(f) == "slim_model.hip":
            continue
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str):
    """HBM traffic of a kernel from the committed counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except Exception:
        return None
    k = rec.get("kernels", {}).get(kernel)
    if k is None or rec.get("sources_sha") != kernel_sources_sha():
        return None
    return k.get("bytes_per_launch")


def bwd_walk_name(dtype: str, M: int, kind: str) -> str:
    """The reverse-walk kernel the library launches: the 8-wave form for bf16
    problems with 32 or 64 features per wave, else the 4-wave form."""
    forced4 = os.environ.get("SLIM_BWD_WAVES") == "4"
    return "bwd_walk8_kernel" if (dtype == "bf16" and M // 4 in (32, 64) and kind != "square" and not forced4) \
        else "bwd_walk_kernel"


def threads_used() -> int:
    try:
        from threadpoolctl import threadpool_info

        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:
        return os.cpu_count() or 1


def mask_w(x):
    """W the oracle takes the ReLU derivative's decisions with: the bf16
    split hi + lo the kernels form the logits from (bf16), else W."""
    import torch

    if x["Q"].dtype != torch.bfloat16:
        return None
    W = x["W"].float()
    hi = W.to(torch.bfloat16).float()
    lo = (W - hi).to(torch.bfloat16).float()
    return hi.double().numpy() + lo.double().numpy()


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--C", type=int, default=64)
    ap.add_argument("--no-sweep", action="store_true", help="skip the slice-length sweep")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workloads and memory-vs-L")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle timing and the parity checks")
    ap.add_argument("--quick", action="store_true", help="headline only (= --no-sweep --no-configs --no-cpu --no-model)")
    ap.add_argument("--no-model", action="store_true", help="skip the s-layer language model (Algorithm 1 over eqs. 5-10)")
    ap.add_argument("--model-only", action="store_true", help="only the s-layer language model section")
    ap.add_argument("--model-seeds", type=int, default=1, help="seeds of the model's gradient discrepancy")
    ap.add_argument("--model-configs", default="I,II,III,IV", help="model configurations to run (comma list)")
    ap.add_argument("--model-C", default="", help="slice lengths of the model section (comma list; default "
                    "64, 256, 1024, 4096 below L, and L)")
    ap.add_argument("--sweep-steps", type=int, default=5)
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="only copy a device buffer of this many MiB (calibration of memory counters) and exit")
    args = ap.parse_args()
    if args.quick:
        args.no_sweep = args.no_configs = args.no_cpu = args.no_model = True
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path runs on a single "
              "MI355X; sharded, GPUs would split the heads and batch rows and sum dW with one all-reduce)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2012_11346_amd import slim
    from synth import make_inputs, workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda", 0)
    if args.copy_mib > 0:
        # a plain copy of known size: reads and writes copy_mib MiB once per launch
        n = args.copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 3}), flush=True)
        return

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    mk = lambda: torch.cuda.Event(enable_timing=True)
    stream = torch.cuda.current_stream()

    class Layer:
        """Device inputs, outputs and workspaces of one attention op."""

        def __init__(self, x, C, kind, within="iter"):
            self.kind = kind
            self.C = C
            self.within = within
            self.x = x
            self.Q, self.K, self.V, self.dY = (x[k].to(dev) for k in ("Q", "K", "V", "dY"))
            self.W = x["W"].to(dev)
            B, H, L, d = self.Q.shape
            M = self.W.shape[0]
            self.shape = (B, H, L, d, M)
            torch.cuda.synchronize()

        def alloc(self):
            B, H, L, d, M = self.shape
            p = slim.problem(B, H, L, d, M, self.C, self.Q.dtype, self.kind, within=self.within)
            self.p = p
            self.Y = torch.empty_like(self.Q)
            # the row normalisers (tile-walk mode), an output like Y
            self.lD = torch.empty((B, H, L), dtype=torch.float32, device=dev) if self.within == "iter" else None
            self.st = torch.empty((B, H, M, d + 1), dtype=torch.float32, device=dev)
            self.ks = torch.empty((B, H), dtype=torch.float32, device=dev) if self.kind == "favor+" else None
            self.dQ, self.dK, self.dV = (torch.empty_like(self.Q) for _ in range(3))
            self.dW = torch.empty((M, d), dtype=torch.float32, device=dev)
            self.out_bytes = sum(t.numel() * t.element_size() for t in
                                 (self.Y, self.st, self.dQ, self.dK, self.dV, self.dW) +
                                 tuple(t for t in (self.ks, self.lD) if t is not None))
            self.wsf = torch.empty(max(1, slim.workspace_bytes(p, slim.PHASE_FWD)), dtype=torch.uint8, device=dev)
            self.wsb = torch.empty(max(1, slim.workspace_bytes(p, slim.PHASE_BWD)), dtype=torch.uint8, device=dev)
            n_ctx = slim.context_bytes(p)
            self.ctx = torch.empty(n_ctx // 4, dtype=torch.float32, device=dev) if n_ctx > 0 else None
            self.ws_bytes = self.wsf.numel() + self.wsb.numel() + n_ctx
            return self

        def free(self):
            for n in ("Y", "lD", "st", "ks", "dQ", "dK", "dV", "dW", "wsf", "wsb", "ctx"):
                setattr(self, n, None)

        def fwd(self):
            slim.fwd(self.Q, self.K, self.V, self.W, self.C, self.kind, ws=self.wsf, Y=self.Y, state_out=self.st,
                     kshift_out=self.ks, ctx=self.ctx, within=self.within, logD=self.lD)

        def bwd(self, dY=None):
            slim.bwd(self.Q, self.K, self.V, self.W, self.dY if dY is None else dY, self.C, self.ks, self.kind,
                     ws=self.wsb, dQ=self.dQ, dK=self.dK, dV=self.dV, dW=self.dW, ctx=self.ctx, within=self.within,
                     Y=self.Y, logD=self.lD)

    def run_step(layers):
        """forward r = 1..n, then backward r = n..1"""
        for ly in layers:
            ly.fwd()
        for ly in reversed(layers):
            ly.bwd()

    def timed(layers, steps, warmup, breakdown=False):
        """warmup + `steps` timed steps bracketed by two events.  Inside the
        timed region only the reverse walks carry events (the library
        records them around that kernel's launch: its duration for the
        roofline); with `breakdown`, a second pass of the same number of
        steps times the calls and the forward walk separately, so that its
        events do not add to the timed steps."""
        torch.cuda.synchronize()
        pre = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        for ly in layers:
            ly.alloc()
        for _ in range(warmup):
            run_step(layers)
        n = len(layers)
        t0, t1 = mk(), mk()
        wb = [[(mk(), mk()) for _ in range(n)] for _ in range(steps)]
        for e in [t0, t1] + [x_ for row in wb for pair in row for x_ in pair]:
            e.record(stream)  # create every event before the timed region
        torch.cuda.synchronize()
        t0.record(stream)
        for i in range(steps):
            for ly in layers:
                ly.fwd()
            for k, ly in enumerate(reversed(layers)):
                slim.time_walk(slim.PHASE_BWD, wb[i][k][0], wb[i][k][1])
                ly.bwd()
        t1.record(stream)
        torch.cuda.synchronize()
        total_ms = t0.elapsed_time(t1)
        walk_ms = sum(a.elapsed_time(b) for row in wb for a, b in row) / (steps * n)
        peak = torch.cuda.max_memory_allocated()
        out_bytes = sum(ly.out_bytes for ly in layers)
        r = dict(ms=total_ms / steps, bwd_walk_ms=walk_ms, peak=peak, extra=peak - pre - out_bytes,
                 ws=sum(ly.ws_bytes for ly in layers), segments=slim.num_segments(layers[0].p))
        if breakdown:
            bd = [[mk() for _ in range(5)] for _ in range(steps)]
            for e5 in bd:
                for e in e5:
                    e.record(stream)
            torch.cuda.synchronize()
            for e in bd:
                e[0].record(stream)
                slim.time_walk(slim.PHASE_FWD, e[1], e[2])
                for ly in layers:
                    ly.fwd()
                e[3].record(stream)
                for ly in reversed(layers):
                    ly.bwd()
                e[4].record(stream)
            torch.cuda.synchronize()
            avg = lambda i, j: sum(e[i].elapsed_time(e[j]) for e in bd) / steps
            r.update(fwd_ms=avg(0, 3), bwd_ms=avg(3, 4), fwd_walk_ms=avg(1, 2))
        return r

    def roofline(kernel, dtype, units, flops_per_unit, launch_ms):
        peak = PEAK_BF16_FLOPS if dtype == "bf16" else PEAK_FP32_FLOPS
        achieved = units * flops_per_unit / (launch_ms / 1e3)
        return {"kernel": kernel, "bound": "mfma", "achieved": achieved / 1e12, "peak": peak / 1e12,
                "unit": "TFLOP/s", "frac": achieved / peak, "flops_per_token_head": flops_per_unit,
                "token_heads_per_launch": units, "launch_ms": launch_ms}

    def rel_errors(a, ref):
        a = np.asarray(a, dtype=np.float64)
        ref = np.asarray(ref, dtype=np.float64)
        return {"max_rel": float(np.max(np.abs(a - ref)) / np.max(np.abs(ref))),
                "l2_rel": float(np.linalg.norm(a - ref) / np.linalg.norm(ref))}

    def h64(t):
        return t.detach().double().cpu().numpy()

    def oracle_heads(x, heads, kind):
        """The fp64 oracle (Algorithm 1 with the in-slice quadratic form; the
        exact result does not depend on the slice length) on sampled heads."""
        import oracle as O

        pick = lambda t: np.stack([h64(t[b, h]) for b, h in heads])[None]
        Q, K, V, dY = (pick(x[k]) for k in ("Q", "K", "V", "dY"))
        W = h64(x["W"])
        Y, st = O.slim_forward(Q, K, V, W, 256, kind, within="quadratic")
        g = O.slim_backward(Q, K, V, W, dY, 256, kind, st, within="quadratic", mask_W=mask_w(x))
        return {"Y": Y, "dQ": g[0], "dK": g[1], "dV": g[2], "dW": g[3]}

    def parity(layer, heads, ref):
        """errors of the last run's outputs on the sampled heads; dW from a
        second backward with dY zero outside them (isolates their share)"""
        pick = lambda t: np.stack([h64(t[b, h]) for b, h in heads])[None]
        out = {n: rel_errors(pick(getattr(layer, n)), ref[n]) for n in ("Y", "dQ", "dK", "dV")}
        mask = torch.zeros(layer.dY.shape[:2], dtype=torch.bool, device=dev)
        for b, h in heads:
            mask[b, h] = True
        dYm = torch.where(mask[:, :, None, None], layer.dY, torch.zeros_like(layer.dY))
        layer.bwd(dYm)
        torch.cuda.synchronize()
        out["dW"] = rel_errors(h64(layer.dW), ref["dW"])
        return out

    if args.model_only:
        print(json.dumps({"model": model_section(args, dev, log)}), flush=True)
        return

    # ------------------------------------------------------------ headline
    wl = workload("sweep_32k")
    B, H, L, d, M, kind = wl.B, wl.H, wl.L, wl.d, wl.M, wl.kind
    C = args.C
    t0 = time.perf_counter()
    x = make_inputs(wl)
    log(f"inputs generated in {time.perf_counter() - t0:.1f}s")
    head = Layer(x, C, kind)
    log(f"timing C={C}: warmup {args.warmup}, steps {args.steps}")
    r = timed([head], args.steps, args.warmup, breakdown=True)
    tokens = B * L
    units = B * H * L  # token-heads per launch of either walk
    value = tokens / (r["ms"] / 1e3)
    alg_f, alg_b = flops_per_token_head(d, M, C)
    blk = min(C, TILE_ROWS)
    given = walk_takes_forward_outputs(wl.dtype, M, kind)
    ex_b = executed_bwd_flops(d, M, blk, given)
    dominant = bwd_walk_name(wl.dtype, M, kind)
    rl = roofline(dominant, wl.dtype, units, alg_b, r["bwd_walk_ms"])
    rl["traffic"] = load_traffic(dominant)
    rl["flops_basis"] = (f"algorithmic count with the slice as one quadratic form (c = C = {C}); the kernel "
                         f"executes {ex_b} flops per token-head with its {blk}-row in-slice block"
                         + (" (N and D from the forward's Y and logD, not recomputed)" if given else "")
                         + f", frac {units * ex_b / (r['bwd_walk_ms'] / 1e3) / PEAK_BF16_FLOPS:.3f} on that count")
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {KIND_LABEL[kind]} attention fwd+bwd, B={B} H={H} L={L} d={d} M={M}, "
                        f"bf16 inputs with fp32 accumulation, float32 W, slice length C={C}",
            "B": B, "H": H, "L": L, "d": d, "M": M, "C": C, "kind": kind,
            "segments_per_head": r["segments"], "in_slice_block": blk,
        },
        "fwd_ms": r["fwd_ms"],
        "bwd_ms": r["bwd_ms"],
        "fwd_walk_ms": r["fwd_walk_ms"],
        "bwd_walk_ms": r["bwd_walk_ms"],
        "roofline": rl,
        "mfma_frac_fwd_bwd": (alg_f + alg_b) * units / (r["ms"] / 1e3) / PEAK_BF16_FLOPS,
        "peak_mem": {"peak_bytes": r["peak"], "beyond_io_bytes": r["extra"], "workspace_and_context": r["ws"]},
    }
    log(f"C={C}: {r['ms']:.3f} ms/step (fwd {r['fwd_ms']:.3f}, bwd {r['bwd_ms']:.3f}; walks "
        f"{r['fwd_walk_ms']:.3f} / {r['bwd_walk_ms']:.3f}), {value:.3e} tokens/s")
    head.free()
    torch.cuda.empty_cache()

    ref = None
    sample = [(0, 0), (3, 7)]
    if not args.no_cpu:
        log("oracle on two sampled heads")
        ref = oracle_heads(x, sample, kind)

    # ------------------------------------------------------------ slice-length sweep
    if not args.no_sweep:
        sweep = []
        for Cs in wl.C:
            ly = Layer(x, Cs, kind)
            rs = timed([ly], args.sweep_steps, 5)
            blk_s = min(Cs, TILE_ROWS)
            exb = executed_bwd_flops(d, M, blk_s, walk_takes_forward_outputs(wl.dtype, M, kind))
            algf, algb = flops_per_token_head(d, M, Cs)
            rec = {"C": Cs, "in_slice_block": blk_s, "tokens_per_s": tokens / (rs["ms"] / 1e3),
                   "ms_per_step": rs["ms"], "bwd_walk_ms": rs["bwd_walk_ms"],
                   "roofline_executed": roofline(dominant, "bf16", units, exb, rs["bwd_walk_ms"]),
                   "algorithmic_flops_per_token_head_at_C": algf + algb,
                   "peak_bytes": rs["peak"], "beyond_io_bytes": rs["extra"]}
            if ref is not None:
                e = parity(ly, sample, ref)
                rec["grad_l2_rel"] = {k: v["l2_rel"] for k, v in e.items() if k != "Y"}
                rec["max_rel"] = {k: v["max_rel"] for k, v in e.items()}
            ly.free()
            del ly
            torch.cuda.empty_cache()
            # lower bound "L/B": the same method on an input of length C only
            xs = {k: (v[:, :, :Cs].contiguous() if k != "W" else v) for k, v in x.items()}
            lb = Layer(xs, Cs, kind)
            rb = timed([lb], 1, 1)
            rec["lower_bound_beyond_io_bytes"] = rb["extra"]
            lb.free()
            del lb, xs
            torch.cuda.empty_cache()
            sweep.append(rec)
            log(f"sweep C={Cs} (block {blk_s}): {rs['ms']:.3f} ms/step, beyond inputs/outputs "
                f"{rs['extra'] / 2**20:.1f} MiB (L/B {rec['lower_bound_beyond_io_bytes'] / 2**20:.1f} MiB)")
        out["sweep"] = sweep
        # the same sweep with each slice evaluated as one masked quadratic form
        # (slices one after another, the slice's tiles in parallel)
        qsweep = []
        for Cs in wl.C:
            ly = Layer(x, Cs, kind, within="quadratic")
            steps_q = args.sweep_steps if Cs <= 4096 else 2
            rs = timed([ly], steps_q, 2)
            algf, algb = flops_per_token_head(d, M, Cs)
            rec = {"C": Cs, "in_slice_block": Cs, "tokens_per_s": tokens / (rs["ms"] / 1e3), "ms_per_step": rs["ms"],
                   "steps": steps_q, "bwd_slices_ms": rs["bwd_walk_ms"],
                   "mfma_frac_algorithmic": (algf + algb) * units / (rs["ms"] / 1e3) / PEAK_BF16_FLOPS,
                   "peak_bytes": rs["peak"], "beyond_io_bytes": rs["extra"]}
            if ref is not None:
                e = parity(ly, sample, ref)
                rec["grad_l2_rel"] = {k: v["l2_rel"] for k, v in e.items() if k != "Y"}
                rec["max_rel"] = {k: v["max_rel"] for k, v in e.items()}
            ly.free()
            del ly
            torch.cuda.empty_cache()
            qsweep.append(rec)
            log(f"quadratic sweep C={Cs}: {rs['ms']:.3f} ms/step, beyond inputs/outputs {rs['extra'] / 2**20:.1f} MiB")
        out["sweep_quadratic"] = qsweep
        # the explicit prefix-sum mode ("PS"): every row's state of a slice
        # written out (C M (d + 1) floats per head, twice in the backward);
        # C = 32768 would hold 2 x 70 GB of states and is left out
        psweep = []
        for Cs in [c for c in wl.C if c <= 4096]:
            ly = Layer(x, Cs, kind, within="ps")
            rs = timed([ly], 2, 1)
            rec = {"C": Cs, "tokens_per_s": tokens / (rs["ms"] / 1e3), "ms_per_step": rs["ms"], "steps": 2,
                   "peak_bytes": rs["peak"], "beyond_io_bytes": rs["extra"], "workspace_bytes": rs["ws"]}
            if ref is not None:
                e = parity(ly, sample, ref)
                rec["grad_l2_rel"] = {k: v["l2_rel"] for k, v in e.items() if k != "Y"}
                rec["max_rel"] = {k: v["max_rel"] for k, v in e.items()}
            ly.free()
            del ly
            torch.cuda.empty_cache()
            psweep.append(rec)
            log(f"PS sweep C={Cs}: {rs['ms']:.3f} ms/step, beyond inputs/outputs {rs['extra'] / 2**20:.1f} MiB")
        out["sweep_ps"] = psweep

    # ------------------------------------------------------------ headline parity and oracle timing
    if not args.no_cpu:
        import oracle as O

        ly = Layer(x, C, kind)
        timed([ly], 1, 1)
        out["parity"] = {"unrounded_W": parity(ly, sample, ref)}
        ly.free()
        del ly
        torch.cuda.empty_cache()
        # the same with a bf16-representable W
        xr = dict(x)
        xr["W"] = make_inputs(wl, tensors=("W",), round_w=True)["W"]
        lr = Layer(xr, C, kind)
        timed([lr], 1, 1)
        refr = oracle_heads(xr, sample[:1], kind)
        out["parity"]["rounded_W"] = parity(lr, sample[:1], refr)
        lr.free()
        del lr, xr
        torch.cuda.empty_cache()
        log("timing the fp64 oracle on the host (whole batch)")
        t0 = time.perf_counter()
        Yo, st = O.slim_forward(x["Q"], x["K"], x["V"], x["W"], C, kind, within="quadratic")
        O.slim_backward(x["Q"], x["K"], x["V"], x["W"], x["dY"], C, kind, st, within="quadratic")
        t = time.perf_counter() - t0
        out["cpu_baseline"] = {
            "value": B * L / t, "unit": "tokens/s", "cores": threads_used(), "kind": "oracle",
            "sample": f"the whole workload batch (B={B}, H={H}, L={L}), fp64 Algorithm 1 forward + backward, "
                      f"{kind}, in-slice quadratic form at C={C}; {t:.1f} s on the host",
            "seconds": t, "host_cpus": os.cpu_count()}
    del x
    torch.cuda.empty_cache()

    # ------------------------------------------------------------ other workloads
    if not args.no_configs:
        configs = []
        for name, heads in (("tiny_exact", [(0, 0)]), ("mid_bf16", [(7, 7)]), ("long_256k", [(0, 5)]),
                            ("relu_stack", [(1, 11)])):
            w2 = workload(name)
            Cw = w2.C[0]
            t0 = time.perf_counter()
            xs = [make_inputs(w2, layer=k) for k in range(w2.layers)]
            layers = [Layer(xk, Cw, w2.kind) for xk in xs]
            log(f"{name}: inputs in {time.perf_counter() - t0:.1f}s")
            steps = 5 if w2.L * w2.B * w2.H * w2.layers >= (1 << 21) else 20
            rc = timed(layers, steps, 5)
            u = w2.B * w2.H * w2.L
            blk_w = min(Cw, TILE_ROWS)
            exb = executed_bwd_flops(w2.d, w2.M, blk_w, walk_takes_forward_outputs(w2.dtype, w2.M, w2.kind))
            algf, algb = flops_per_token_head(w2.d, w2.M, Cw)
            kname = bwd_walk_name(w2.dtype, w2.M, w2.kind)
            rec = {"workload": f"{name}: {KIND_LABEL[w2.kind]}, {w2.layers} layer(s) x (B={w2.B} H={w2.H} L={w2.L} "
                               f"d={w2.d} M={w2.M}), {w2.dtype}, C={Cw}"
                               + (", forward r=1..6 then backward r=6..1" if w2.layers > 1 else ""),
                   "C": Cw, "in_slice_block": blk_w, "ms_per_step": rc["ms"],
                   "tokens_per_s": w2.B * w2.L * w2.layers / (rc["ms"] / 1e3),
                   "tokens_counted": "B*L per layer" if w2.layers > 1 else "B*L",
                   "roofline": roofline(kname, w2.dtype, u, algb, rc["bwd_walk_ms"]),
                   "roofline_executed": roofline(kname, w2.dtype, u, exb, rc["bwd_walk_ms"]),
                   "peak_bytes": rc["peak"], "beyond_io_bytes": rc["extra"], "segments_per_head": rc["segments"]}
            if not args.no_cpu:
                # the first layer (its backward runs last in a step) on a sampled head
                rec["parity_layer1"] = parity(layers[0], heads, oracle_heads(xs[0], heads, w2.kind))
            configs.append(rec)
            log(f"{name}: {rc['ms']:.3f} ms/step, {rec['tokens_per_s']:.3e} tokens/s, reverse walk frac "
                f"{rec['roofline']['frac']:.3f}")
            for ly in layers:
                ly.free()
            del layers, xs
            torch.cuda.empty_cache()
        # the headline shape in float32: of the three within-slice modes only
        # the explicit prefix-sum one takes float32 with d M > 4096
        w32 = workload("sweep_32k").with_(name="sweep_32k_f32", dtype="f32")
        x32 = make_inputs(w32)
        ly = Layer(x32, 64, w32.kind, within="ps")
        rc = timed([ly], 2, 1)
        rec = {"workload": f"sweep_32k_f32: {KIND_LABEL[w32.kind]}, B={w32.B} H={w32.H} L={w32.L} d={w32.d} M={w32.M}, "
                           "float32, C=64, explicit prefix-sum within-slice mode",
               "C": 64, "ms_per_step": rc["ms"], "tokens_per_s": w32.B * w32.L / (rc["ms"] / 1e3),
               "peak_bytes": rc["peak"], "beyond_io_bytes": rc["extra"]}
        if not args.no_cpu:
            rec["parity_sampled_head"] = parity(ly, [(2, 5)], oracle_heads(x32, [(2, 5)], w32.kind))
        configs.append(rec)
        log(f"sweep_32k_f32 (PS mode): {rc['ms']:.3f} ms/step")
        ly.free()
        del ly, x32
        torch.cuda.empty_cache()
        out["configs"] = configs

        # peak memory beyond inputs and outputs versus L at fixed C
        w4 = workload("long_256k")
        x4 = make_inputs(w4, tensors=("Q", "K", "V", "dY", "W"))
        mem = []
        for Ls in (4096, 32768, 262144):
            xs = {k: (v[:, :, :Ls].contiguous() if k != "W" else v) for k, v in x4.items()}
            ly = Layer(xs, 512, w4.kind)
            rm = timed([ly], 1, 1)
            mem.append({"L": Ls, "beyond_io_bytes": rm["extra"], "workspace_and_context": rm["ws"]})
            ly.free()
            del ly, xs
            torch.cuda.empty_cache()
        out["peak_mem_vs_L"] = {"B": w4.B, "H": w4.H, "d": w4.d, "M": w4.M, "C": 512, "rows": mem}
        del x4
        log("memory vs L: " + ", ".join(f"L={m['L']}: {m['beyond_io_bytes'] / 2**20:.1f} MiB" for m in mem))

        # the paper's feature map at its per-layer shapes (configurations I-IV)
        from synth import Workload

        sq = []
        for Ls, Hs in ((512, 4), (1024, 8), (4096, 16), (16384, 16)):
            ws = Workload(f"square_{Ls}", 700 + Hs, 1, Hs, Ls, 64, 64, (64,), "bf16", "square")
            xs = make_inputs(ws)
            xs["W"] = torch.eye(64, dtype=torch.float32)
            ly = Layer(xs, 64, "square")
            rq = timed([ly], 20, 5)
            u = Hs * Ls
            f_, b_ = flops_per_token_head(64, 64, 64)
            sq.append({"L": Ls, "H": Hs, "B": 1, "d": 64, "M": 64, "C": 64, "ms_per_step": rq["ms"],
                       "tokens_per_s": Ls / (rq["ms"] / 1e3),
                       "roofline": roofline("bwd_walk_kernel", "bf16", u, b_, rq["bwd_walk_ms"])})
            ly.free()
            del ly, xs
            torch.cuda.empty_cache()
        out["square_paper_shapes"] = sq
        log("square map: " + ", ".join(f"L={s['L']} H={s['H']}: {s['tokens_per_s']:.3e} tok/s" for s in sq))

    if not args.no_model:
        out["model"] = model_section(args, dev, log)

    print(json.dumps(out), flush=True)


def model_flops(cfg, C):
    """Algorithmic flops of one step of Algorithm 1 over the model (2 per
    multiply-add): the forward, and in the backward the recomputation plus
    twice the forward's products, so four times the forward's GEMMs
    (Q/K/V, FFN, logits) and, per head, the attention's forward three times
    (forward, the slice's own sum, recomputation) and its backward once, with
    the in-slice block of TILE_ROWS rows the attention kernels execute."""
    D, F, V, s, L, B = cfg.D, cfg.F, cfg.vocab, cfg.s, cfg.L, cfg.B
    gemm = 2 * (3 * D * D + 2 * D * F) * s + 2 * D * V
    af, ab = flops_per_token_head(64, 64, min(C, L, TILE_ROWS))
    return B * L * (4 * gemm + s * cfg.k * (3 * af + ab))


def model_section(args, dev, log):
    """The paper's language-model experiment (Sec. 4, configurations I-IV:
    s = 3 layers, d_ff = 4 d_model, 256-symbol alphabet, B = 1, random
    initialisation, random byte strings): time and device memory of one
    step of Algorithm 1 per slice length C, the lower bound "L/B" (the same
    step on an input of length C), and the relative gradient discrepancy
    ||g_C - g_full|| / ||g_full|| against the one-slice step (C = L) and,
    where the host can afford it, against the fp64 oracle."""
    import numpy as np
    import torch

    from paper_2012_11346_amd import slim
    from synth import MODEL_CONFIGS, make_model, make_tokens

    stream = torch.cuda.current_stream()
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def step(cfg, P, tok, C, steps, warmup):
        """median-free timing: warmup, then `steps` steps between two events;
        returns (ms, peak bytes beyond parameters/gradients/tokens, workspace
        bytes, loss, grads)"""
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        pre = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        m = slim.model_desc(cfg.B, tok.shape[1], cfg.D, cfg.s, cfg.vocab, cfg.F, C)
        ws = torch.empty(slim.model_workspace_bytes(m), dtype=torch.uint8, device=dev)
        grads = {k: torch.empty_like(v) for k, v in P.items()}
        loss = torch.empty(1, dtype=torch.float32, device=dev)
        io = sum(g.numel() * 4 for g in grads.values()) + 4
        for _ in range(warmup):
            slim.model_step(P, tok, C, ws=ws, grads=grads, loss=loss)
        a, b = mk(), mk()
        a.record(stream)
        for _ in range(steps):
            slim.model_step(P, tok, C, ws=ws, grads=grads, loss=loss)
        b.record(stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        extra = torch.cuda.max_memory_allocated() - pre - io
        return ms, extra, ws.numel(), float(loss.item()), grads

    def disc(g, ref):
        num = sum(float(torch.sum((g[k].double() - ref[k].double()) ** 2)) for k in ref)
        den = sum(float(torch.sum(ref[k].double() ** 2)) for k in ref)
        return (num / den) ** 0.5

    rows = []
    for name in args.model_configs.split(","):
        cfg = MODEL_CONFIGS[name]
        Cs = [c for c in (64, 256, 1024, 4096) if c < cfg.L] + [cfg.L]
        if args.model_C:
            Cs = sorted({min(int(c), cfg.L) for c in args.model_C.split(",")} | {cfg.L})
        steps = 5 if cfg.L * cfg.D <= (1 << 22) else 2
        for seed in range(args.model_seeds):
            P = {k: v.to(dev) for k, v in make_model(cfg, seed=seed).items()}
            tok = make_tokens(cfg, seed=seed).to(dev)
            ms_f, ex_f, ws_f, loss_f, g_full = step(cfg, P, tok, cfg.L, steps, 1)
            g_full = {k: v.clone() for k, v in g_full.items()}
            ref64 = None
            if cfg.L * cfg.D <= (1 << 19) and not args.no_cpu:
                import oracle as O

                t0 = time.perf_counter()
                lo, go = O.model_full({k: v.cpu() for k, v in P.items()}, tok.cpu())
                ref64 = {k: torch.from_numpy(v) for k, v in go.items()}
                log(f"model {name}: fp64 oracle in {time.perf_counter() - t0:.1f}s")
            for C in Cs:
                ms, extra, wsb, loss, g = (ms_f, ex_f, ws_f, loss_f, g_full) if C == cfg.L else step(cfg, P, tok, C, steps, 1)
                rec = {"config": name, "L": cfg.L, "d_model": cfg.D, "s": cfg.s, "heads": cfg.k, "d_ff": cfg.F,
                       "vocab": cfg.vocab, "B": cfg.B, "C": C, "seed": seed, "loss": loss,
                       "grad_discrepancy_vs_C_eq_L": disc(g, g_full)}
                if ref64 is not None:
                    rec["grad_discrepancy_vs_fp64_oracle"] = disc({k: v.cpu() for k, v in g.items()}, ref64)
                if seed == 0:
                    fl = model_flops(cfg, C)
                    rec.update(ms_per_step=ms, tokens_per_s=cfg.B * cfg.L / (ms / 1e3), flops=fl,
                               fp32_frac=fl / (ms / 1e3) / PEAK_FP32_FLOPS, beyond_io_bytes=extra, workspace_bytes=wsb)
                    if C < cfg.L:  # lower bound "L/B": the same step on an input of length C
                        _, lb, _, _, _ = step(cfg, P, tok[:, :C].contiguous(), C, 1, 1)
                        rec["lower_bound_beyond_io_bytes"] = lb
                rows.append(rec)
                log(f"model {name} C={C} seed={seed}: " + (f"{ms:.2f} ms/step, " if seed == 0 else "")
                    + f"discrepancy {rec['grad_discrepancy_vs_C_eq_L']:.2e}"
                    + (f" (fp64: {rec['grad_discrepancy_vs_fp64_oracle']:.2e})" if ref64 is not None else "")
                    + (f", beyond io {extra / 2**20:.0f} MiB" if seed == 0 else ""))
            del P, tok, g_full, ref64
            torch.cuda.empty_cache()
    return {"workload": "s-layer Performer language model (square map, M = d = 64), float32, Algorithm 1; "
                        "configurations I-IV (L, d_model) = (512, 256), (1024, 512), (4096, 1024), (16384, 1024)",
            "rows": rows}


if __name__ == "__main__":
    main()
