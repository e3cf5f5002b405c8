#!/usr/bin/env python3
"""Benchmark of slice-wise causal FAVOR+ attention, forward + backward, on one GPU.

One step = slim_fwd + slim_bwd over one batch of the L = 32768 workload
(B=4, H=8, d=64, M=256, bf16 inputs, FAVOR+), inputs resident in device memory.
Prints one JSON line with throughput (tokens/s = B*L / step time), a roofline
entry for the dominant kernel, the fp64 CPU oracle timed on a bounded sample,
and a slice-length sweep with peak device memory per C.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--C 64] [--no-sweep] [--no-cpu]
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
PEAK_HBM_BYTES = 8.0e12
TILE_ROWS = 32  # rows per tile of the kernels (block of the in-slice evaluation)


def algo_flops_per_token_head(d: int, M: int, C: int, tile: int = TILE_ROWS):
    """Algorithmic flops (2 per multiply-add) per token and head.

    The in-slice prefix sum is evaluated block-iteratively with blocks of
    c = min(C, tile) rows; inside a block the causal quadratic form costs half
    of the c x c products (c + 1 per row).
      fwd: 4dM (Q, K logits) + 4M(d+1) (state read + update) + (M+d+1)(c+1)
      bwd: 24dM + 10M + (3M+3d+1)(c+1) (recompute, downdate, gradients, chain
           rule through the feature map, dW)
    """
    c = min(C, tile)
    fwd = 4 * d * M + 4 * M * (d + 1) + (M + d + 1) * (c + 1)
    bwd = 24 * d * M + 10 * M + (3 * M + 3 * d + 1) * (c + 1)
    return fwd, bwd


def kernel_sources_sha() -> str:
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2012_11346_amd", "csrc", "*"))):
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, units_per_launch: float):
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


def bwd_walk_name(wl, d: int, M: int) -> str:
    """Name of the reverse-walk kernel the library launches for this problem:
    the 8-wave form for bf16 problems with 32 or 64 features per wave."""
    forced4 = os.environ.get("SLIM_BWD_WAVES") == "4"
    return "bwd_walk8_kernel" if (wl.dtype == "bf16" and M // 4 in (32, 64) and not forced4) else "bwd_walk_kernel"


def cpu_baseline(x, C: int, B: int, H: int, L: int):
    """Time the fp64 oracle (Algorithm 1 with the in-slice quadratic form) on
    the whole batch of the workload (every batch element and head, full
    length).  Returns the record and the oracle's Y/gradients for a parity
    check of the timed configuration."""
    import oracle as O

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    Q, K, V, dY = (x[k] for k in ("Q", "K", "V", "dY"))
    t0 = time.perf_counter()
    Y, st = O.slim_forward(Q, K, V, x["W"], C, "favor+", within="quadratic")
    g = O.slim_backward(Q, K, V, x["W"], dY, C, "favor+", st, within="quadratic")
    t = time.perf_counter() - t0
    rec = {
        "value": B * L / t,
        "unit": "tokens/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"the whole workload batch (B={B}, H={H}, L={L}), fp64 Algorithm 1 forward + backward with "
        f"the in-slice quadratic form at C={C}; {t:.1f} s on the host",
        "seconds": t,
        "host_cpus": os.cpu_count(),
    }
    return rec, Y, g


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--C", type=int, default=64)
    ap.add_argument("--workload", default="sweep_32k")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--sweep-steps", type=int, default=3)
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="only copy a device buffer of this many MiB (calibration of memory counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path runs on a single "
              "MI355X; sharded, GPUs would split the heads and batch rows and sum dW with one all-reduce)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2012_11346_amd import slim
    from synth import make_inputs, workload

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.copy_mib > 0:
        # a plain copy of known size: reads and writes copy_mib MiB once per launch
        n = args.copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 3}), flush=True)
        return
    wl = workload(args.workload)
    B, H, L, d, M = wl.B, wl.H, wl.L, wl.d, wl.M
    kind = wl.kind
    t0 = time.perf_counter()
    x = make_inputs(wl)
    print(f"[bench] inputs generated in {time.perf_counter() - t0:.1f}s", file=sys.stderr, flush=True)
    dev = torch.device("cuda", 0)
    Q, K, V, dY = (x[k].to(dev) for k in ("Q", "K", "V", "dY"))
    W = x["W"].to(dev)
    torch.cuda.synchronize()
    io_bytes = torch.cuda.memory_allocated()

    def buffers(C):
        p = slim.problem(B, H, L, d, M, C, Q.dtype, kind)
        bufs = dict(
            Y=torch.empty_like(Q),
            st=torch.empty((B, H, M, d + 1), dtype=torch.float32, device=dev),
            ks=torch.empty((B, H), dtype=torch.float32, device=dev),
            dQ=torch.empty_like(Q),
            dK=torch.empty_like(K),
            dV=torch.empty_like(V),
            dW=torch.empty((M, d), dtype=torch.float32, device=dev),
            wsf=torch.empty(max(1, slim.workspace_bytes(p, slim.PHASE_FWD)), dtype=torch.uint8, device=dev),
            wsb=torch.empty(max(1, slim.workspace_bytes(p, slim.PHASE_BWD)), dtype=torch.uint8, device=dev),
        )
        # the forward's segment boundary states, handed to the backward (state-sized)
        n_ctx = slim.context_bytes(p)
        if n_ctx > 0:
            bufs["wsctx"] = torch.empty(n_ctx // 4, dtype=torch.float32, device=dev)
        return p, bufs

    def step(C, b):
        slim.fwd(Q, K, V, W, C, kind, ws=b["wsf"], Y=b["Y"], state_out=b["st"], kshift_out=b["ks"],
                 ctx=b.get("wsctx"))
        slim.bwd(Q, K, V, W, dY, C, b["ks"], kind, ws=b["wsb"], dQ=b["dQ"], dK=b["dK"], dV=b["dV"],
                 dW=b["dW"], ctx=b.get("wsctx"))

    def timed(C, steps, warmup):
        """warmup + `steps` timed steps, bracketed by two events.  Inside the
        timed region only the reverse walk's launches carry events (recorded
        by the library around that launch: its duration for the roofline);
        the per-call breakdown (forward, backward, forward walk) comes from a
        separate pass of the same steps afterwards, so that its events do not
        add to the timed steps."""
        torch.cuda.synchronize()
        pre = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        p, b = buffers(C)
        for _ in range(warmup):
            step(C, b)
        stream = torch.cuda.current_stream()
        mk = lambda: torch.cuda.Event(enable_timing=True)
        t0, t1 = mk(), mk()
        wb = [(mk(), mk()) for _ in range(steps)]
        bd = [[mk() for _ in range(5)] for _ in range(steps)]
        for e in [t0, t1] + [x_ for pair in wb for x_ in pair] + [x_ for e5 in bd for x_ in e5]:
            e.record(stream)  # create every event before the timed region
        torch.cuda.synchronize()
        t0.record(stream)
        for i in range(steps):
            slim.fwd(Q, K, V, W, C, kind, ws=b["wsf"], Y=b["Y"], state_out=b["st"], kshift_out=b["ks"],
                     ctx=b.get("wsctx"))
            slim.time_walk(slim.PHASE_BWD, wb[i][0], wb[i][1])
            slim.bwd(Q, K, V, W, dY, C, b["ks"], kind, ws=b["wsb"], dQ=b["dQ"], dK=b["dK"], dV=b["dV"],
                     dW=b["dW"], ctx=b.get("wsctx"))
        t1.record(stream)
        torch.cuda.synchronize()
        total_ms = t0.elapsed_time(t1)
        bwd_walk_ms = sum(x.elapsed_time(y) for x, y in wb) / steps
        peak = torch.cuda.max_memory_allocated()
        # breakdown pass (not timed as steps)
        for e in bd:
            e[0].record(stream)
            slim.time_walk(slim.PHASE_FWD, e[1], e[2])
            slim.fwd(Q, K, V, W, C, kind, ws=b["wsf"], Y=b["Y"], state_out=b["st"], kshift_out=b["ks"],
                     ctx=b.get("wsctx"))
            e[3].record(stream)
            slim.bwd(Q, K, V, W, dY, C, b["ks"], kind, ws=b["wsb"], dQ=b["dQ"], dK=b["dK"], dV=b["dV"],
                     dW=b["dW"], ctx=b.get("wsctx"))
            e[4].record(stream)
        torch.cuda.synchronize()
        avg = lambda i, j: sum(e[i].elapsed_time(e[j]) for e in bd) / steps
        out_bytes = sum(t.numel() * t.element_size() for k, t in b.items() if not k.startswith("ws"))
        return dict(total_ms=total_ms, ms=total_ms / steps, fwd_ms=avg(0, 3), bwd_ms=avg(3, 4),
                    fwd_walk_ms=avg(1, 2), bwd_walk_ms=bwd_walk_ms, peak=peak, extra=peak - pre - out_bytes,
                    out_bytes=out_bytes, ws_fwd=b["wsf"].numel(), ws_bwd=b["wsb"].numel(),
                    ctx=b["wsctx"].numel() * 4 if "wsctx" in b else 0,
                    segments=slim.num_segments(p)), b

    C = args.C
    print(f"[bench] timing C={C}: warmup {args.warmup}, steps {args.steps}", file=sys.stderr, flush=True)
    r, b = timed(C, args.steps, args.warmup)
    tokens = B * L
    value = tokens / (r["ms"] / 1e3)
    fl_f, fl_b = algo_flops_per_token_head(d, M, C)
    units = B * H * L  # token-heads per launch of either walk kernel
    # the walk kernels do all of the algorithmic work of their phase; the
    # segment pre-passes and scans are extra work of the parallel split
    if r["bwd_walk_ms"] >= r["fwd_walk_ms"]:
        dominant, dom_ms, dom_flops = bwd_walk_name(wl, d, M), r["bwd_walk_ms"], fl_b * units
    else:
        dominant, dom_ms, dom_flops = "fwd_walk_kernel", r["fwd_walk_ms"], fl_f * units
    achieved = dom_flops / (dom_ms / 1e3)
    traffic = load_traffic(dominant, units)
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
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: causal FAVOR+ attention fwd+bwd, B={B} H={H} L={L} d={d} M={M}, "
            f"bf16 inputs with fp32 accumulation, slice length C={C}",
            "B": B, "H": H, "L": L, "d": d, "M": M, "C": C, "kind": kind,
            "segments_per_head": r["segments"],
        },
        "fwd_ms": r["fwd_ms"],
        "bwd_ms": r["bwd_ms"],
        "fwd_walk_ms": r["fwd_walk_ms"],
        "bwd_walk_ms": r["bwd_walk_ms"],
        "roofline": {
            "kernel": dominant,
            "bound": "mfma",
            "achieved": achieved / 1e12,
            "peak": PEAK_BF16_FLOPS / 1e12,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_FLOPS,
            "traffic": traffic,
            "flops_per_token_head": {"fwd": fl_f, "bwd": fl_b},
            "token_heads_per_launch": units,
            "launch_ms": dom_ms,
        },
        "mfma_frac_fwd_bwd": (fl_f + fl_b) * units / (r["ms"] / 1e3) / PEAK_BF16_FLOPS,
        "peak_mem": {"peak_bytes": r["peak"], "input_bytes": io_bytes, "output_bytes": r["out_bytes"],
                     "beyond_io_bytes": r["extra"],
                     "workspace_fwd": r["ws_fwd"], "workspace_bwd": r["ws_bwd"], "context": r["ctx"]},
    }
    print(f"[bench] C={C}: {r['ms']:.3f} ms/step (fwd {r['fwd_ms']:.3f}, bwd {r['bwd_ms']:.3f}; walks "
          f"{r['fwd_walk_ms']:.3f} / {r['bwd_walk_ms']:.3f}), {value:.3e} tokens/s", file=sys.stderr, flush=True)

    if not args.no_sweep:
        sweep = []
        for Cs in wl.C:
            rs, bs = timed(Cs, args.sweep_steps, 5)
            del bs
            sweep.append({"C": Cs, "tokens_per_s": tokens / (rs["ms"] / 1e3), "ms_per_step": rs["ms"],
                          "peak_bytes": rs["peak"], "beyond_io_bytes": rs["extra"], "workspace_bwd": rs["ws_bwd"]})
            print(f"[bench] sweep C={Cs}: {rs['ms']:.3f} ms/step, extra memory {rs['extra'] / 2**20:.1f} MiB",
                  file=sys.stderr, flush=True)
        out["sweep"] = sweep

    if not args.no_cpu:
        print("[bench] timing the fp64 oracle on the host", file=sys.stderr, flush=True)
        rec, Yo, go = cpu_baseline(x, C, B, H, L)
        out["cpu_baseline"] = rec

        # parity of the timed configuration against the oracle, whole batch
        def mr(a, ref):
            return float(np.max(np.abs(a.double().cpu().numpy() - ref)) / np.max(np.abs(ref)))

        out["parity"] = {"Y": mr(b["Y"], Yo), "dQ": mr(b["dQ"], go[0]), "dK": mr(b["dK"], go[1]),
                         "dV": mr(b["dV"], go[2]), "dW": mr(b["dW"], go[3])}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
