"""Throughput of one ResBM boundary forward + backward on one MI355X.

A step is the whole hot path over one batch: resbm_encode_fwd, resbm_decode_fwd,
resbm_decode_bwd, resbm_encode_bwd on T tokens of width n at rank r, all on
torch's current HIP stream, inputs resident in HBM.  Consecutive steps rotate
over several copies of the inputs and outputs so that no step finds its
streams in the 256 MB Infinity Cache left behind by the previous one.

Prints one JSON line: tokens/s (value), algorithmic HBM GB/s and its fraction
of the 8 TB/s peak, per-op times from HIP events recorded inside the timed
steps, the roofline entry of the dominant op, and the CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
OPS = ("encode_fwd", "decode_fwd", "decode_bwd", "encode_bwd")


def op_bytes(T: int, n: int, r: int) -> dict:
    """Bytes each op must move (activations per token plus weights once)."""
    w = 4 * n * r
    return {
        "encode_fwd": T * (2 * n + 8 * r) + w,          # z, skip cols, b, a_save; W_e
        "decode_fwd": T * (2 * n + 2 * r) + w,          # b, z~; W_d
        "decode_bwd": T * (2 * n + 6 * r) + 2 * w,      # g_z~, b, g_id cols, g_b; W_d, dW_d
        "encode_bwd": T * (4 * n + 6 * r) + 2 * w,      # z, g_z, g_b, a_save; W_e, dW_e
    }


def parse():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default=None, help="workload name (default: the headline n=4096 r=32)")
    p.add_argument("--sets", type=int, default=4, help="rotating input/output copies")
    p.add_argument("--act", default="silu", choices=["silu", "identity"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-op-events", action="store_true", help="time whole steps only")
    p.add_argument("--copy-probe-mib", type=int, default=256,
                   help="size of the plain device copy timed as the achievable-bandwidth reference (0: skip)")
    p.add_argument("--cpu-tokens", type=int, default=None, help="tokens in the CPU oracle sample")
    return p.parse_args()


def cpu_baseline(d: dict, r: int, act: int, tokens: int, min_seconds: float = 10.0) -> dict:
    """The float64 oracle over the first `tokens` tokens, all four ops, repeated
    until at least `min_seconds` have elapsed; reports the mean rate."""
    import numpy as np

    import oracle as O
    from paper_2604_11947_amd import inputs as I

    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        threads = int(os.environ.get("OMP_NUM_THREADS", "1"))
    W_e = I.bf16_to_f64(d["W_e"])
    W_d = I.bf16_to_f64(d["W_d"])
    n = W_e.shape[0]
    chunk = 2048
    reps = 0
    t0 = time.perf_counter()
    while True:
        dW_d = np.zeros((r, n))
        dW_e = np.zeros((n, r))
        for c0 in range(0, tokens, chunk):
            c1 = min(tokens, c0 + chunk)
            x = I.bf16_to_f64(d["x_attn"][c0:c1])
            z = I.bf16_to_f64(d["z"][c0:c1])
            gzt = I.bf16_to_f64(d["g_zt"][c0:c1])
            gid = I.bf16_to_f64(d["g_id"][c0:c1])
            b, a = O.encode_fwd(x, z, W_e, act)
            b_w = O.rne_bf16(b)
            O.decode_fwd(b_w, W_d, False)
            g_b, dwd = O.decode_bwd(b_w, W_d, gzt, gid)
            g_z, dwe = O.encode_bwd(z, W_e, a, O.rne_bf16(g_b), act)
            dW_d += dwd
            dW_e += dwe
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": reps * tokens / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {tokens} tokens of the workload (all of it when equal to T), all four ops in "
                      f"float64 with bf16 wire rounding, {reps} repetition(s) in {dt:.1f} s; "
                      f"{len(os.sched_getaffinity(0))} host cores visible"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested): this build runs the "
              f"boundary module on a single MI355X; across GPUs it would shard by tokens", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2604_11947_amd import inputs as I
    from paper_2604_11947_amd import resbm as R

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    name = args.workload or I.HEADLINE
    w = I.WORKLOADS[name]
    T, n, r = w.tokens, w.n, w.r
    act = R.ACT_SILU if args.act == "silu" else R.ACT_IDENTITY
    lib = R.library("bf16")
    dev = torch.device("cuda:0")

    t_gen = time.perf_counter()
    d = I.make_inputs(T, n, r, w.dist, w.seed)
    t_gen = time.perf_counter() - t_gen
    io = lib.io_dtype
    sets = []
    for _ in range(max(1, args.sets)):
        s = {k: d[k].to(dev) for k in ("x_attn", "z", "W_e", "W_d", "g_zt", "g_id")}
        s.update(
            b=torch.empty(T, r, dtype=io, device=dev),
            a=torch.empty(T, r, dtype=torch.float32, device=dev),
            zt=torch.empty(T, n, dtype=io, device=dev),
            gb=torch.empty(T, r, dtype=io, device=dev),
            gz=torch.empty(T, n, dtype=io, device=dev),
            dWd=torch.empty(r, n, dtype=torch.float32, device=dev),
            dWe=torch.empty(n, r, dtype=torch.float32, device=dev),
            ws=lib.workspace(T, n, r, dev),
        )
        sets.append(s)
    torch.cuda.synchronize()

    def step(s, ev=None):
        if ev is not None:
            ev[0].record()
        lib.encode_fwd(s["x_attn"], s["z"], s["W_e"], s["b"], s["a"], act=act, ws=s["ws"])
        if ev is not None:
            ev[1].record()
        lib.decode_fwd(s["b"], s["W_d"], s["zt"], ws=s["ws"])
        if ev is not None:
            ev[2].record()
        lib.decode_bwd(s["b"], s["W_d"], s["g_zt"], s["g_id"], s["gb"], s["dWd"], ws=s["ws"])
        if ev is not None:
            ev[3].record()
        lib.encode_bwd(s["z"], s["W_e"], s["a"], s["gb"], s["gz"], s["dWe"], act=act, ws=s["ws"])
        if ev is not None:
            ev[4].record()

    copy_gbs = None
    if args.copy_probe_mib > 0:
        # plain copy of known size: reference for achievable bandwidth and for
        # scaling the FETCH_SIZE / WRITE_SIZE counters
        nel = args.copy_probe_mib * 2**20 // 2
        src = torch.empty(nel, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(5):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        copy_gbs = 2 * nel * 2 * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
        del src, dst

    for i in range(args.warmup):
        step(sets[i % len(sets)])
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record()
    for i in range(args.steps):
        step(sets[i % len(sets)], None if args.no_op_events else events[i])
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps

    op_ms = {}
    for k, nm in enumerate(OPS):
        op_ms[nm] = (float("nan") if args.no_op_events
                     else sum(e[k].elapsed_time(e[k + 1]) for e in events) / args.steps)
    ob = op_bytes(T, n, r)
    total_bytes = sum(ob.values())
    gbs = total_bytes / (ms_step * 1e-3) / 1e9
    dom = "encode_bwd" if args.no_op_events else max(OPS, key=lambda k: op_ms[k])
    dom_gbs = ob[dom] / (op_ms[dom] * 1e-3) / 1e9

    out = {
        "metric": "tokens/s and achieved HBM GB/s (% peak), ResBM fwd+bwd, n=4096 r=32",
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": name, "tokens": T, "n": n, "r": r, "batch": w.batch, "seq_len": w.seq,
                   "activations": w.dist, "act": args.act, "io": "bf16 activations, fp32 weights",
                   "parallelism": "single GPU", "rotating_sets": len(sets)},
        "hbm_gbps": gbs,
        "hbm_frac": gbs / HBM_PEAK_GBS,
        "bytes_per_step": total_bytes,
        "copy_probe_gbps": copy_gbs,
        "ops": {k: {"ms": op_ms[k], "gbps": ob[k] / (op_ms[k] * 1e-3) / 1e9, "bytes": ob[k]} for k in OPS},
        "roofline": {"bound": "hbm", "op": dom, "achieved": dom_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": dom_gbs / HBM_PEAK_GBS, "traffic": None},
        "wall_s_timed": wall,
        "input_gen_s": t_gen,
    }
    if not args.no_cpu_baseline:
        tokens = args.cpu_tokens or T
        out["cpu_baseline"] = cpu_baseline(d, r, act, min(tokens, T))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
