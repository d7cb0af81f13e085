"""Throughput of one ResBM boundary forward + backward on one MI355X.

A step is the whole hot path over one batch: resbm_encode_fwd, resbm_decode_fwd,
resbm_decode_bwd, resbm_encode_bwd on T tokens of width n at rank r, all on
one HIP stream, inputs resident in HBM.  Consecutive steps rotate over several
copies of the inputs and outputs so that no step finds its streams in the
256 MB Infinity Cache left behind by the previous one; the library's scratch
workspace is one buffer shared by all steps, as a caller would keep it.

The step is timed twice: captured in HIP graphs of several consecutive steps
(input copies in turn) and replayed (the reported value; a graph removes the
host's launch gaps between the ops, as the enclosing training step's graph
would), and launched eagerly with HIP events between the ops.  Each op is also
timed alone from graph replays of several calls (per-op times, the roofline
entry of the dominant op).  Prints one JSON line, with the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

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
    p.add_argument("--steps", type=int, default=200)
    # the GPU reaches its steady clocks only after ~20 ms of this load; 200 steps
    # (~35 ms, untimed) get it there (10 steps left the timed steps ~6 % slower)
    p.add_argument("--warmup", type=int, default=200)
    p.add_argument("--workload", default=None, help="workload name (default: the headline n=4096 r=32)")
    p.add_argument("--sets", type=int, default=4, help="rotating input/output copies")
    p.add_argument("--act", default="silu", choices=["silu", "identity"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-op-events", action="store_true", help="time whole steps only")
    p.add_argument("--copy-probe-mib", type=int, default=COPY_PROBE_MIB,
                   help="size of the plain device copy timed as the achievable-bandwidth reference (0: skip)")
    p.add_argument("--cpu-tokens", type=int, default=None, help="tokens in the CPU oracle sample")
    p.add_argument("--no-graph", action="store_true", help="report the eager launches instead of graph replays")
    p.add_argument("--graph-steps", type=int, default=8,
                   help="consecutive steps captured in one HIP graph (input copies in turn) for the sweep and "
                        "per-op timings; the timed steps use the largest divisor of --steps up to twice this")
    p.add_argument("--no-optimizer", action="store_true",
                   help="skip timing the optimizer-side ops (Muon update, spectrum) on the bottleneck weights")
    p.add_argument("--two-m", type=int, default=1024,
                   help="intermediate width m of the two-linears-per-side variant (0: skip timing it)")
    p.add_argument("--qkv-width", type=int, default=6144,
                   help="N of the QKV projection the fused decoder is timed on (0 skips it)")
    p.add_argument("--ffn-width", type=int, default=14336,
                   help="FFN hidden width for timing the encoder fused into the FFN output projection (0: skip)")
    p.add_argument("--no-sweep", action="store_true",
                   help="skip the compression-ratio sweep (r = 16 .. 256 at n = 4096) and the 70B-class line")
    p.add_argument("--step-times", action="store_true", help="list every timed step's duration")
    p.add_argument("--summarize-profiles", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                   help="write profiles/ summaries from rocprofv3 output of this script (no GPU work)")
    p.add_argument("--summarize-trace", metavar="TRACE_DIR",
                   help="write profiles/kernels_<workload>.txt from a rocprofv3 kernel trace alone (no GPU work)")
    p.add_argument("--summarize-counters", nargs="+", metavar="PMC_DIR",
                   help="write profiles/counters_<workload>.json from rocprofv3 --pmc runs of this script (no GPU work)")
    p.add_argument("--commands", nargs="+", default=None, help="the rocprofv3 commands, recorded in the summaries")
    return p.parse_args()


KERNEL_OP = (("k_enc_fwd", "encode_fwd"), ("k_dec_bwd", "decode_bwd"), ("k_enc_bwd", "encode_bwd"))


def kernel_op(name: str):
    """The boundary op a kernel name belongs to (prologue and finishing kernels included).
    The expand kernel <KS, CT, ADD, GZ, R8> serves decode_fwd (GZ false) and the g_z pass
    of encode_bwd (GZ true)."""
    import re
    base = re.sub(r"\(.*", "", name)
    if "k_expand" in base:
        m = re.search(r"k_expand(?:_wide)?<([^>]*)>", base)
        if m:
            gz = m.group(1).split(",")[3].strip() == "true"
        else:  # mangled: two int arguments, then the ADD and GZ flags
            gz = re.search(r"k_expand(?:_wide)?I(?:Li\d+E){2}Lb[01]ELb1E", base) is not None
        return "encode_bwd" if gz else "decode_fwd"
    for key in ("k_rowc_wide", "k_tokc_wide"):
        if key in base:  # <NT, NTW, flag, ...>: the flag marks the decode_bwd instance
            m = re.search(key + r"<([^>]*)>", base)
            flag = m.group(1).split(",")[2].strip() == "true" if m else \
                re.search(key + r"I(?:Li\d+E){2}Lb1E", base) is not None
            return "decode_bwd" if flag else ("encode_fwd" if key == "k_rowc_wide" else "encode_bwd")
    if "k_wd_prep" in base:
        return "decode_bwd"
    if re.search(r"k_gh\b|4k_ghE", base):
        return "encode_bwd"
    for key, op in KERNEL_OP:
        if key in base or key.replace("_", "") in base.replace("_", ""):
            return op
    return None


def summarize_profiles(trace_dir: str, fetch_dir: str, write_dir: str, name: str, commands) -> None:
    """Kernel-time statistics of a traced bench run and per-op HBM traffic from FETCH_SIZE /
    WRITE_SIZE runs, scaled by what the same counters read for the plain device copy."""
    import glob
    import re
    import sqlite3

    def db(d):
        f = sorted(glob.glob(os.path.join(d, "**", "*results.db"), recursive=True))
        if not f:
            raise SystemExit(f"no rocprofv3 database under {d}")
        return sqlite3.connect(f[0])

    def short(k):
        return re.sub(r"\(.*", "", k).replace("void ", "")

    rows = list(db(trace_dir).execute("select name, end - start from kernels"))
    stats = {}
    for k, dur in rows:
        stats.setdefault(short(k), []).append(dur / 1000.0)

    def counter(d, cname):
        out = {}
        for k, cn, v in db(d).execute("select kernel_name, counter_name, value from counters_collection"):
            if cn == cname:
                out.setdefault(short(k), []).append(v)
        return out

    fetch_all, write_all = counter(fetch_dir, "FETCH_SIZE"), counter(write_dir, "WRITE_SIZE")
    copy_bytes = None
    for k in fetch_all:
        if "copyBuffer" in k or "copy" in k.lower():
            # the probe is the largest copy of the run (inputs are also copied, in smaller pieces)
            copy_bytes = COPY_PROBE_MIB * 2**20
            f_fetch = copy_bytes / (max(fetch_all[k]) * 1024)
            f_write = copy_bytes / (max(write_all[k]) * 1024)
            break
    if copy_bytes is None:
        raise SystemExit("the runs hold no plain copy kernel to calibrate the counters")
    fetch = {k: sum(v) / len(v) for k, v in fetch_all.items()}
    write = {k: sum(v) / len(v) for k, v in write_all.items()}
    ops = {}
    for k in fetch:
        op = kernel_op(k)
        if op is None or k not in write:
            continue
        e = ops.setdefault(op, {"kernels": {}, "hbm_bytes": 0.0})
        b = fetch[k] * 1024 * f_fetch + write[k] * 1024 * f_write
        e["kernels"][k] = {"fetch_kib": fetch[k], "write_kib": write[k], "hbm_bytes": b}
        e["hbm_bytes"] += b
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    rec = {"workload": name, "source_sha256": source_digest(), "fetch_scale": f_fetch, "write_scale": f_write,
           "calibration": f"plain device copy of {COPY_PROBE_MIB} MiB", "commands": commands, "ops": ops}
    with open(os.path.join(ROOT, "profiles", f"traffic_{name}.json"), "w") as fh:
        json.dump(rec, fh, indent=1)
    lines = [f"# rocprofv3 kernel trace, workload {name}", "", "command:", f"    {commands[0] if commands else '?'}", "",
             f"{'kernel':60s} {'calls':>6s} {'avg us':>9s} {'min us':>9s} {'max us':>9s}"]
    for k, v in sorted(stats.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"{k[:60]:60s} {len(v):6d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f}")
    lines += ["", "HBM traffic per call (FETCH_SIZE x %.3f + WRITE_SIZE x %.3f, calibrated on a plain copy):"
              % (f_fetch, f_write)]
    for op, e in ops.items():
        lines.append(f"    {op:12s} {e['hbm_bytes'] / 1e6:10.1f} MB")
    if commands:
        lines += ["", "counter commands:", f"    {commands[1]}", f"    {commands[2]}"]
    with open(os.path.join(ROOT, "profiles", f"kernels_{name}.txt"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    two = {k: v for k, v in stats.items() if k.startswith("resbm2::")}
    if two:
        lines = [f"# rocprofv3 kernel trace of the two-linears-per-side step (bench.py two_linear, m = 1024)"
                 f" and of the encoder fused into the FFN projection (ffn_encode, d_ff = 14336), workload {name}",
                 "", "command:", f"    {commands[0] if commands else '?'}", "",
                 f"{'kernel':60s} {'calls':>6s} {'avg us':>9s} {'min us':>9s} {'max us':>9s}"]
        for k, v in sorted(two.items(), key=lambda kv: -sum(kv[1])):
            lines.append(f"{k[:60]:60s} {len(v):6d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f}")
        with open(os.path.join(ROOT, "profiles", f"kernels_two_linear_{name}.txt"), "w") as fh:
            fh.write("\n".join(lines) + "\n")


def summarize_trace(trace_dir: str, name: str, commands) -> None:
    """Per-kernel duration statistics of a traced bench run of one workload."""
    import glob
    import re
    import sqlite3

    f = sorted(glob.glob(os.path.join(trace_dir, "**", "*results.db"), recursive=True))
    if not f:
        raise SystemExit(f"no rocprofv3 database under {trace_dir}")
    stats = {}
    for k, dur in sqlite3.connect(f[0]).execute("select name, end - start from kernels"):
        stats.setdefault(re.sub(r"\(.*", "", k).replace("void ", ""), []).append(dur / 1000.0)
    lines = [f"# rocprofv3 kernel trace, workload {name}", "", "command:",
             f"    {commands[0] if commands else '?'}", "",
             f"{'kernel':64s} {'op':11s} {'calls':>6s} {'avg us':>9s} {'med us':>9s} {'min us':>9s}"]
    for k, v in sorted(stats.items(), key=lambda kv: -sum(kv[1])):
        if "resbm" not in k:
            continue
        vs = sorted(v)
        lines.append(f"{k[:64]:64s} {kernel_op(k) or '-':11s} {len(v):6d} {sum(v) / len(v):9.2f} "
                     f"{vs[len(vs) // 2]:9.2f} {vs[0]:9.2f}")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"kernels_{name}.txt"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


COUNTER_PASSES = (
    "SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_INSTS_VMEM_RD "
    "SQ_INSTS_VMEM_WR SQ_INSTS_SALU",
    "SQ_WAVES SQ_BUSY_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_LDS SQ_WAIT_INST_LDS "
    "SQ_WAVE_CYCLES SQ_WAIT_ANY GRBM_GUI_ACTIVE",
    "TCC_HIT_sum TCC_MISS_sum TCC_EA0_RDREQ_DRAM_sum TCC_REQ_sum",
    "TCC_EA0_WRREQ_sum TCC_EA0_WRREQ_64B_sum TCC_WRITEBACK_sum TCP_TCC_READ_REQ_sum",
)


def summarize_counters(dirs, name: str, commands) -> None:
    """Per-kernel averages of the rocprofv3 --pmc passes in `dirs` (one pass per
    directory, COUNTER_PASSES) for the boundary kernels, with derived ratios:
    matrix-core share of the vector instructions, LDS bank-conflict cycles per
    LDS instruction cycle, L2 hit rate.  Writes profiles/counters_<name>.json."""
    import glob
    import re
    import sqlite3

    vals = {}
    for d in dirs:
        f = sorted(glob.glob(os.path.join(d, "**", "*results.db"), recursive=True))
        if not f:
            raise SystemExit(f"no rocprofv3 database under {d}")
        for k, cn, v in sqlite3.connect(f[0]).execute(
                "select kernel_name, counter_name, value from counters_collection"):
            k = re.sub(r"\(.*", "", k).replace("void ", "")
            if kernel_op(k) is None:
                continue
            vals.setdefault(k, {}).setdefault(cn, []).append(v)
    out = {}
    for k, cs in vals.items():
        avg = {cn: sum(v) / len(v) for cn, v in cs.items()}
        e = {"op": kernel_op(k), "dispatches": max(len(v) for v in cs.values()), "avg_per_dispatch": avg}
        g = avg.get
        if g("SQ_INSTS_VALU"):
            e["mfma_share_of_valu_insts"] = g("SQ_INSTS_MFMA", 0.0) / g("SQ_INSTS_VALU")
        if g("SQ_ACTIVE_INST_LDS"):
            e["lds_bank_conflict_cycles_per_lds_active_cycle"] = g("SQ_LDS_BANK_CONFLICT", 0.0) / g("SQ_ACTIVE_INST_LDS")
        if g("TCC_HIT_sum") is not None and g("TCC_MISS_sum") is not None and g("TCC_HIT_sum") + g("TCC_MISS_sum"):
            e["l2_hit_rate"] = g("TCC_HIT_sum") / (g("TCC_HIT_sum") + g("TCC_MISS_sum"))
        if g("SQ_WAVE_CYCLES"):
            e["wait_share_of_wave_cycles"] = g("SQ_WAIT_ANY", 0.0) / g("SQ_WAVE_CYCLES")
        if g("SQ_INSTS_MFMA") and g("GRBM_GUI_ACTIVE"):
            # 16-cycle 16x16x32 bf16 products per SIMD (1024 SIMDs) over the kernel's
            # active cycles (GRBM counts each of the 8 XCDs)
            e["mfma_issue_share"] = g("SQ_INSTS_MFMA") * 16.0 / 1024 / (g("GRBM_GUI_ACTIVE") / 8)
        out[k] = e
    rec = {"workload": name, "source_sha256": source_digest(), "passes": list(COUNTER_PASSES),
           "commands": commands, "kernels": out}
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"counters_{name}.json"), "w") as fh:
        json.dump(rec, fh, indent=1)
    for k, e in sorted(out.items(), key=lambda kv: kv[1]["op"]):
        print(f"{e['op']:11s} {k[:58]:58s} mfma/valu={e.get('mfma_share_of_valu_insts', float('nan')):.3f} "
              f"lds_conf={e.get('lds_bank_conflict_cycles_per_lds_active_cycle', float('nan')):.3f} "
              f"l2_hit={e.get('l2_hit_rate', float('nan')):.3f}")


def source_digest() -> str:
    """sha256 over the kernel sources; HBM traffic measured on other sources is not reported."""
    import hashlib
    h = hashlib.sha256()
    for f in ("resbm_kernels.hip", "resbm_plan.hpp", "resbm_mfma.hpp", "resbm_buffer.hpp"):
        with open(os.path.join(ROOT, "paper_2604_11947_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(name: str, op: str):
    """HBM bytes per call of `op` on workload `name` from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE scaled by the plain-copy calibration), if it was taken
    on the current kernel sources; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_sha256") != source_digest():
        return None
    return rec.get("ops", {}).get(op, {}).get("hbm_bytes")


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


def optimizer_timing(lib, d: dict, r: int, dev, iters: int, cpu: bool) -> dict:
    """Graph-replayed time of one Muon update of each bottleneck weight (Sec. 3.4)
    and of the spectrum / r_eff of W_d (App. B.1), with the float64 oracle timed
    on the same update when `cpu` is set."""
    import torch

    from paper_2604_11947_amd import inputs as I
    from paper_2604_11947_amd import resbm as R

    def graph_us(fn):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        for _ in range(20):
            g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / iters

    steps = 5
    # short side <= 64: load + Gram, ordered sum, the recurrence on the s x s Gram
    # (one block), output pass; wider: load, then per step reduce + poly + row update
    launches = 4 if r <= 64 else 1 + 3 * steps
    out = {"ns_steps": steps, "coefficients": list(R.NS_QUINTIC),
           "launches_per_update": launches,
           "timing": "hip graph replay of one call", "iterations": iters}
    keep = {}
    for nm in ("W_e", "W_d"):
        W0 = d[nm]
        p, q = W0.shape
        W, M = W0.to(dev).clone(), torch.zeros(p, q, device=dev)
        G = I.make_matrix(p, q, "gaussian", seed=11, scale=1e-2).to(dev)
        ws = lib.matrix_workspace(p, q, dev)
        out[f"muon_update_us_{nm}"] = graph_us(
            lambda W=W, G=G, M=M, ws=ws: lib.muon_update(W, G, M, 1e-4, momentum=0.95, ws=ws, steps=steps))
        keep[nm] = (W0, G, ws)
    # algorithmic flops of one update: per step the Gram (2 L s^2), B (2 s^3) and
    # X B (2 L s^2), plus the Gram of the loaded matrix; float64 vector peak
    W0 = d["W_e"]
    L_, s_ = max(W0.shape), min(W0.shape)
    flops = 2 * L_ * s_ * s_ + steps * (4 * L_ * s_ * s_ + 2 * s_ ** 3)
    tf = flops / (out["muon_update_us_W_e"] * 1e-6) / 1e12
    out["roofline"] = {"bound": "latency", "kernel": "muon_update", "achieved": tf, "peak": 78.6,
                       "unit": "TFLOP/s", "frac": tf / 78.6, "flops_per_update": flops,
                       "note": f"{launches} launches; launch and memory latency bound the chain"}
    if r <= 128:
        W0, _, ws = keep["W_d"]
        Wd = W0.to(dev)
        sig = torch.empty(min(W0.shape), dtype=torch.float64, device=dev)
        reff = torch.empty(1, dtype=torch.float64, device=dev)
        out["spectrum_us_W_d"] = graph_us(lambda: lib.spectrum(Wd, sig, reff, ws=ws))
        out["r_eff_W_d"] = float(reff.item())
    if cpu:
        from oracle import muon_oracle as MU
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 2.0:
            for nm in ("W_e", "W_d"):
                W0, G, _ = keep[nm]
                MU.muon_update(W0.double().numpy(), G.cpu().double().numpy(), np.zeros(tuple(W0.shape)), 1e-4, 0.95)
            reps += 1
        out["oracle_us_per_update_pair"] = (time.perf_counter() - t0) * 1e6 / reps
    return out


def two_linear_timing(lib, d: dict, r: int, m: int, dev, iters: int, cpu: bool, act: int) -> dict:
    """One training step of the two-linears-per-side bottleneck (Sec. 3.2) on the
    workload's activations: encode2_fwd, decode2_fwd, decode2_bwd, encode2_bwd
    (g_x fused into g_z).  Per-op times from HIP events on the launch stream
    around eager calls; the whole step from graph replays."""
    import torch

    from paper_2604_11947_amd import inputs as I

    T, n = d["z"].shape
    bf = torch.bfloat16
    w = {k: v.to(dev) for k, v in I.make_two_weights(n, m, r, seed=1).items()}
    x, z, g_zt, g_id = (d[k].to(dev) for k in ("x_attn", "z", "g_zt", "g_id"))
    b, u = torch.empty(T, r, dtype=bf, device=dev), torch.empty(T, m, dtype=bf, device=dev)
    zt, v = torch.empty(T, n, dtype=bf, device=dev), torch.empty(T, m, dtype=bf, device=dev)
    g_b, g_z = torch.empty(T, r, dtype=bf, device=dev), torch.empty(T, n, dtype=bf, device=dev)
    dW1, dW2 = torch.empty(n, m, device=dev), torch.empty(m, r, device=dev)
    dW3, dW4 = torch.empty(r, m, device=dev), torch.empty(m, n, device=dev)
    ws = lib.two_workspace(T, n, m, r, dev)
    ops = {
        "encode2_fwd": lambda: lib.encode2_fwd(x, z, w["W1"], w["W2"], b, u, act=act, ws=ws),
        "decode2_fwd": lambda: lib.decode2_fwd(b, w["W3"], w["W4"], zt, v, act=act, ws=ws),
        "decode2_bwd": lambda: lib.decode2_bwd(b, v, g_zt, g_id, w["W3"], w["W4"], g_b, dW3, dW4, act=act, ws=ws),
        "encode2_bwd": lambda: lib.encode2_bwd(z, u, g_b, w["W1"], w["W2"], g_z, dW1, dW2, g_x=g_z, act=act, ws=ws),
    }

    def step():
        for f in ops.values():
            f()

    for _ in range(5):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(ops) + 1)] for _ in range(iters)]
    for i in range(iters):
        ev[i][0].record(stream)
        for k, f in enumerate(ops.values()):
            f()
            ev[i][k + 1].record(stream)
    torch.cuda.synchronize()
    op_us = {nm: sum(e[k].elapsed_time(e[k + 1]) for e in ev) * 1e3 / iters for k, nm in enumerate(ops)}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(5):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / iters
    big, small = 2.0 * T * n * m, 2.0 * T * m * r
    # algorithmic flops per op: the n x m products and the r-wide ones
    flops = {"encode2_fwd": big + small, "decode2_fwd": big + small,
             "decode2_bwd": 2 * big + 2 * small, "encode2_bwd": 2 * big + 2 * small}
    dom = max(op_us, key=op_us.get)
    tf = flops[dom] / (op_us[dom] * 1e-6) / 1e12
    out = {"m": m, "tokens": T, "us_per_step": us, "tokens_per_s": T / (us * 1e-6),
           "tflops_step": sum(flops.values()) / (us * 1e-6) / 1e12,
           "ops_us": op_us, "iterations": iters, "timing": "ops: events around eager calls; step: graph replay",
           "roofline": {"bound": "mfma", "op": dom, "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": tf / MFMA_BF16_PEAK_TFLOPS, "flops": flops[dom]}}
    if cpu:
        from oracle import resbm_oracle as RO
        from oracle import two_linear_oracle as TL
        f64 = lambda t: t.to(torch.float64).cpu().numpy()  # noqa: E731
        W = {k: f64(v) for k, v in w.items()}
        Ts = 256
        xs, zs, gzs, gis = (f64(t[:Ts]) for t in (x, z, g_zt, g_id))
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 10.0:
            bb, uu = TL.encode2_fwd(xs, zs, W["W1"], W["W2"], act)
            _, vv = TL.decode2_fwd(bb, W["W3"], W["W4"], act)
            gb, _, _ = TL.decode2_bwd(bb, vv, gzs, gis, W["W3"], W["W4"], act)
            gz, _, _ = TL.encode2_bwd(zs, uu, gb, W["W1"], W["W2"], act)
            RO.skip_grad(gz, gb)
            reps += 1
        sec = (time.perf_counter() - t0) / reps
        out["cpu_baseline"] = {"value": Ts / sec, "unit": "tokens/s", "cores": torch.get_num_threads(),
                               "kind": "oracle", "sample": f"{Ts} tokens of the same step, {reps} repetitions"}
    return out


def ffn_encode_timing(lib, d: dict, r: int, d_ff: int, dev, iters: int, act: int, cpu: bool) -> dict:
    """The encoder fused into the FFN output projection (resbm_ffn_encode_fwd: z = h W_down
    with the encoder in the epilogue) against the unfused pair: the same projection by
    the framework's library GEMM (torch.matmul, hipBLASLt) followed by resbm_encode_fwd,
    called back to back (each part also timed alone).  HIP events on the launch stream."""
    import torch

    from paper_2604_11947_amd import inputs as I

    T, n = d["z"].shape
    bf = torch.bfloat16
    h = I.make_bf16(T, d_ff, 41).to(dev)
    W_down = I.make_bf16(d_ff, n, 42, std=d_ff ** -0.5).to(dev)
    x, W_e = d["x_attn"].to(dev), d["W_e"].to(dev)
    z, b = torch.empty(T, n, dtype=bf, device=dev), torch.empty(T, r, dtype=bf, device=dev)
    a = torch.empty(T, r, device=dev)
    ws = lib.workspace(T, n, r, dev)
    def unfused():
        torch.matmul(h, W_down, out=z)
        lib.encode_fwd(x, z, W_e, b, a_save=a, act=act, ws=ws)

    calls = {
        "fused": lambda: lib.ffn_encode_fwd(h, W_down, x, W_e, z, b, a_save=a, act=act),
        "unfused": unfused,
        "library_gemm": lambda: torch.matmul(h, W_down, out=z),
        "encode_fwd": lambda: lib.encode_fwd(x, z, W_e, b, a_save=a, act=act, ws=ws),
    }
    stream = torch.cuda.current_stream()
    us = {}
    for nm, f in calls.items():
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        us[nm] = e0.elapsed_time(e1) * 1e3 / iters
    flops = 2.0 * T * d_ff * n + 2.0 * T * n * r
    tf = flops / (us["fused"] * 1e-6) / 1e12
    out = {"d_ff": d_ff, "tokens": T, "us": us, "unfused_us": us["unfused"],
           "fused_over_unfused": us["fused"] / us["unfused"], "iterations": iters,
           "timing": "HIP events around each call; unfused = the library GEMM and resbm_encode_fwd back to back",
           "tokens_per_s": T / (us["fused"] * 1e-6),
           "roofline": {"bound": "mfma", "kernel": "k_gemm<256x256, encoder epilogue>", "achieved": tf,
                        "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": tf / MFMA_BF16_PEAK_TFLOPS,
                        "flops": flops}}
    if cpu:
        from oracle import fusion_oracle as FO
        Ts = 64
        f64 = lambda t: t.to(torch.float64).cpu().numpy()  # noqa: E731
        hs, Wd, xs, We = f64(h[:Ts]), f64(W_down), f64(x[:Ts]), W_e.double().cpu().numpy()
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 10.0:
            FO.ffn_encode_fwd(hs, Wd, xs, We, act)
            reps += 1
        sec = (time.perf_counter() - t0) / reps
        out["cpu_baseline"] = {"value": Ts / sec, "unit": "tokens/s", "cores": torch.get_num_threads(),
                               "kind": "oracle", "sample": f"{Ts} tokens of the same op, {reps} repetitions"}
    return out


def decode_qkv_timing(lib, d: dict, r: int, N: int, dev, iters: int, cpu: bool) -> dict:
    """The decoder fused into the next block's RMS normalisation and QKV projection
    (resbm_decode_qkv_fwd) against the unfused chain: resbm_decode_fwd, the framework's
    RMS normalisation (torch.nn.functional.rms_norm) and its library GEMM (torch.matmul,
    hipBLASLt), called back to back (each part also timed alone).  HIP events."""
    import torch
    import torch.nn.functional as TF

    from paper_2604_11947_amd import inputs as I

    T, n = d["z"].shape
    bf = torch.bfloat16
    eps = 1e-5
    b = I.make_bf16(T, r, 44).to(dev)
    W_d = d["W_d"].to(dev)
    gamma = I.make_gain(n, 45).to(dev)
    gamma_bf = gamma.to(bf)
    W_qkv = I.make_bf16(n, N, 46, std=n ** -0.5).to(dev)
    out = torch.empty(T, N, dtype=bf, device=dev)
    zt = torch.empty(T, n, dtype=bf, device=dev)
    y = torch.empty(T, n, dtype=bf, device=dev)
    ws = lib.workspace(T, n, r, dev)
    qws = torch.empty(int(lib.cdll.resbm_decode_qkv_workspace_bytes(n, r)) + 256, dtype=torch.uint8, device=dev)
    qws = qws[(-qws.data_ptr()) % 256:]

    def norm():
        y.copy_(TF.rms_norm(zt, (n,), weight=gamma_bf, eps=eps))

    def unfused():
        lib.decode_fwd(b, W_d, zt, ws=ws)
        norm()
        torch.matmul(y, W_qkv, out=out)

    calls = {
        "fused": lambda: lib.decode_qkv_fwd(b, W_d, gamma, W_qkv, out, eps=eps, ws=qws),
        "unfused": unfused,
        "decode_fwd": lambda: lib.decode_fwd(b, W_d, zt, ws=ws),
        "rms_norm": norm,
        "library_gemm": lambda: torch.matmul(y, W_qkv, out=out),
    }
    stream = torch.cuda.current_stream()
    us = {}
    for nm, f in calls.items():
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(iters):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        us[nm] = e0.elapsed_time(e1) * 1e3 / iters
    KS = (r + 31) // 32
    flops = 2.0 * T * n * N
    rebuild = 2.0 * T * r * n * 2 * ((N + 255) // 256)  # hi + lo products, once per 256-column tile of N
    tf = flops / (us["fused"] * 1e-6) / 1e12
    res = {"N": N, "tokens": T, "us": us, "unfused_us": us["unfused"],
           "fused_over_unfused": us["fused"] / us["unfused"], "iterations": iters,
           "timing": "HIP events around each call; unfused = decode_fwd, rms_norm and the library GEMM back to back",
           "rebuild_share_of_products": 2 * KS * 32 / 256 if r <= 64 else None,
           "tokens_per_s": T / (us["fused"] * 1e-6),
           "roofline": {"bound": "mfma", "kernel": "k_dec_qkv (256x256 tiles, A tiles rebuilt from b W_d)",
                        "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": tf / MFMA_BF16_PEAK_TFLOPS, "flops": flops, "rebuild_flops": rebuild}}
    if cpu:
        from oracle import fusion_oracle as FO
        Ts = 64
        f64 = lambda t: t.to(torch.float64).cpu().numpy()  # noqa: E731
        bs, Wd, g, W = f64(b[:Ts]), W_d.double().cpu().numpy(), gamma.double().cpu().numpy(), f64(W_qkv)
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 5.0:
            FO.decode_qkv_fwd(bs, Wd, g, W, eps)
            reps += 1
        sec = (time.perf_counter() - t0) / reps
        res["cpu_baseline"] = {"value": Ts / sec, "unit": "tokens/s", "cores": torch.get_num_threads(),
                               "kind": "oracle", "sample": f"{Ts} tokens of the same op, {reps} repetitions"}
    return res


def sweep_timing(lib, dev, names, steps: int, warmup: int, act: int, G: int = 1) -> dict:
    """The whole step (four ops, graph replay) at each workload in `names`: the
    compression-ratio sweep at n = 4096 and the 70B-class boundary.  Inputs are
    drawn on the device (torch, seeded) with each workload's shape and
    distribution; kernel time does not depend on the values.  Two rotating input
    sets; G consecutive steps per graph replay (steps and warmup are multiples
    of G).  Reports per-step median time (per replay, divided by G), algorithmic HBM GB/s, and matrix-core
    rates: algorithmic (12 T n r flops per step) and issued (24 T n r: the hi and
    lo bf16 products of the float32 weights and of g_h)."""
    import torch

    from paper_2604_11947_amd import inputs as I

    out = {}
    for name in names:
        w = I.WORKLOADS[name]
        T, n, r = w.tokens, w.n, w.r
        gen = torch.Generator(device=dev)
        gen.manual_seed(1000 + r)
        bf = torch.bfloat16

        def act_tensor():
            x = torch.randn(T, n, device=dev, generator=gen)
            if w.dist == "token_lognormal":
                x *= torch.exp(0.5 * torch.randn(T, 1, device=dev, generator=gen))
            return x.to(bf)

        sets = []
        for _ in range(2):
            sets.append({
                "x_attn": act_tensor(), "z": act_tensor(),
                "g_zt": (0.1 * torch.randn(T, n, device=dev, generator=gen)).to(bf),
                "g_id": (0.1 * torch.randn(T, n, device=dev, generator=gen)).to(bf),
                "W_e": torch.randn(n, r, device=dev, generator=gen) / n ** 0.5,
                "W_d": torch.randn(r, n, device=dev, generator=gen) / r ** 0.5,
                "b": torch.empty(T, r, dtype=bf, device=dev), "a": torch.empty(T, r, device=dev),
                "zt": torch.empty(T, n, dtype=bf, device=dev), "gb": torch.empty(T, r, dtype=bf, device=dev),
                "gz": torch.empty(T, n, dtype=bf, device=dev), "dWd": torch.empty(r, n, device=dev),
                "dWe": torch.empty(n, r, device=dev)})
        ws = lib.workspace(T, n, r, dev)

        def step(s):
            lib.encode_fwd(s["x_attn"], s["z"], s["W_e"], s["b"], s["a"], act=act, ws=ws)
            lib.decode_fwd(s["b"], s["W_d"], s["zt"], ws=ws)
            lib.decode_bwd(s["b"], s["W_d"], s["g_zt"], s["g_id"], s["gb"], s["dWd"], ws=ws)
            lib.encode_bwd(s["z"], s["W_e"], s["a"], s["gb"], s["gz"], s["dWe"], act=act, ws=ws)

        for s_ in sets:
            step(s_)
        torch.cuda.synchronize()
        G = max(1, G)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(G):
                step(sets[i % 2])
        for i in range(max(1, warmup // G)):
            g.replay()
        nrep = max(1, steps // G)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(nrep + 1)]
        ev[0].record()
        for i in range(nrep):
            g.replay()
            ev[i + 1].record()
        torch.cuda.synchronize()
        st = np.asarray([ev[i].elapsed_time(ev[i + 1]) / G for i in range(nrep)]) * 1e3
        med = float(np.median(st))
        nbytes = sum(op_bytes(T, n, r).values())
        alg = 12.0 * T * n * r
        out[name] = {"n": n, "r": r, "tokens": T, "us_median": med, "us_mean": float(st.mean()),
                     "us_p10": float(np.percentile(st, 10)), "us_p90": float(np.percentile(st, 90)),
                     "tokens_per_s": T / (med * 1e-6), "gbps": nbytes / (med * 1e-6) / 1e9,
                     "hbm_frac": nbytes / (med * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     "tflops_alg": alg / (med * 1e-6) / 1e12, "tflops_issued": 2 * alg / (med * 1e-6) / 1e12,
                     "mfma_frac_issued": 2 * alg / (med * 1e-6) / 1e12 / MFMA_BF16_PEAK_TFLOPS}
        del g, sets, ws
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return {"workloads": out, "steps": max(1, steps // G) * G, "warmup": max(1, warmup // G) * G,
            "timing": f"hip graph replay, {G} steps per graph, events between replays",
            "inputs": "drawn on the device (torch, seeded), each workload's shape and distribution"}


SWEEP = ("sweep_n4096_r16", "sweep_n4096_r32", "sweep_n4096_r64", "sweep_n4096_r128", "sweep_n4096_r256",
         "n8192_r64_lognormal")


MFMA_BF16_PEAK_TFLOPS = 2500.0
COPY_PROBE_MIB = 256


def main():
    args = parse()
    if args.summarize_profiles:
        from paper_2604_11947_amd import inputs as I
        summarize_profiles(*args.summarize_profiles, args.workload or I.HEADLINE, args.commands)
        return
    if args.summarize_trace:
        from paper_2604_11947_amd import inputs as I
        summarize_trace(args.summarize_trace, args.workload or I.HEADLINE, args.commands)
        return
    if args.summarize_counters:
        from paper_2604_11947_amd import inputs as I
        summarize_counters(args.summarize_counters, args.workload or I.HEADLINE, args.commands)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested): the boundary module runs "
              f"on a single MI355X; across GPUs it would shard by tokens", file=sys.stderr)
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
    ws = lib.workspace(T, n, r, dev)
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
        )
        sets.append(s)
    torch.cuda.synchronize()

    def step(s, ev=None):
        if ev is not None:
            ev[0].record()
        lib.encode_fwd(s["x_attn"], s["z"], s["W_e"], s["b"], s["a"], act=act, ws=ws)
        if ev is not None:
            ev[1].record()
        lib.decode_fwd(s["b"], s["W_d"], s["zt"], ws=ws)
        if ev is not None:
            ev[2].record()
        lib.decode_bwd(s["b"], s["W_d"], s["g_zt"], s["g_id"], s["gb"], s["dWd"], ws=ws)
        if ev is not None:
            ev[3].record()
        lib.encode_bwd(s["z"], s["W_e"], s["a"], s["gb"], s["gz"], s["dWe"], act=act, ws=ws)
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

    # HIP graphs captured first: one of G consecutive steps (input copies in
    # turn) and one single step per input copy (for warmup and a remainder of K
    # modulo G).  A training step runs these ops inside a larger captured graph;
    # replaying one step per graph would add the ~9 us launch of each replay to
    # every step.  The compression-ratio sweep then keeps the GPU busy for a few
    # seconds, and the headline replays follow it directly, so that they run at
    # the clocks a busy GPU holds (after an idle spell the first ~100 steps of
    # this load ran up to ~8 % slower).
    for s in sets:
        step(s)
    torch.cuda.synchronize()
    G = max(1, args.graph_steps)
    # the timed steps' graph: the largest divisor of K up to 2 G, so that K
    # steps are whole replays of it (else G steps per graph and single-step
    # replays for the remainder)
    GH = next((g for g in range(min(args.steps, 2 * G), 1, -1) if args.steps % g == 0), G)
    g_multi, g_single = None, []
    if not args.no_graph:
        for s in sets:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(s)
            g_single.append(g)
        if GH > 1:
            g_multi = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_multi):
                for i in range(GH):
                    step(sets[i % len(sets)])
    sweep = None if args.no_sweep else sweep_timing(lib, dev, SWEEP, 48, 24, act, G)

    ms_graph = None
    if g_single:
        def replays(k):
            # (graph, steps) covering exactly k steps
            full = k // GH if g_multi is not None else 0
            return [(g_multi, GH)] * full + [(g_single[i % len(sets)], 1) for i in range(k - full * GH)]
        for g, _ in replays(args.warmup):
            g.replay()
        plan = replays(args.steps)
        # one event between consecutive replays: per-step times (averaged over
        # the G steps of a multi-step replay), and the first and last bracket
        # exactly the K timed steps
        gev = [torch.cuda.Event(enable_timing=True) for _ in range(len(plan) + 1)]
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        gev[0].record()
        for i, (g, _) in enumerate(plan):
            g.replay()
            gev[i + 1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        ms_graph = gev[0].elapsed_time(gev[-1]) / args.steps
        per = [(gev[i].elapsed_time(gev[i + 1]) / k, k) for i, (_, k) in enumerate(plan)]
        multi = [t for t, k in per if k == GH]
        step_ms = multi if multi else [t for t, _ in per]

    # eager launches, HIP events between the ops (on the stream the ops run on):
    # per-op times, and the headline itself with --no-graph
    for i in range(args.warmup):
        step(sets[i % len(sets)])
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall_e = time.perf_counter()
    start.record()
    for i in range(args.steps):
        step(sets[i % len(sets)], None if args.no_op_events else events[i])
    stop.record()
    torch.cuda.synchronize()
    wall_e = time.perf_counter() - wall_e
    ms_eager = start.elapsed_time(stop) / args.steps
    if not g_single:
        wall = wall_e
        step_ms = [sum(e[k].elapsed_time(e[k + 1]) for k in range(4)) for e in events] if not args.no_op_events \
            else []
    ms_step = ms_graph if ms_graph is not None else ms_eager
    step_stats = None
    if step_ms:
        q = np.percentile(np.asarray(step_ms), [10, 50, 90])
        step_stats = {"p10_ms": float(q[0]), "median_ms": float(q[1]), "p90_ms": float(q[2]),
                      "first_ms": float(step_ms[0]), "last_ms": float(step_ms[-1])}

    op_ms_eager = {}
    for k, nm in enumerate(OPS):
        op_ms_eager[nm] = (float("nan") if args.no_op_events
                           else sum(e[k].elapsed_time(e[k + 1]) for e in events) / args.steps)
    # per-op times without the host's launch gaps: each op alone, G calls per
    # graph (input copies in turn), replays bracketed by events
    op_ms = dict(op_ms_eager)
    if g_single and not args.no_op_events:
        op_fn = {
            "encode_fwd": lambda s: lib.encode_fwd(s["x_attn"], s["z"], s["W_e"], s["b"], s["a"], act=act, ws=ws),
            "decode_fwd": lambda s: lib.decode_fwd(s["b"], s["W_d"], s["zt"], ws=ws),
            "decode_bwd": lambda s: lib.decode_bwd(s["b"], s["W_d"], s["g_zt"], s["g_id"], s["gb"], s["dWd"], ws=ws),
            "encode_bwd": lambda s: lib.encode_bwd(s["z"], s["W_e"], s["a"], s["gb"], s["gz"], s["dWe"], act=act,
                                                   ws=ws),
        }
        nrep = max(16, args.steps // G)  # at least 128 calls per op, whatever K
        for nm in OPS:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(G):
                    op_fn[nm](sets[i % len(sets)])
            for _ in range(3):
                g.replay()
            o0, o1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            o0.record()
            for _ in range(nrep):
                g.replay()
            o1.record()
            torch.cuda.synchronize()
            op_ms[nm] = o0.elapsed_time(o1) / (nrep * G)
            del g
    ob = op_bytes(T, n, r)
    total_bytes = sum(ob.values())
    gbs = total_bytes / (ms_step * 1e-3) / 1e9
    dom = "encode_bwd" if args.no_op_events else max(OPS, key=lambda k: op_ms[k])
    dom_gbs = ob[dom] / (op_ms[dom] * 1e-3) / 1e9

    traffic = measured_traffic(name, dom)
    out = {
        "metric": f"tokens/s and achieved HBM GB/s (% peak), ResBM fwd+bwd, n={n} r={r}",
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "timing": (f"hip graph replay, {GH} steps per graph" if ms_graph is not None else "eager launches"),
        "step_time_stats": step_stats,
        "ms_per_step_eager": ms_eager,
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
        "ops": {k: {"ms": op_ms[k], "ms_eager": op_ms_eager[k], "gbps": ob[k] / (op_ms[k] * 1e-3) / 1e9,
                    "bytes": ob[k]} for k in OPS},
        "ops_timing": ("each op alone, HIP graph replays of G calls; ms_eager: events around eager calls"
                       if g_single and not args.no_op_events else "events around eager calls"),
        "roofline": {"bound": "hbm", "op": dom, "achieved": dom_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": dom_gbs / HBM_PEAK_GBS, "traffic": traffic},
        "wall_s_timed": wall,
        "input_gen_s": t_gen,
    }
    if args.step_times:
        out["step_ms"] = step_ms
    if sweep is not None:
        out["sweep"] = sweep
    if not args.no_optimizer:
        out["optimizer"] = optimizer_timing(lib, d, r, dev, 200, cpu=not args.no_cpu_baseline)
    if args.two_m > 0:
        out["two_linear"] = two_linear_timing(lib, d, r, args.two_m, dev, 50, not args.no_cpu_baseline, act)
    if args.ffn_width > 0:
        out["ffn_encode"] = ffn_encode_timing(lib, d, r, args.ffn_width, dev, 20, act, not args.no_cpu_baseline)
    if args.qkv_width > 0 and r <= 64:
        out["decode_qkv"] = decode_qkv_timing(lib, d, r, args.qkv_width, dev, 20, not args.no_cpu_baseline)
    if not args.no_cpu_baseline:
        tokens = args.cpu_tokens or T
        out["cpu_baseline"] = cpu_baseline(d, r, act, min(tokens, T))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
