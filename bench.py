"""Benchmark of the gated delta-rule hot path on one MI355X.

Default workload: chunked prefill of one recurrent layer, B=1, T=10240, H=16,
dk=dv=128, chunk 64, bf16 q/k/v/o with fp32 gates and state (the paper's
16 value heads with H_k = H_v = 128, section 2.2, at its 10k-token tier).
A step is one gdn_chunk_prefill call over the whole prompt (every kernel of
the path).  Prints ONE JSON line on stdout.

Inputs are resident in HBM before timing starts; each step reads a different
one of ``--sets`` input sets (4 x 171 MB by default, larger than the 256 MB
Infinity Cache), so no step finds its inputs in cache from the previous one.
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

PEAK = {"hbm": 8.0e12, "bf16": 2.5e15, "f32": 157.3e12}   # MI355X published peaks


def algorithmic(w, lens, dk, dv, H, io, s0, decode=False, chunk=64):
    """Bytes and flops the method must move / perform (no padding, no re-reads), for chunks of ``chunk`` tokens."""
    s_io = 2 if io == "bf16" else 4
    ntok = sum(lens)
    if decode:
        n = len(lens)
        byts = n * H * ((2 * dk + 2 * dv) * s_io + 8 + 2 * 4 * dv * dk)
        flops = n * H * 6 * dk * dv
        return byts, flops
    byts = ntok * H * ((2 * dk + 2 * dv) * s_io + 8) + len(lens) * H * 4 * dv * dk * (2 if s0 else 1)
    flops = 0
    for L in lens:
        for c0 in range(0, L, chunk):
            n = min(chunk, L - c0)
            flops += (n * (n - 1) * dk + n * (n + 1) * dk + n * (n - 1) * (dk + dv) + n * (n + 1) * dv
                      + 6 * n * dk * dv)
    return byts, flops * H


def kernel_source_sha():
    """sha256 over the library's kernel sources (every file of csrc/, in name order)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_14568_amd", "csrc")
    for fn in sorted(os.listdir(csrc)):
        h.update(fn.encode())
        h.update(open(os.path.join(csrc, fn), "rb").read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per call from the committed rocprofv3 counter summary, if it was taken on this kernel source."""
    path = os.path.join(ROOT, "profiles", "%s_traffic.md" % workload)
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    sha = kernel_source_sha()
    if fields.get("kernel source sha256") != sha or "HBM bytes per call" not in fields:
        return None
    return float(fields["HBM bytes per call"])


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, x, budget_s):
    """The fp64 oracle, as it stands, on this host's cores, on the same inputs; and on one thread."""
    import oracle
    from paper_2607_14568_amd import inputs as I
    f = I.as_f64
    if w.decode:
        args = [f(x[k][0]) for k in ("q", "k", "v", "g", "beta")]
        S = f(x["S"])
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.decode_step(*args, S)
            reps += 1
            el = time.perf_counter() - t0
            if el > budget_s or reps >= 1000:
                break
        tok = reps * w.B
        sample = "%d decode steps of the %d-sequence batch" % (reps, w.B)
    else:
        cu = None if x["cu_seqlens"] is None else x["cu_seqlens"].numpy()
        args = [f(x[k]) for k in ("q", "k", "v", "g", "beta")]
        S0 = f(x["S0"])
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.recurrence(*args, S0, cu_seqlens=cu)
            reps += 1
            el = time.perf_counter() - t0
            if el > budget_s:
                break
        tok = reps * int(x["q"].shape[0] * x["q"].shape[1])
        sample = "%d full call(s) of the same workload (all %d heads)" % (reps, w.H)
    out = {"value": tok / el, "unit": "tokens/s", "cores": oracle.max_threads(), "kind": "oracle",
           "sample": sample, "seconds": round(el, 3), "cpu_model": cpu_model()}
    # one thread: a prefix of the same inputs (a bounded sample, a few seconds)
    if w.decode:
        t0 = time.perf_counter()
        oracle.decode_step(*args, S, n_threads=1)
        el1, tok1 = time.perf_counter() - t0, w.B
        sample1 = "one decode step of the %d-sequence batch" % w.B
    elif x["cu_seqlens"] is None:
        n1 = min(int(x["q"].shape[1]), 512)
        a1 = [a[:1, :n1] for a in args]
        t0 = time.perf_counter()
        oracle.recurrence(*a1, None if S0 is None else S0[:1], n_threads=1)
        el1, tok1 = time.perf_counter() - t0, n1
        sample1 = "the first %d tokens of one sequence (all %d heads)" % (n1, w.H)
    else:
        el1, tok1, sample1 = None, None, None
    if el1:
        out["value_1thread"] = tok1 / el1
        out["sample_1thread"] = sample1
    return out


ATTN = {   # causal attention prefill workloads (the backbone's softmax-attention layers): B, T, H, H_kv, d
    "attn_10k_bf16": (1, 10240, 16, 8, 128),
    "attn_2k_bf16": (1, 2048, 16, 8, 128),
}


def attention_bench(args):
    """Causal attention prefill: one gdn_attention_prefill call per step over the whole prompt."""
    import numpy as np
    import torch
    import paper_2607_14568_amd as gdn
    from paper_2607_14568_amd import inputs as I

    B, T, H, Hkv, d = ATTN[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    x_host = I.make_attention(B, T, H, Hkv, d, seed=1005)
    sets = []
    for i in range(max(1, args.sets)):
        dd = {kk: vv.to(dev) for kk, vv in x_host.items()}
        if i > 0:
            dd = {kk: vv.clone() for kk, vv in dd.items()}
        dd["o"] = torch.empty_like(dd["q"])
        sets.append(dd)
    scale = 1.0 / d ** 0.5

    def step(i):
        dd = sets[i % len(sets)]
        gdn.gdn_attention_prefill(dd["q"], dd["k"], dd["v"], scale=scale, o=dd["o"])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(args.warmup + i)
    ev1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t0
    avg_call_s = ev0.elapsed_time(ev1) / args.steps * 1e-3
    ms_per_step = t_wall * 1e3 / args.steps
    flops = 2.0 * d * H * B * T * (T + 1)                 # Q K^T and P V over each query's causal prefix
    byts = B * T * (2 * H + 2 * Hkv) * d * 2              # q, k, v read, o written (bf16)
    roof = {"bound": "mfma", "achieved": flops / avg_call_s / 1e12, "peak": PEAK["bf16"] / 1e12, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None
    roof["kernel"] = "one gdn_attention_prefill call (k_attn_causal)"
    roof["alg_flops"] = flops
    roof["alg_bytes"] = byts
    roof["avg_call_us"] = avg_call_s * 1e6
    out = {
        "metric": "causal softmax-attention prefill tokens/s (T=%d, H=%d, H_kv=%d, d=%d); %% of roofline" % (T, H, Hkv, d),
        "value": B * T / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "B": B, "T": T, "H": H, "H_kv": Hkv, "d": d, "io": "bf16",
                   "parallelism": "none (1 GPU)", "input_sets": len(sets)},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        from oracle import attention as att
        f = I.as_f64
        q, k, v = f(x_host["q"]), f(x_host["k"]), f(x_host["v"])
        rng = np.random.default_rng(0)
        done, t0 = 0, time.perf_counter()
        while True:   # query rows drawn uniformly: their mean cost is the mean cost of a token
            rows = np.sort(rng.integers(0, T, 32))
            att.causal_attention(q, k, v, scale, rows=rows)
            done += len(rows)
            el = time.perf_counter() - t0
            if el > args.cpu_budget:
                break
        try:   # the threads numpy's BLAS ran the oracle's products on
            from threadpoolctl import threadpool_info
            cores = max([pi.get("num_threads", 1) for pi in threadpool_info() if pi.get("user_api") == "blas"] or [1])
        except Exception:
            cores = None
        out["cpu_baseline"] = {"value": done * B / el, "unit": "tokens/s", "cores": cores, "kind": "oracle",
                               "sample": "%d query rows drawn uniformly from the %d-token prompt (all %d heads)"
                                         % (done, T, H), "seconds": round(el, 3)}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="prefill_10k_bf16")
    ap.add_argument("--sets", type=int, default=4, help="rotating resident input sets")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--plan", default="auto", choices=["auto", "seq", "seg", "wide"],
                    help="evaluation plan of the prefill (auto: the library chooses)")
    ap.add_argument("--chunk", type=int, default=64, choices=[16, 32, 64, 128],
                    help="chunk length of the prefill (64: the tuned kernels; others: the generic path)")
    ap.add_argument("--segments", type=int, default=0,
                    help="segments per sequence of a segmented plan (0: the plan's own count)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run one plain device copy of MIB MiB before timing (scale for rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the benchmark runs on exactly one GPU; --gpus %d is not supported "
              "(sharding across GPUs is described, not implemented)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    if args.workload in ATTN:
        return attention_bench(args)

    import torch
    import paper_2607_14568_amd as gdn
    from paper_2607_14568_amd import inputs as I

    if not os.path.exists(gdn.LIB_PATH):
        from paper_2607_14568_amd import build as B
        B.build_library(force=True)
    w = I.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    plan_flags = {"auto": 0, "seq": gdn.GDN_PLAN_SEQUENTIAL, "seg": gdn.GDN_PLAN_SEGMENTED,
                  "wide": gdn.GDN_PLAN_WIDE}[args.plan]
    stream = torch.cuda.current_stream(dev)

    x_host = I.make_workload(args.workload)
    sets = []
    for i in range(max(1, args.sets)):
        d = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in x_host.items()}
        if i > 0:   # distinct buffers with the same values (the parity tests cover the values)
            d = {k: (v.clone() if isinstance(v, torch.Tensor) else v) for k, v in d.items()}
        sets.append(d)

    if w.decode:
        lens = [1] * w.B
        for d in sets:
            d["S"] = d["S"].clone()
            d["o"] = torch.empty_like(d["v"][0])

        def step(i):
            d = sets[i % len(sets)]
            j = i % d["q"].shape[0]
            gdn.gdn_decode_step(d["q"][j], d["k"][j], d["v"][j], d["g"][j], d["beta"][j], d["S"], o=d["o"])
    else:
        cu = x_host["cu_seqlens"]
        lens = [int(a) for a in (cu[1:] - cu[:-1])] if cu is not None else [w.T] * w.B
        n_seqs = 0 if cu is None else len(lens)
        io_code = gdn.GDN_BF16 if w.io == "bf16" else gdn.GDN_F32
        B_, T_ = x_host["q"].shape[0], x_host["q"].shape[1]
        need = gdn.gdn_chunk_prefill_workspace_bytes_ex(B_, T_, w.H, w.dk, w.dv, args.chunk, n_seqs, io_code,
                                                        plan_flags, args.segments)
        if need == 0 and T_ > 0:
            print("bench.py: chunk=%d does not take plan %s" % (args.chunk, args.plan), file=sys.stderr)
            sys.exit(2)
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
        if args.chunk == 64:
            form, segments = gdn.gdn_chunk_prefill_plan(B_, T_, w.H, w.dk, w.dv, n_seqs, io_code, plan_flags,
                                                        args.segments, need)
        else:   # other chunk lengths: the generic path, sequential
            form, segments = gdn.GDN_PLAN_SEQUENTIAL, 1
        for d in sets:
            d["o"] = torch.empty_like(d["v"])
            d["S_T"] = torch.empty_like(d["S0"]) if d["S0"] is not None else None

        def step(i):
            d = sets[i % len(sets)]
            gdn.gdn_chunk_prefill_ex(d["q"], d["k"], d["v"], d["g"], d["beta"], d["S0"], flags=plan_flags,
                                     segments=args.segments, chunk=args.chunk, cu_seqlens=d["cu_seqlens"], o=d["o"],
                                     S_T=d["S_T"], workspace=ws)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    if args.copy_calibration > 0:   # a copy of known size: its FETCH_SIZE / WRITE_SIZE calibrate the counters
        src = torch.empty(args.copy_calibration << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # average call duration: HIP events on the stream the library launches on, around the whole timed region
    # (events between calls would add their own gaps to calls of a few microseconds)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(args.warmup + i)
    ev1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall0
    ms_per_step = t_wall * 1e3 / args.steps
    avg_call_s = ev0.elapsed_time(ev1) / args.steps * 1e-3

    ntok = sum(lens)
    value = ntok / (ms_per_step * 1e-3)
    byts, flops = algorithmic(w, lens, w.dk, w.dv, w.H, w.io, w.s0_std > 0, decode=w.decode, chunk=args.chunk)
    t_hbm = byts / PEAK["hbm"]
    t_mfma = flops / PEAK[w.io]
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    if bound == "hbm":
        roof = {"bound": "hbm", "achieved": byts / avg_call_s / 1e9, "peak": PEAK["hbm"] / 1e9, "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": flops / avg_call_s / 1e12, "peak": PEAK[w.io] / 1e12,
                "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None if (w.decode or args.chunk != 64) else measured_traffic(w.name)
    if w.decode:
        roof["kernel"] = "one gdn_decode_step call"
    elif form == gdn.GDN_PLAN_WIDE:
        roof["kernel"] = ("one gdn_chunk_prefill call, wide segment-parallel form with %d segments (chunk terms, "
                          "segment states, scan, output pass: four launches)" % segments)
    elif args.chunk != 64:
        roof["kernel"] = ("one gdn_chunk_prefill call at chunk %d, generic path (decay-masked products, forward "
                          "substitution, chain: three launches)" % args.chunk)
    elif segments > 1:
        roof["kernel"] = ("one gdn_chunk_prefill call, segment-parallel form with %d segments (segment "
                          "setup, chunk terms, paired chain, scan, output pass)" % segments)
    elif w.io == "bf16":
        roof["kernel"] = "one gdn_chunk_prefill call, sequential form (k_prefill_fused_bf16, or chunk terms + chain)"
    else:
        roof["kernel"] = "one gdn_chunk_prefill call, sequential form (k_chunk_terms + k_state_chain)"
    roof["alg_bytes"] = byts
    roof["alg_flops"] = flops
    roof["avg_call_us"] = avg_call_s * 1e6

    out = {
        "metric": "gated-delta-rule prefill tokens/s at T=10240,H=16,d=128; % of roofline",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.io, "data": "synthetic",
        "config": {"workload": w.name, "B": len(lens) if w.ragged else w.B, "T": ntok if w.ragged else w.T,
                   "H": w.H, "dk": w.dk, "dv": w.dv, "chunk": args.chunk, "io": w.io, "state": "fp32",
                   "parallelism": "none (1 GPU)", "input_sets": len(sets)},
        "roofline": roof,
    }
    if not w.decode:
        out["config"]["plan"] = {gdn.GDN_PLAN_SEQUENTIAL: "sequential", gdn.GDN_PLAN_SEGMENTED: "segmented",
                                 gdn.GDN_PLAN_WIDE: "wide"}.get(form, "?")
        out["config"]["segments"] = segments
    if w.decode:
        out["metric"] = "gated-delta-rule decode-step tokens/s (B=%d,H=%d,d=%d)" % (w.B, w.H, w.dk)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, x_host, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
