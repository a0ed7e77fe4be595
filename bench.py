"""Benchmark of the KDA decode step with a 4-bit-mean mixed-precision state.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload decode]

One step = one kda_step call: a decode token for B x H heads with its
write-back (recurrence, outputs, weights, layer-budget allocation, fitted
quantiser, packing).  Workload "decode": B=64 sequences, H=32 heads,
d_k=d_v=128, mean payload 4 bits, widths in [2, 8], normalisation groups of
64 rows; prior state = 512 warm-up decode tokens from the zero state (per-token
write-back), run by the library before timing.  Steps rotate over L
independent layer records (copies of the prior state) so the working set
exceeds the 256 MB last-level cache.  Inputs are resident in HBM before the
timed region.

Prints one JSON line (see the fields below).  Only the "cpu_baseline" leg runs
the CPU oracle: on one sequence of the same workload, from its own warm-up.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBPS = 8000.0
# 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz: one VALU lane-op per lane per clock
# (packed float32 issue is not used: the library is compiled without it)
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# Algorithmic lane-ops of the requantisation kernel: every evaluated clip
# factor costs 5 per element of its 64-column row segment (scale, round,
# clamp, residual fma, square-accumulate fma); every element then costs 6
# (final scale, round, clamp, int conversion, field mask, shift-or into the
# stream).  The number of evaluated candidates is counted by the kernel.
FIT_OPS_PER_ELEMENT = 5
SEG_COLS = 64
FINAL_OPS_PER_ELEMENT = 6
BLOCK_ROWS = 32   # rows of one scale group of a head unit


def kernel_source_hash():
    """Hash of the device-kernel sources (what the counter summaries describe)."""
    from paper_2609_30950_amd.pmc_summary import source_hash
    return source_hash()


def committed_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    e = d.get(workload, {}).get(kernel)
    if not e or e.get("source_hash") != kernel_source_hash():
        return None
    return e["hbm_bytes_per_launch"]


def _oracle_cfg(w, head_units):
    from oracle import step
    return step.Cfg(dk=w.dk, dv=w.dv, G=w.G, mean_bits=w.mean_bits, b_min=w.b_min, b_max=w.b_max,
                    erase=w.erase, unit="head" if head_units else "row")


def _oracle_worker(job):
    """One host process: decode steps of sequence `seq` of the workload for
    about budget_s seconds after its own oracle warm-up; path "mirror" is the
    float32-contract step with its write-back (recurrence, statistics,
    allocation, fitted quantiser), "truth" the float64 recurrence and outputs
    of the same steps.  Returns (state-tokens, seconds)."""
    name, seq, path, budget_s, warm_tokens, head_units = job
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1):   # one thread per process: BLAS pools off
        return _oracle_steps(name, seq, path, budget_s, warm_tokens, head_units)


def _oracle_steps(name, seq, path, budget_s, warm_tokens, head_units):
    from oracle import step
    w = W.WORKLOADS[name]
    if head_units:
        w = W.sized(w, b_min=2, G=w.dk)
    oc = _oracle_cfg(w, head_units)
    base = W.base_rates(w)
    xs = {n: [] for n in ("q", "k", "v", "s", "beta")}
    for t in range(warm_tokens):
        x = W.token(w, t, base=base)
        for n in xs:
            xs[n].append(x[n][seq:seq + 1])
    xs = {n: np.stack(a, axis=1) for n, a in xs.items()}
    st, S = step.warm_state(xs["q"], xs["k"], xs["v"], xs["s"], xs["beta"], oc)
    n = 0
    t0 = time.perf_counter()
    while True:
        x = W.token(w, warm_tokens + n, base=base)
        x = {k: v[seq:seq + 1] for k, v in x.items()}
        if path == "mirror":
            st, _, _ = step.mirror_decode_step(st, x["q"], x["k"], x["v"], x["s"], x["beta"], oc)
        else:
            from oracle import recurrence
            S, _ = recurrence.truth_step_rowform(S, x["q"], x["k"], x["v"], x["s"], x["beta"],
                                                 oc.erase)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return w.H * n, el


def cpu_baseline(name, budget_s=6.0, warm_tokens=32, head_units=False):
    """The CPU oracle on the host's cores (a reported baseline, not a
    target): both oracle paths, on one thread and on all cores with one
    process per sequence (sequences are independent; the layer budget couples
    the heads of one), each timed on decode steps after its own warm-up."""
    import multiprocessing as mp
    import platform
    import subprocess
    ncpu = os.cpu_count() or 1
    nproc = max(1, min(ncpu, 16))
    try:
        model = [l.split(":", 1)[1].strip() for l in
                 subprocess.run(["lscpu"], capture_output=True, text=True).stdout.splitlines()
                 if l.startswith("Model name")][0]
    except Exception:   # lscpu missing or unparsable
        model = platform.processor() or "unknown"
    ctx = mp.get_context("spawn")   # fresh interpreters: nothing of this process's GPU state
    paths = {}
    for path in ("mirror", "truth"):
        tok, sec = _oracle_worker((name, 0, path, budget_s, warm_tokens, head_units))
        one = tok / sec
        with ctx.Pool(nproc) as pool:
            res = pool.map(_oracle_worker, [(name, s, path, budget_s, warm_tokens, head_units)
                                            for s in range(nproc)])
        allc = sum(t / s for t, s in res)
        paths[path] = {"one_thread": one, "all_cores": allc, "processes": nproc}
    w = W.WORKLOADS[name]
    return dict(value=paths["mirror"]["all_cores"], unit="state-tokens/s", cores=nproc,
                kind="oracle",
                sample=f"decode steps of 1 sequence per process ({w.H} heads, {w.dk}x{w.dv} "
                       f"states, {budget_s:g} s each after a {warm_tokens}-token oracle warm-up), "
                       f"float32-contract oracle with its write-back (value), {nproc} processes; "
                       f"also one thread, and the float64 recurrence alone",
                paths=paths, os_cpu_count=ncpu, cpu_model=model)


def run_state32_reference(w, args, K, torch):
    """The same decode step in 32-bit mode (float32 state records, no
    quantiser): the memory-side reference of the step."""
    cfg = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, state32=1)
    L = args.layers
    base = W.base_rates(w)
    n_tok = args.warmup + args.steps
    toks = [{n: torch.from_numpy(a).cuda() for n, a in W.token(w, 1000 + t, base=base).items()}
            for t in range(n_tok)]
    layers = torch.zeros(L, K.record_bytes(cfg) * w.B * w.H, dtype=torch.uint8, device="cuda")
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")

    def run(i):
        x = toks[i]
        K.kda_step(cfg, layers[i % L], x["q"], x["k"], x["v"], x["s"], x["beta"], o, None)

    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for i in range(args.warmup, n_tok):
        run(i)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    nbh = w.B * w.H
    step_bytes = nbh * (2 * w.dk * w.dv * 4 + 4 * (3 * w.dk + w.dv) + 4 + 4 * w.dv)
    # context: torch's device copy of the same state bytes (read + write), same rotation
    half = layers.shape[1] // 2
    ev0.record()
    for i in range(args.steps):
        layers[i % L, half:].copy_(layers[(i + 1) % L, :half])
    ev1.record()
    torch.cuda.synchronize()
    copy_ms = ev0.elapsed_time(ev1) / args.steps
    del layers
    return dict(ms_per_step=ms, value=nbh / (ms * 1e-3), unit="state-tokens/s",
                hbm_GBps=step_bytes / (ms * 1e-3) / 1e9,
                hbm_frac=step_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, bytes_per_step=step_bytes,
                device_copy_GBps=2 * half / (copy_ms * 1e-3) / 1e9)


# Chunked prefill: what the apply reads of one chunk record per head at
# d_k = d_v = 128: Wk, Qhat, Ktil^T [64][128] and A [64][64] as bf16 hi and lo
# planes, Uv float32 [64][128], gamma_end float32 [128], Gamma float64 [128]
# and the rate codes u32 [128] (the EMA sums stored beside them are read by
# the rate pass, not by the apply)
CHUNK_RECORD_BYTES = (2 * (3 * 64 * 128 * 2 + 64 * 64 * 2) + 64 * 128 * 4 + 128 * 4
                      + 128 * 8 + 128 * 4)
MFMA_BF16_PEAK_TFLOPS = 2500.0


def chunk_mfma_flops(dk):
    """bf16 MFMA flops issued per chunk and head (16x16x32 tiles, 16384 flops
    each; operands split into hi and lo parts take three products, or two
    against an exact bf16 operand): prep forms L and A on the ten tiles of the
    lower 16-token blocks (d_k / 32 steps each, three products), T diag(beta)
    V (two) and T diag(beta) Khat (three) on six tile rows x d_k / 16
    columns; apply forms Wk S0 and Qhat S0 (4 x d_v/16 tiles, d_k / 32
    steps), A U (six tile rows) and Ktil^T U (d_k/16 x d_v/16 tiles, two
    steps), three products each."""
    t = 16 * 16 * 32 * 2
    prep = 3 * 10 * 2 * (dk // 32) * t + (2 + 3) * 6 * (dk // 16) * t
    apply_ = 3 * (2 * 4 * (dk // 16) * (dk // 32) + 6 * (dk // 16) + (dk // 16) * (dk // 16) * 2) * t
    return prep, apply_


def run_prefill(args, K, torch):
    """Prefill of the bf16 workload (B=4 H=32 d=128 T=8192, write-back every
    64 tokens) from the empty state: one kda_prefill call per pass; with
    --chunked, in the chunked (WY/UT, bf16 MFMA) form."""
    w = W.WORKLOADS["prefill"]
    cfg = K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                   b_min=w.b_min, b_max=w.b_max, chunked=int(args.chunked))
    t0 = time.time()
    xs = W.tokens(w, 0, w.T)
    print(f"# prefill inputs generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    dev = {n: torch.from_numpy(np.ascontiguousarray(xs[n])).cuda() for n in ("s", "beta")}
    for n in ("q", "k", "v"):
        dev[n] = torch.from_numpy(np.ascontiguousarray(xs[n])).to(torch.bfloat16).cuda()
    del xs
    recs = K.new_records(cfg)
    ws = K.new_workspace(cfg)
    o = torch.zeros(w.B * w.T * w.H * w.dv, dtype=torch.float32, device="cuda")
    # the chunked form prepares later chunks on a second stream of ours
    aux = torch.cuda.Stream() if args.chunked else None

    def run():
        recs.zero_()
        K.kda_prefill(cfg, w.T, w.C, recs, dev["q"], dev["k"], dev["v"], dev["s"], dev["beta"], o, ws,
                      aux_stream=aux)

    run()
    torch.cuda.synchronize()
    K.kda_profile_enable(K.api.PROFILE_EVENTS)
    K.kda_profile_read()
    run()
    torch.cuda.synchronize()
    prof = K.kda_profile_read()
    K.kda_profile_enable(0)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    reps = max(1, args.steps // 20)
    ev0.record()
    for _ in range(reps):
        run()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / reps
    nbh = w.B * w.H
    head_tok = 3 * 2 * w.dk + 4 * w.dk + 4 + 4 * w.dv          # q, k, v bf16; s; beta; o
    meta = 16 + w.dk // 2 + 6 * w.dk
    wb = -(-w.T // w.C)
    rec_bytes = 2 * wb * nbh * (meta + w.mean_bits * w.dk * w.dv / 8)
    total = nbh * w.T * head_tok + rec_bytes
    kern = {k: dict(ms_avg=v[0] / v[1], launches=v[1]) for k, v in prof.items()}
    # recurrence lane-ops: a S, k.S', S + g w, q.S per element and token
    rec_ops = 4.0 * nbh * w.T * w.dk * w.dv
    t_stats = prof["stats"][0] * 1e-3 if "stats" in prof else None
    out = {
        "metric": "state-tokens/s (B·H·T), KDA prefill w/ 4-bit mixed state (write-back every 64)",
        "value": nbh * w.T / (ms * 1e-3),
        "unit": "state-tokens/s",
        "n_gpus": 1, "steps": reps, "warmup": 1, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"prefill B={w.B} H={w.H} d_k=d_v={w.dk} T={w.T} C={w.C}, bf16 "
                               f"q/k/v, mean {w.mean_bits} bits, widths [{w.b_min},{w.b_max}], "
                               f"groups of {w.G} rows, layer budget, from the empty state"
                               + (", chunked (WY/UT) form on bf16 MFMA" if args.chunked else
                                  ", token-sequential float32 recurrence")},
        "hbm_GBps_step": total / (ms * 1e-3) / 1e9,
        "hbm_frac_step": total / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "bytes_per_step": total,
        "kernels": kern,
        "kernel_source_hash": kernel_source_hash(),
    }
    if args.chunked and "apply" in prof:
        # apply moves per head: its chunk record, the record's code words at
        # the budgeted payload and metadata, the outputs and the float32 state
        nch = -(-w.T // w.C)
        per_head = (CHUNK_RECORD_BYTES + w.mean_bits * w.dk * w.dv / 8 + meta
                    + w.C * w.dv * 4 + w.dk * w.dv * 4)
        t_apply = prof["apply"][0] / prof["apply"][1] * 1e-3
        ach = nbh * per_head / t_apply / 1e9
        out["roofline"] = dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBPS, unit="GB/s",
                               frac=ach / HBM_PEAK_GBPS, traffic=committed_traffic("apply", "prefill_chunked"),
                               kernel="apply", bytes_per_launch=nbh * per_head)
        fp, fa = chunk_mfma_flops(w.dk)
        t_prep = prof["prep"][0] / prof["prep"][1] * 1e-3
        chunks_per_prep = nbh * nch / prof["prep"][1]
        out["mfma"] = {
            "prep": dict(tflops=fp * chunks_per_prep / t_prep / 1e12,
                         frac=fp * chunks_per_prep / t_prep / 1e12 / MFMA_BF16_PEAK_TFLOPS),
            "apply": dict(tflops=fa * nbh / t_apply / 1e12,
                          frac=fa * nbh / t_apply / 1e12 / MFMA_BF16_PEAK_TFLOPS),
            "peak_tflops": MFMA_BF16_PEAK_TFLOPS}
        # the same two kernels against HBM: prep reads a chunk's inputs and
        # writes its record (less the Gamma and rate codes the rate chain adds)
        prep_bytes = (3 * w.C * w.dk * 2 + w.C * w.dk * 4 + w.C * 4
                      + CHUNK_RECORD_BYTES - w.dk * 12 + 4 * w.dk * 8)
        pg = prep_bytes * chunks_per_prep / t_prep / 1e9
        out["hbm"] = {"apply": dict(GBps=ach, frac=ach / HBM_PEAK_GBPS, bytes_per_launch=nbh * per_head),
                      "prep": dict(GBps=pg, frac=pg / HBM_PEAK_GBPS,
                                   bytes_per_launch=prep_bytes * chunks_per_prep),
                      "peak_GBps": HBM_PEAK_GBPS}
        out["metric"] = out["metric"].replace("prefill", "chunked prefill")
    elif t_stats:
        ach = rec_ops / t_stats / 1e12
        out["roofline"] = dict(bound="alu", achieved=ach, peak=VALU_PEAK_TOPS, unit="TOP/s",
                               frac=ach / VALU_PEAK_TOPS, traffic=committed_traffic("stats", "prefill"),
                               kernel="stats", lane_ops_per_pass=rec_ops)
    print(json.dumps(out), flush=True)


def kcfg(K, w, **kw):
    """Library config of workload w."""
    return K.Config(B=w.B, H=w.H, d_k=w.dk, d_v=w.dv, group_rows=w.G, mean_bits=w.mean_bits,
                    b_min=w.b_min, b_max=w.b_max, decay_per_head=int(w.decay == "head"),
                    no_erase=int(not w.erase), **kw)


# float64 lane-ops of the exact Gramian recursion per matrix element and token:
# X = q q^T + M, u += X k, two rank-one corrections, the decay product d_i d_j
# and its multiply
EXACT_OPS_PER_ELEMENT = 6


def run_weights(args, K, torch):
    """Window weights of the long-context layer (B=128 H=32 d=128, W=1024):
    the exact Gramian recursion (kda_weights_exact, dominant) and the
    diagonal-erase estimate (kda_weights), one call each per pass."""
    w = W.WORKLOADS["long"]
    Wn = w.window
    t0 = time.time()
    xs = W.tokens(W.sized(w, B=2), 0, Wn)
    print(f"# weights inputs (2 sequences, tiled to {w.B}) in {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    rep = w.B // 2
    dev = {n: torch.from_numpy(np.ascontiguousarray(a)).cuda().repeat(
        (rep,) + (1,) * (a.ndim - 1)).contiguous() for n, a in xs.items()}
    del xs
    cfg = kcfg(K, w)
    g = torch.zeros(w.B * w.H * w.dk, dtype=torch.float64, device="cuda")

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        K.kda_profile_enable(K.api.PROFILE_EVENTS)
        K.kda_profile_read()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(reps):
            fn()
        ev1.record()
        torch.cuda.synchronize()
        prof = K.kda_profile_read()
        K.kda_profile_enable(0)
        return ev0.elapsed_time(ev1) / reps, prof["weights"][0] / prof["weights"][1]

    reps = max(2, args.steps // 20)
    ms_exact, k_exact = timed(lambda: K.kda_weights_exact(
        cfg, Wn, 1, dev["q"], dev["s"], dev["beta"], dev["k"], g), reps)
    ms_diag, k_diag = timed(lambda: K.kda_weights(
        cfg, Wn, 1, dev["q"], dev["s"], dev["beta"], dev["k"], g), reps)
    nbh = w.B * w.H
    ops = float(EXACT_OPS_PER_ELEMENT) * nbh * (Wn - 1) * w.dk * w.dk
    ach = ops / (k_exact * 1e-3) / 1e12
    in_bytes = nbh * Wn * (4 * w.dk * 3 + 4)          # q, k, s, beta
    out = {
        "metric": "head-windows/s, exact Gramian row weights (1024-token window)",
        "value": nbh / (ms_exact * 1e-3), "unit": "head-windows/s",
        "n_gpus": 1, "steps": reps, "warmup": 1, "ms_per_step": ms_exact,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"weights B={w.B} H={w.H} d_k={w.dk} W={Wn} C=1, long-context "
                               f"inputs (2 sequences tiled)"},
        "diagonal_estimate_ms": ms_diag,
        "diagonal_estimate_hbm_GBps": in_bytes / (k_diag * 1e-3) / 1e9,
        "roofline": dict(bound="alu", achieved=ach, peak=VALU_PEAK_TOPS, unit="TOP/s",
                         frac=ach / VALU_PEAK_TOPS, traffic=None, kernel="weights (exact)",
                         lane_ops_per_launch=ops),
        "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="decode",
                    choices=["decode", "prefill", "mamba2", "weights", "gdn2", "gdn6", "long"])
    ap.add_argument("--layers", type=int, default=20)
    ap.add_argument("--warm-tokens", type=int, default=512)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-count-pass", action="store_true",
                    help="skip the untimed counting replay (e.g. under a profiler)")
    ap.add_argument("--no-ref32", action="store_true",
                    help="skip the 32-bit-mode reference step")
    ap.add_argument("--graph", action="store_true",
                    help="decode workloads: also time the steps replayed from one HIP graph")
    ap.add_argument("--head-units", action="store_true",
                    help="decode workloads: one width per head with block scales")
    ap.add_argument("--chunked", action="store_true",
                    help="prefill workload: chunked (WY/UT) form on bf16 MFMA")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(sequences shard across GPUs without communication)",
              file=sys.stderr)
        sys.exit(2)

    # the CPU oracle first, in host processes started before this process
    # touches the GPU (decode workloads)
    cpu = None
    if not args.no_cpu_baseline and args.workload not in ("prefill", "weights"):
        cpu = cpu_baseline(args.workload, head_units=args.head_units)
        print(f"# cpu baseline: {cpu['paths']}", file=sys.stderr, flush=True)

    import torch
    import paper_2609_30950_amd as K

    torch.cuda.set_device(0)
    if args.workload == "prefill":
        run_prefill(args, K, torch)
        return
    if args.workload == "weights":
        run_weights(args, K, torch)
        return
    w = W.WORKLOADS[args.workload]
    if args.head_units:
        # one width per head, block scales: per-head normalisation, b_min = 2
        w = W.sized(w, b_min=2, G=w.dk)
    cfg = kcfg(K, w, head_units=int(args.head_units))
    ws = K.new_workspace(cfg)
    o = torch.zeros(w.B * w.H * w.dv, dtype=torch.float32, device="cuda")
    base = W.base_rates(w)
    # prior state: warm-up decode tokens from the zero state, on the GPU
    t0 = time.time()
    prior = K.new_records(cfg)
    for t in range(args.warm_tokens):
        x = {n: torch.from_numpy(a).cuda() for n, a in W.token(w, t, base=base).items()}
        K.kda_step(cfg, prior, x["q"], x["k"], x["v"], x["s"], x["beta"], o, ws)
    torch.cuda.synchronize()
    print(f"# prior state: {args.warm_tokens} warm-up decode tokens in {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    L = args.layers
    layers = prior.repeat(L).view(L, -1)
    del prior
    n_tok = args.warmup + args.steps
    toks = [W.token(w, args.warm_tokens + t, base=base) for t in range(n_tok)]
    dtoks = [{n: torch.from_numpy(a).cuda() for n, a in x.items()} for x in toks]

    def run(i):
        x = dtoks[i]
        K.kda_step(cfg, layers[i % L], x["q"], x["k"], x["v"], x["s"], x["beta"], o, ws)

    for i in range(args.warmup):
        run(i)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)

    def timed():
        torch.cuda.synchronize()
        ev0.record()
        for i in range(args.warmup, n_tok):
            run(i)
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / args.steps

    snapshot = layers.clone()          # records before the timed steps
    # pass A: per-kernel HIP events recorded by the library on the launch
    # stream around every kernel (kernel durations; the events add idle gaps
    # between kernels, so the step time of this pass is reported separately)
    K.kda_profile_enable(K.api.PROFILE_EVENTS)
    K.kda_profile_read()
    ms_events = timed()
    prof = K.kda_profile_read()
    K.kda_profile_enable(0)
    # pass B: the same steps from the same records without events -> value
    layers.copy_(snapshot)
    ms = timed()
    ms_graph = None
    if args.graph:
        # pass G: the same steps captured in one HIP graph and replayed
        layers.copy_(snapshot)
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            run(args.warmup)                   # warm-up launch outside the capture
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        layers.copy_(snapshot)
        with torch.cuda.graph(g):
            for i in range(args.warmup, n_tok):
                run(i)
        torch.cuda.synchronize()
        layers.copy_(snapshot)
        ev0.record()
        g.replay()
        ev1.record()
        torch.cuda.synchronize()
        ms_graph = ev0.elapsed_time(ev1) / args.steps
        del g
    # pass C (untimed): the same launches once more with the quantiser's
    # evaluation counter on, for the algorithmic work of pass A's launches
    fit_evals = None
    if not args.no_count_pass:
        layers.copy_(snapshot)
        K.kda_profile_enable(K.api.PROFILE_COUNTERS)
        K.kda_profile_counters()
        for i in range(args.warmup, n_tok):
            run(i)
        fit_evals = K.kda_profile_counters()
        K.kda_profile_enable(0)
    del snapshot

    kern = {k: dict(ms_avg=v[0] / v[1], launches=v[1]) for k, v in prof.items()}
    dom = max(prof, key=lambda k: prof[k][0])
    elems = w.B * w.H * w.dk * w.dv
    # algorithmic HBM bytes of one step: records read and written (metadata
    # plus the budgeted code bits), inputs q, k, v, s, beta and outputs o
    meta = 16 + w.dk // 2 + 6 * w.dk
    if args.head_units:
        meta = 16 + 4 * w.dk + (w.dk // 32) * w.dv * 2   # rate codes, erase rates, block scales
    code_bytes = w.mean_bits * elems / 8
    s_elems = 1 if w.decay == "head" else w.dk
    io = w.B * w.H * (4 * (w.dk * 2 + s_elems + w.dv) + 4 + 4 * w.dv)   # q k s v beta, o
    step_bytes = 2 * (w.B * w.H * meta + code_bytes) + io
    hbm = step_bytes / (ms * 1e-3) / 1e9
    evals_per_launch = (fit_evals or 0) / max(1, kern.get("requant", {}).get("launches", 1))
    rows = w.B * w.H * w.dk
    segs = rows * (w.dv // SEG_COLS)
    if dom == "requant" and fit_evals is not None:
        t_dom = kern[dom]["ms_avg"] * 1e-3
        ops = evals_per_launch * SEG_COLS * FIT_OPS_PER_ELEMENT + elems * FINAL_OPS_PER_ELEMENT
        achieved = ops / t_dom / 1e12
        roof = dict(bound="alu", achieved=achieved, peak=VALU_PEAK_TOPS, unit="TOP/s",
                    frac=achieved / VALU_PEAK_TOPS,
                    traffic=committed_traffic("requant", args.workload), kernel="requant",
                    lane_ops_per_launch=ops,
                    candidates_per_row_segment=evals_per_launch / segs)
    elif dom == "step" and args.head_units and fit_evals is not None:
        # head units: the step kernel fits every (32-row block, column) group
        # with the same candidates, 5 lane-ops per element each, then codes it
        t_dom = kern[dom]["ms_avg"] * 1e-3
        evals = fit_evals / max(1, kern[dom]["launches"])
        ops = evals * BLOCK_ROWS * FIT_OPS_PER_ELEMENT + elems * FINAL_OPS_PER_ELEMENT
        achieved = ops / t_dom / 1e12
        roof = dict(bound="alu", achieved=achieved, peak=VALU_PEAK_TOPS, unit="TOP/s",
                    frac=achieved / VALU_PEAK_TOPS, traffic=None, kernel="step",
                    lane_ops_per_launch=ops,
                    candidates_per_block=evals / (elems / BLOCK_ROWS))
    else:
        t_dom = kern[dom]["ms_avg"] * 1e-3
        roof = dict(bound="hbm", achieved=step_bytes / t_dom / 1e9, peak=HBM_PEAK_GBPS,
                    unit="GB/s", frac=step_bytes / t_dom / 1e9 / HBM_PEAK_GBPS,
                    traffic=committed_traffic(dom, args.workload), kernel=dom)

    out = {
        "metric": f"state-tokens/s (B·H·T) and achieved HBM GB/s, KDA step w/ {w.mean_bits:g}-bit mixed state",
        "value": w.B * w.H / (ms * 1e-3),
        "unit": "state-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_with_kernel_events": ms_events,
        "ms_per_step_hip_graph": ms_graph,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": ("" if w.name == "decode" else f"{w.name} ")
                               + f"decode step B={w.B} H={w.H} d_k=d_v={w.dk}, mean "
                               f"{w.mean_bits} bits, widths [{w.b_min},{w.b_max}], groups of "
                               f"{w.G} rows, layer budget, "
                               f"{'per-head' if w.decay == 'head' else 'per-channel'} decay, "
                               f"{'KDA erase' if w.erase else 'no erasure'}, "
                               + ("head units (one width per head, FP16 scales per 32 rows "
                                  "of a column), " if args.head_units else "")
                               + f"prior state after {args.warm_tokens} warm-up decode tokens",
                   "layers_rotated": L},
        "hbm_GBps_step": hbm,
        "hbm_frac_step": hbm / HBM_PEAK_GBPS,
        "bytes_per_step": step_bytes,
        "kernels": kern,
        "kernel_source_hash": kernel_source_hash(),
        "roofline": roof,
    }
    if not args.no_ref32 and w.name == "decode":
        del layers
        out["state32_reference"] = run_state32_reference(w, args, K, torch)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
