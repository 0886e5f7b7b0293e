"""Benchmark of the CE-Router routed block on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload N] [--no-cpu-baseline]

One step = one fused routed block (ce_routed_block: core/expansion scoring ->
per-sequence TopK -> SwiGLU FFN on the retained rows -> residual scatter) over
the whole synthetic batch, in place, with inputs resident in HBM. Every timed
step works on its own pristine copy of the hidden states, and weight sets
rotate so that they exceed twice the 256 MB last-level cache. Prints ONE JSON
line (rank 0, one GPU).

`value` = input tokens per second (every token of the batch is routed: scored,
then kept or bypassed). The roofline entry covers the dominant kernel, the
gate/up + SwiGLU GEMM, timed per launch with HIP events on the stream it runs
on; its HBM traffic comes from the committed rocprofv3 counter summary when
that summary matches the current kernel source, else null.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "routed tokens/sec per layer (score+topk+FFN+scatter); % MFMA / HBM peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0
MALL_BYTES = 256 << 20
# HBM traffic of the gate/up GEMM per workload, from rocprofv3 counter runs
TRAFFIC_FILES = {2: "ffn_gateup_showo2_understanding_traffic.txt", 4: "ffn_gateup_7b_mixed_varlen_traffic.txt"}
KERNEL_SOURCES = ["paper_2608_29291_amd/csrc/ce_ffn.hip", "paper_2608_29291_amd/csrc/ce_device.hpp"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(wid: int):
    """HBM bytes per gate/up launch from the committed counter summary of this
    workload, if it was taken on the current kernel source (else None)."""
    if wid not in TRAFFIC_FILES:
        return None
    try:
        with open(os.path.join(ROOT, "profiles", TRAFFIC_FILES[wid])) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith(" "))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("kernel_source_hash") != kernel_source_hash():
        return None
    try:
        return int(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, n_seq: int, min_seconds: float = 10.0, max_reps: int = 50):
    """The oracle (float64 NumPy) on the first n_seq sequences, repeated until
    about min_seconds of CPU work; reports tokens per second over all runs."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
                      or [1])
    except Exception:  # pragma: no cover - threadpoolctl missing
        threads = os.cpu_count() or 1
    hi = int(wl.seq_offsets[n_seq])
    offs = wl.seq_offsets[: n_seq + 1]
    reps, total = 0, 0.0
    while reps < max_reps and (reps == 0 or total < min_seconds):
        t0 = time.perf_counter()
        oracle.routed_block(wl.hidden[:hi], wl.flags[:hi], offs, wl.t[:n_seq], wl.keep, wl.scorer, wl.ffn)
        total += time.perf_counter() - t0
        reps += 1
    return {"value": round(reps * hi / total, 1), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{n_seq} of {wl.B} sequences ({hi} tokens) x {reps} runs, one routed block each "
                      f"in float64 NumPy, {total:.1f} s total on {platform.processor() or platform.machine()} "
                      f"({os.cpu_count()} logical CPUs visible, BLAS threads {threads})"}


def time_drop_stability(ce, stream, reps: int) -> dict:
    """Drop-set Jaccard / RDA between two timesteps (section 3.4, Eq. 10-11) on
    the Show-o2 generation workload's shape: 4 x [4096 latent, 128 text]."""
    import torch
    from ce_workloads import TOK_GEN, TOK_KEEP, make_drop_pair
    offs, flags, tp_t, tp_r = make_drop_pair([[(4096, TOK_GEN), (128, TOK_KEEP)]] * 4, 0.5, 0.5, 0.05, 1)
    up = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to("cuda")
    B, T = len(offs) - 1, int(offs[-1])
    batch = ce.Batch(up(offs), up(flags), up(np.zeros(B, np.float32)), 0.5, 0)
    a, b = up(tp_t), up(tp_r)
    jac, jr, rda = (torch.empty(B, device="cuda") for _ in range(3))
    for _ in range(3):
        ce.ce_drop_stability(batch, a, b, jac, jr, rda, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(20_000_000)  # let the host enqueue every call before the first starts
    e0.record(stream)
    for _ in range(reps):
        ce.ce_drop_stability(batch, a, b, jac, jr, rda, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    return {"drop_stability": {"us_per_call": round(us, 2), "sequences": B, "tokens": T,
                               "bytes_per_call": 9 * T, "bound": "latency",
                               "workload": "showo2-generation shape, adjacent steps"}}


def time_attention(ce, stream, reps: int) -> dict:
    """Routed attention over the packed retained tokens (section 3.4 token
    compaction), at the Show-o2 shapes (12 query heads, 2 key/value heads,
    head_dim 128): understanding prefill over the retained rows of the
    understanding workload (8 x 551, causal, the compressed KV cache's
    prefill) and generation over 4 x [2048 latent + 128 text] retained rows
    (full attention)."""
    import torch
    from ce_workloads import make_attention_inputs
    out = {}
    for name, lens, causal in (("understanding_prefill", [551] * 8, True),
                               ("generation", [2176] * 4, False)):
        q, k, v, qo, ko = make_attention_inputs(lens, lens, 12, 2, 128, seed=3)
        up = lambda x, dt=None: (torch.from_numpy(np.ascontiguousarray(x)).to(dt) if dt is not None
                                 else torch.from_numpy(np.ascontiguousarray(x))).to("cuda")
        dq, dk, dv = up(q, torch.bfloat16), up(k, torch.bfloat16), up(v, torch.bfloat16)
        o = torch.empty_like(dq)
        dqo, dko = up(qo), up(ko)
        for _ in range(3):
            ce.ce_routed_attention(dq, dk, dv, o, dqo, dko, causal, 128 ** -0.5, stream=stream)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20_000_000)
        e0.record(stream)
        for _ in range(reps):
            ce.ce_routed_attention(dq, dk, dv, o, dqo, dko, causal, 128 ** -0.5, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        pairs = sum(n * (n + 1) // 2 if causal else n * n for n in lens)
        flops = 4.0 * 128 * 12 * pairs
        tf = flops / (us * 1e-6) / 1e12
        out[name] = {"us_per_call": round(us, 2), "sequences": len(lens), "rows_per_sequence": lens[0],
                     "causal": causal, "flops_per_call": flops, "bound": "mfma", "achieved_TFLOPs": round(tf, 1),
                     "peak_TFLOPs": PEAK_BF16_TFLOPS, "frac": round(tf / PEAK_BF16_TFLOPS, 4)}
        log(f"attention {name}: {us:.1f} us, {tf:.0f} TFLOP/s")
    return out


def achievable_peaks(kt: int, d: int, f: int) -> dict:
    """Context for the spec peaks, each after about 150 ms of untimed calls
    (the engine clock settles under load): a 1 GiB device-to-device copy (read
    + write bytes per second), an 8192^3 bf16 GEMM through torch (hipBLASLt),
    and torch GEMMs of the FFN shapes ([Kt x d] x [d x 2 d_ff] for gate and up
    together, [Kt x d_ff] x [d_ff x d] for down) without the gather, SwiGLU
    and scatter the routed block fuses."""
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    b = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    x = torch.randn(kt, d, device="cuda").to(torch.bfloat16)
    wgu = torch.randn(d, 2 * f, device="cuda").to(torch.bfloat16)
    hh = torch.randn(kt, f, device="cuda").to(torch.bfloat16)
    wd = torch.randn(f, d, device="cuda").to(torch.bfloat16)
    out = {}
    for name, fn, work, unit in (
            ("device_copy_GBps", lambda: dst.copy_(src), 2.0 * n / 1e9, "rate"),
            ("torch_bf16_gemm_8192_TFLOPs", lambda: torch.matmul(a, b), 2.0 * 8192 ** 3 / 1e12, "rate"),
            ("torch_bf16_gateup_shape_us", lambda: torch.matmul(x, wgu), 0.0, "us"),
            ("torch_bf16_down_shape_us", lambda: torch.matmul(hh, wd), 0.0, "us")):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        per = (time.perf_counter() - t0) / 3
        for _ in range(int(min(2000, max(10, 0.150 / per)))):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(20):
            fn()
        e1.record()
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) / 20 * 1e-3
        out[name] = round(work / sec, 1) if unit == "rate" else round(sec * 1e6, 2)
    log(f"achievable: copy {out['device_copy_GBps']} GB/s, bf16 GEMM {out['torch_bf16_gemm_8192_TFLOPs']} TFLOP/s, "
        f"FFN shapes through torch: gate/up {out['torch_bf16_gateup_shape_us']} us, "
        f"down {out['torch_bf16_down_shape_us']} us")
    del src, dst, a, b, x, wgu, hh, wd
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", type=int, default=4,
                    help="named workload 1..5 (default 4, the largest: 7B width, mixed varlen batch)")
    ap.add_argument("--step3", type=int, default=-1,
                    help="workload 3: one denoising step s (0..49), or -1 (default) for all 50 in turn")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seqs", type=int, default=0,
                    help="sequences in the oracle sample (0 = every sequence of the batch)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 5 plain device-to-device copies of MIB MiB (reference kernel of "
                         "known traffic for the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 5}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the routed block shards by sequence with no exchange between GPUs)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_29291_amd as ce
    from ce_workloads import CONFIG_NAMES, CONFIG_DESCRIPTIONS, make_config

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wid = args.workload
    log(f"generating workload {wid}: {CONFIG_DESCRIPTIONS[wid]}")
    sweep3 = wid == 3 and args.step3 < 0
    wl = make_config(wid, step=(0 if sweep3 else args.step3) if wid == 3 else None)
    bf16 = wl.dtype == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    dtc = ce.CE_BF16 if bf16 else ce.CE_F32
    cap = ce.ce_kept_count_host(wl.seq_offsets, wl.flags, float(wl.keep))
    T, d, F = wl.T, wl.d, wl.d_ff

    def up(x, dtype=None):
        t = torch.from_numpy(np.ascontiguousarray(x))
        return (t.to(dtype) if dtype is not None else t).to(dev)

    batch = ce.Batch(up(wl.seq_offsets), up(wl.flags), up(wl.t), float(wl.keep), cap)
    sw = wl.scorer
    opt = lambda x: None if x is None else up(x.astype(np.float32))
    base_scorer = ce.Scorer(up(sw.w1_core, dt), up(sw.w2_core), up(sw.w1_exp, dt), up(sw.w2_exp),
                            b1_core=opt(sw.b1_core), b2_core=float(sw.b2_core), b1_exp=opt(sw.b1_exp),
                            b2_exp=opt(sw.b2_exp))
    base_ffn = ce.FFN([up(f.w_gate, dt) for f in wl.ffn], [up(f.w_up, dt) for f in wl.ffn],
                      [up(f.w_down, dt) for f in wl.ffn])
    base_h = up(wl.hidden, dt)  # pristine: never written
    elem = 2 if bf16 else 4
    w_bytes = ((sw.r_core + sw.n_seg * sw.r_exp) * d + 3 * d * F * len(wl.ffn)) * elem
    n_sets = max(2, int(np.ceil(2 * MALL_BYTES / w_bytes)))
    log(f"T={T} Kt={cap} d={d} F={F}; rotating {n_sets} weight sets of {w_bytes / 2**20:.0f} MiB")
    wsets = [(base_scorer, base_ffn)]
    for _ in range(n_sets - 1):
        sc = ce.Scorer(*(x.clone() if x is not None else None for x in
                         (base_scorer.w1_core, base_scorer.w2_core, base_scorer.w1_exp, base_scorer.w2_exp,
                          base_scorer.b1_core)), b2_core=base_scorer.b2_core,
                       b1_exp=None if base_scorer.b1_exp is None else base_scorer.b1_exp.clone(),
                       b2_exp=None if base_scorer.b2_exp is None else base_scorer.b2_exp.clone())
        ff = ce.FFN([w.clone() for w in base_ffn.w_gate], [w.clone() for w in base_ffn.w_up],
                    [w.clone() for w in base_ffn.w_down])
        wsets.append((sc, ff))
    ws = ce.alloc_workspace(ce.CE_WS_BLOCK, batch, d, F, dtc, device=dev)
    stream = torch.cuda.current_stream()

    # Hidden states: the block works in place, and applied again to its own
    # output it drives the rows to inf / NaN within a few passes (there is no
    # normalization in the block and the synthetic FFN has gain above one), on
    # which the MFMAs draw less power and run faster. So every timed step gets
    # its own pristine copy (restored before the timed loop; the warm-up
    # restores them after each pass over the pool), which also keeps the
    # hidden states cold in the caches.
    # Workload 3 by default runs its 50 denoising steps in turn: step s has its
    # own hidden states and timestep (so its own expansion segment).
    src = [(base_h, batch)]
    if sweep3:
        from ce_workloads import CONFIG3_STEPS, config3_step_hidden, config3_t
        log(f"generating the {CONFIG3_STEPS} denoising steps of workload 3")
        src = []
        for s3 in range(CONFIG3_STEPS):
            t_s = np.full(wl.B, config3_t(s3), np.float32)
            src.append((up(config3_step_hidden(wl.hidden, s3), dt),
                        ce.Batch(batch.seq_offsets, batch.flags, up(t_s), float(wl.keep), cap)))
    n_pool = args.steps
    h_bytes = T * d * elem
    free, _ = torch.cuda.mem_get_info()
    if n_pool * h_bytes > free // 2:
        sys.exit(f"bench.py: {n_pool} pristine copies of the hidden states ({n_pool * h_bytes / 2**30:.1f} GiB) "
                 f"need more than half the free device memory; use fewer --steps")
    pool = [torch.empty_like(base_h) for _ in range(n_pool)]

    def restore():
        for j, x in enumerate(pool):
            x.copy_(src[j % len(src)][0])

    def step(i):
        sc, ff = wsets[i % n_sets]
        j = i % n_pool
        ce.ce_routed_block(src[j % len(src)][1], pool[j], pool[j], sc, ff, ws, stream=stream)

    # ---- whole routed block ----
    for i in range(args.warmup):
        if i % n_pool == 0:
            restore()
        step(i)
    restore()
    torch.cuda.synchronize()
    assert ce.ce_workspace_status(ws) == 0, "device status error"
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    # one event before every step as well, for the per-step statistics; the
    # value is the total over the K steps
    sev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev0.record(stream)
    for i in range(args.steps):
        sev[i].record(stream)
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    n_bad = sum(int((~torch.isfinite(x.float())).sum()) for x in pool[:4])
    assert n_bad == 0, f"{n_bad} non-finite hidden values after one block"
    ms = ev0.elapsed_time(ev1) / args.steps
    marks = sev + [ev1]
    step_us = [marks[i].elapsed_time(marks[i + 1]) * 1e3 for i in range(args.steps)]
    cut = args.steps // 16  # drop the first and last 1/16 in run order, average the middle 7/8
    mid = step_us[cut:args.steps - cut] or step_us
    step_stats = {"median": round(float(np.median(step_us)), 2), "mean_middle_7_8": round(float(np.mean(mid)), 2),
                  "min": round(min(step_us), 2), "max": round(max(step_us), 2)}
    log(f"routed block: {ms * 1e3:.1f} us/step (median {step_stats['median']}, middle 7/8 "
        f"{step_stats['mean_middle_7_8']})")

    # The block with the layer-skipping gap (Eq. 7) from the down GEMM's
    # epilogue (ce_routed_block_gap) against the plain block: pairs of blocks,
    # plain then with the gap, each on its own pristine copy, an event pair
    # around each, so that both see the same engine clock.
    ws_gap = ce.alloc_workspace(ce.CE_WS_BLOCK_GAP, batch, d, F, dtc, device=dev)
    cos_g = torch.empty(T, device=dev)
    ra_g, rr_g, gp_g = (torch.empty(wl.B, device=dev) for _ in range(3))
    sk_g = torch.empty(wl.B, dtype=torch.uint8, device=dev)
    pool_b = [torch.empty_like(base_h) for _ in range(n_pool)]

    def step_gap(i):
        sc, ff = wsets[i % n_sets]
        j = i % n_pool
        ce.ce_routed_block_gap(src[j % len(src)][1], pool_b[j], pool_b[j], sc, ff, ws_gap, 0.0040, cos_g, ra_g,
                               rr_g, gp_g, sk_g, stream=stream)

    restore()
    for j, x in enumerate(pool_b):
        x.copy_(src[j % len(src)][0])
    torch.cuda.synchronize()
    pairs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for i in range(args.steps):
        pairs[i][0].record(stream)
        step(i)
        pairs[i][1].record(stream)
        step_gap(i)
        pairs[i][2].record(stream)
    torch.cuda.synchronize()
    plain_us = float(np.mean([e[0].elapsed_time(e[1]) for e in pairs])) * 1e3
    gap_block_us = float(np.mean([e[1].elapsed_time(e[2]) for e in pairs])) * 1e3
    log(f"pairs: routed block {plain_us:.1f} us, with the fused layer gap {gap_block_us:.1f} us")
    del pool, pool_b, ws_gap

    # ---- per-stage launches (staged entry points on the same data) ----
    logits = torch.empty(T, device=dev)
    kept_idx = torch.empty(cap, dtype=torch.int32, device=dev)
    kept_off = torch.empty(wl.B + 1, dtype=torch.int32, device=dev)
    compact = torch.empty((cap, d), dtype=dt, device=dev)
    act = torch.empty((cap, F), dtype=dt, device=dev)
    ffn_out = torch.empty((cap, d), dtype=dt, device=dev)
    ws_topk = ce.alloc_workspace(ce.CE_WS_TOPK, batch, d, F, dtc, device=dev)
    ws_score = ce.alloc_workspace(ce.CE_WS_SCORE, batch, d, F, dtc, device=dev)
    ws_ffn = ce.alloc_workspace(ce.CE_WS_FFN, batch, d, F, dtc, device=dev)
    h0 = base_h
    sc0, ff0 = wsets[0]
    ce.ce_score_ws(batch, h0, sc0, logits, ws_score, stream=stream)
    ce.ce_topk_compact(batch, logits, kept_idx, kept_off, ws_topk, hidden=h0, compact=compact,
                       stream=stream)
    torch.cuda.synchronize()

    def timed(fn, reps, warm=0):
        """Mean GPU time per call. A short device-side delay is queued first so
        that the host has enqueued every call before the first one starts: the
        events then time the kernels back to back, not the host's launch rate.
        `warm` untimed calls run between the delay and the timed ones."""
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        torch.cuda._sleep(20_000_000)
        for i in range(warm):
            fn(i)
        for i in range(reps):
            evs[i][0].record(stream)
            fn(i)
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in evs])) * 1e3  # us

    reps = max(args.steps, 10)
    gemm_warm = 20  # untimed rounds after the delay, before the timed ones

    def timed_pipeline(fns, reps, warm):
        """Mean GPU time per call of each of `fns`, called in turn (the staged
        entry points in the order ce_routed_block runs them), one event pair
        around every call: each kernel runs under the same mix of load as in
        the fused block (a GEMM timed back to back against itself draws more
        power and gets a lower clock). Same device-side delay first as timed()."""
        evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in fns] for _ in range(reps)]
        torch.cuda._sleep(20_000_000)
        for i in range(warm):
            for fn in fns:
                fn(i)
        for i in range(reps):
            for f, fn in enumerate(fns):
                evs[i][f][0].record(stream)
                fn(i)
                evs[i][f][1].record(stream)
        torch.cuda.synchronize()
        return [float(np.mean([evs[i][f][0].elapsed_time(evs[i][f][1]) for i in range(reps)])) * 1e3
                for f in range(len(fns))]

    stage_names = ("score", "topk_compact", "ffn_gateup", "ffn_down")
    stage_fns = (
        lambda i: ce.ce_score_ws(batch, h0, wsets[i % n_sets][0], logits, ws_score, stream=stream),
        lambda i: ce.ce_topk_compact(batch, logits, kept_idx, kept_off, ws_topk, stream=stream),
        lambda i: ce.ce_ffn_gateup(batch, compact, kept_idx, kept_off, wsets[i % n_sets][1], act, ws_ffn,
                                   stream=stream),
        lambda i: ce.ce_ffn_down(batch, act, kept_idx, kept_off, wsets[i % n_sets][1], ffn_out, ws_ffn,
                                 stream=stream))
    stages = dict(zip(stage_names, timed_pipeline(stage_fns, reps, gemm_warm)))
    log("stages (us): " + ", ".join(f"{k}={v:.1f}" for k, v in stages.items()))
    # the workspace-free ce_score (single-launch scorer) on the same data
    score_single_us = timed(lambda i: ce.ce_score(batch, h0, wsets[i % n_sets][0], logits, stream=stream), reps)
    log(f"ce_score without a workspace: {score_single_us:.1f} us")

    # FFN-pruning signal (section 3.4, Eq. 8-9) on this step's activations: one
    # read of act plus the per-sequence saliency rows; a 30% static mask
    ffn0 = wsets[0][1]
    n_fs = len(wl.ffn)
    norms = torch.empty(n_fs * F, device=dev)
    ce.ce_ffn_down_colnorms(ffn0, norms, stream=stream)
    pmask = torch.from_numpy((np.random.default_rng(3).random(F) < 0.3).astype(np.uint8)).to(dev)
    sal = torch.empty(wl.B * F, device=dev)
    lam = torch.empty(wl.B, device=dev)
    use = torch.empty(wl.B, dtype=torch.uint8, device=dev)
    sal_us = timed(lambda i: ce.ce_ffn_saliency(batch, act, kept_idx, kept_off, ffn0, norms, pmask, 0.150,
                                                sal, lam, ws_ffn, use, stream=stream), reps)
    sal_bytes = cap * F * (2 if bf16 else 4) + wl.B * F * 4 + F  # activations, saliency rows, mask
    ucs_ffn = {"us_per_call": round(sal_us, 2), "bytes_per_call": sal_bytes, "bound": "hbm",
               "achieved_GBps": round(sal_bytes / (sal_us * 1e-6) / 1e9, 1), "peak_GBps": PEAK_HBM_GBS,
               "frac": round(sal_bytes / (sal_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    log(f"ffn saliency + leakage: {sal_us:.1f} us")

    # the pruned FFN in one call (bf16): P = the channel tail, about 30% of
    # d_ff in whole 64-channel groups; every sequence pruned (delta = 1), none
    # (delta = -1), beside the full FFN, in turn under the same load
    if bf16:
        n_keep = F - 64 * max(1, int(round(0.3 * F / 64)))
        ws_pr = ce.alloc_workspace(ce.CE_WS_FFN_PRUNED, batch, d, F, dtc, device=dev)
        out_pr = torch.empty_like(ffn_out)
        pr = lambda delta: (lambda i: ce.ce_routed_ffn_pruned(
            batch, compact, kept_idx, kept_off, ffn0, norms, n_keep, delta, out_pr, sal, lam, use, ws_pr,
            stream=stream))
        full_us, all_us, none_us = timed_pipeline(
            (lambda i: ce.ce_routed_ffn(batch, compact, kept_idx, kept_off, ffn0, ffn_out, ws_ffn, stream=stream),
             pr(1.0), pr(-1.0)), reps, gemm_warm)
        ucs_ffn["pruned_ffn"] = {
            "n_keep": n_keep, "pruned_channels": F - n_keep, "full_ffn_us": round(full_us, 2),
            "pruned_ffn_all_sequences_us": round(all_us, 2), "pruned_ffn_no_sequence_us": round(none_us, 2),
            "staged_signal_path_us": round(full_us + sal_us, 2),
            "note": "ce_routed_ffn_pruned: saliency sums in the gate/up epilogue, P's channels skipped in the "
                    "down GEMM; staged = ce_routed_ffn + ce_ffn_saliency (mask launch not counted)"}
        log(f"pruned ffn: full {full_us:.1f} us, all pruned {all_us:.1f} us, none pruned {none_us:.1f} us "
            f"(P = {F - n_keep} of {F})")
        del ws_pr, out_pr

    # layer-skipping gap (section 3.4, Eq. 7) over this workload's hidden
    # states: two [T x d] reads, the per-token cosines written and re-read
    kt = int(kept_off[-1].item())
    tok_pos = torch.full((T,), -1, dtype=torch.int32, device=dev)
    tok_pos[kept_idx[:kt].long()] = torch.arange(kt, dtype=torch.int32, device=dev)
    cos_tok = torch.empty(T, device=dev)
    rho_a, rho_r, gap_b = (torch.empty(wl.B, device=dev) for _ in range(3))
    skip_b = torch.empty(wl.B, dtype=torch.uint8, device=dev)
    x_out = torch.empty_like(h0)
    x_out.copy_(src[min(1, len(src) - 1)][0])
    gap_us = timed(lambda i: ce.ce_layer_gap(batch, h0, x_out, tok_pos, 0.0040, cos_tok, rho_a, rho_r, gap_b,
                                             skip_b, stream=stream), reps)
    gap_bytes = 2 * T * d * (2 if bf16 else 4) + 12 * T
    ucs_gap = {"us_per_call": round(gap_us, 2), "bytes_per_call": gap_bytes, "bound": "hbm",
               "achieved_GBps": round(gap_bytes / (gap_us * 1e-6) / 1e9, 1), "peak_GBps": PEAK_HBM_GBS,
               "frac": round(gap_bytes / (gap_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    log(f"layer gap: {gap_us:.1f} us")

    gateup_flops = 4.0 * cap * d * F  # gate and up: 2 GEMMs of Kt x d x F, 2 flops per MAC
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    achieved = gateup_flops / (stages["ffn_gateup"] * 1e-6) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": load_traffic(wid),
                "kernel": "ffn_gemm_pp2_kernel gate/up + SwiGLU (ce_ffn_gateup)",
                "flops_per_launch": gateup_flops, "timed_launches": reps, "warm_launches": gemm_warm}

    block_flops = (2.0 * cap * d * 3 * F
                   + 2.0 * float(np.sum((wl.flags & 2) == 0)) * d * sw.r_core
                   + 2.0 * float(np.sum(((wl.flags & 1) != 0) & ((wl.flags & 2) == 0))) * d * sw.r_exp)
    result = {
        "metric": METRIC,
        "value": round(T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": CONFIG_NAMES[wid], "description": CONFIG_DESCRIPTIONS[wid], "B": wl.B,
                   "T": T, "kept_rows": cap, "d": d, "d_ff": F, "r_core": sw.r_core, "r_exp": sw.r_exp,
                   "keep": float(wl.keep), "ffn_sets": len(wl.ffn), "weight_sets": n_sets,
                   "hidden_copies": args.steps,
                   "parallelism": "single GPU",
                   **({"denoising_steps": "all 50 in turn, value per step"} if sweep3 else
                      {"denoising_step": args.step3} if wid == 3 else {})},
        "kept_tokens_per_s": round(cap / (ms * 1e-3), 1),
        "block_tflops": round(block_flops / (ms * 1e-3) / 1e12, 2),
        "step_us": step_stats,
        "stages_us": {k: round(v, 2) for k, v in stages.items()},
        "score_single_launch_us": round(score_single_us, 2),
        "roofline": roofline,
    }
    result["ucs_signals"] = time_drop_stability(ce, stream, max(args.steps, 10))
    result["ucs_signals"]["ffn_saliency_leakage"] = ucs_ffn
    result["ucs_signals"]["layer_gap"] = ucs_gap
    result["ucs_signals"]["layer_gap_fused_in_block"] = {
        "block_with_gap_us": round(gap_block_us, 2), "block_us": round(plain_us, 2),
        "extra_us": round(gap_block_us - plain_us, 2), "pairs": args.steps,
        "note": "ce_routed_block_gap vs ce_routed_block in alternating pairs; the gap sums come from the "
                "down GEMM's epilogue (no [T x d] re-read)"}
    result["routed_attention"] = time_attention(ce, stream, max(args.steps, 10))
    result["achievable_peaks"] = (achievable_peaks(cap, d, F) if bf16 else None)
    if not args.no_cpu_baseline:
        n_seq = args.cpu_seqs or wl.B
        log(f"oracle CPU baseline on {n_seq} sequence(s)...")
        result["cpu_baseline"] = cpu_baseline(wl, n_seq)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
