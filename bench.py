"""Throughput of one wave of paged chunked-prefill attention on one MI355X.

A step is one pass of the whole hot path over one wave: host plan -> metadata upload -> K/V append ->
attention (-> split merge), once per layer of the workload.  Inputs are resident in HBM before the
timed region.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--config 5|1|2|3|4|6p|small16...] [--extras 3,4|none]
                    [--no-cpu-baseline]

The default headline is the latent-attention wave (8 requests, 131072 cached + 8192 new tokens each,
128 heads over a 576-wide latent), the largest wave that fits one GPU; the grouped-query waves named
by --extras (default: the shared-prefix wave and the four-layer concurrency-128 wave) are measured
after it and reported under "extra".

Metric: attention TFLOP/s (algorithmic FLOP = 2 * Hq * (d_qk + d_v) * sum_r [c_r p_r + c_r (c_r + 1) / 2]
per layer, exact causal pairs only), new tokens/s, % of the bf16 dense MFMA peak.

    python bench.py --config kda_wave|kda_long|kda_short|kda_small

times the KDA chunked prefill instead (one layer per step: plan -> upload -> chunked prefill, resuming
from and writing snapshots).  It is bound by HBM: its metric is new tokens/s and its roofline the
algorithmic bytes per launch (q, k, v, alpha, beta, out, and the snapshots read and written) over the
kernel time, against 8 TB/s.

    python bench.py --config mpu

times the native MPU wave planner on the host (planning decisions per second over a seeded admission
trace shaped like the paper's eight-stage runs), against the reference planner as the CPU baseline.

    python bench.py --config hints

times reuse-hint discovery on the host: chained block hashing of 200K-token requests and the
gallop/bisect prefix probe against a sharded index holding 64 such cached prompts (the paper's
stress shape), with the plain scan and the reference as comparisons.

    python bench.py --config peak

measures what the matrix cores sustain on this GPU (a register-only MFMA probe) and the shader clock
meanwhile, the reference point beside the nominal 2516.6 TFLOP/s.
"""
import argparse
import gc
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0
RIDGE_FLOP_PER_BYTE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)     # ~315 FLOP/B
METRIC = "chunked-prefill attention TFLOP/s + new tokens/s on 1 GPU; % of bf16 MFMA peak"


def run_timed(step, sync, warmup=None, steps=None):
    """Warm up, then time exactly `steps` steps between two device synchronizations, with Python's
    garbage collector off (a collection pauses the host for tens of ms, and the idle GPU drops its
    clock).  The first three steps run synchronized, and the last two of them give the step time t.
    warmup None: untimed steps for max(0.3 s, min(2 s, 300 t)) in all, so that the runtime's one-time
    pool growth and the clock ramp fall inside them.  steps None: about one second of timed work,
    3 to 2000 steps.  Returns (warmup, steps, elapsed seconds)."""
    first = 3 if warmup is None else min(3, warmup)
    done = 0
    t_pair = None
    for k in range(first):
        if k == 1:
            sync()
            t_pair = time.perf_counter()
        step()
        done += 1
        sync()
    per = (time.perf_counter() - t_pair) / (done - 1) if done >= 2 else None
    if warmup is None:
        target = max(0.3, min(2.0, 300 * per))
        extra = max(0, math.ceil(target / per) - done)
    else:
        extra = warmup - done
    for _ in range(extra):
        step()
        done += 1
    sync()
    if steps is None:
        if per is None:
            t0 = time.perf_counter()
            step()
            sync()
            per = time.perf_counter() - t0
            done += 1
        steps = int(min(2000, max(3, math.ceil(1.0 / max(per, 1e-6)))))
    gc.collect()
    gc.disable()
    try:
        sync()
        t1 = time.perf_counter()
        for _ in range(steps):
            step(record=True)
        sync()
        elapsed = time.perf_counter() - t1
    finally:
        gc.enable()
    return done, steps, elapsed


def flops_alg(spec) -> float:
    """Algorithmic FLOP of one layer's attention: exact visible pairs x 2 (QK) + 2 (PV) per dim."""
    return 2.0 * spec.num_q_heads * (spec.head_dim_qk + spec.head_dim_v) * float(spec.pairs().sum())


def bytes_alg(spec) -> float:
    """Algorithmic HBM bytes of one layer: Q + O + the prefix K/V each request reads + the chunk's K/V
    read once and written once by the append."""
    T = spec.total_tokens
    per_tok = (spec.head_dim_qk * 2 if spec.kv_shared
               else spec.num_kv_heads * (spec.head_dim_qk + spec.head_dim_v) * 2)
    q = T * spec.num_q_heads * spec.head_dim_qk * 2
    o = T * spec.num_q_heads * spec.head_dim_v * 2
    return float(q + o + float(spec.prefix_lens.sum()) * per_tok + 2.0 * T * per_tok)


def append_bytes(spec) -> float:
    per_tok = (spec.head_dim_qk * 2 if spec.kv_shared
               else spec.num_kv_heads * (spec.head_dim_qk + spec.head_dim_v) * 2)
    return 2.0 * spec.total_tokens * per_tok


def cpu_baseline(spec, tensors, budget_s=12.0):
    """Time the fp64 oracle (as it stands) on the host cores on a bounded sample of the same wave.

    Small waves (<= 1 TFLOP) are timed whole, repeated until the runs add up to about `budget_s`;
    larger ones on random (token, head) rows, each over all of its visible keys, with the sample
    grown until one run takes about `budget_s`.  The append is done beforehand and is not timed.
    """
    import numpy as np
    import oracle
    import workloads as wl
    host = host_cpu_info()
    threads = host["blas_threads"] or host["cpu_count"]
    pools = {k: wl.to_bits(tensors[k]) for k in ("k_pool", "v_pool", "k_new", "v_new")}
    k1, v1 = oracle.append_kv(pools["k_pool"], pools["v_pool"], pools["k_new"], pools["v_new"], spec.prefix_lens,
                              spec.chunk_lens, spec.block_table, spec.page_size)
    del pools
    kw = dict(page_size=spec.page_size, num_kv_heads=spec.num_kv_heads, softmax_scale=spec.softmax_scale,
              kv_shared=spec.kv_shared, head_dim_v=spec.head_dim_v)
    total_flop = flops_alg(spec)
    if total_flop <= 1e12:
        q = wl.to_bits(tensors["q"])
        runs, dt = 0, 0.0
        while runs == 0 or (dt < budget_s * 0.8 and runs < 10000):
            t0 = time.perf_counter()
            oracle.chunked_prefill(q, k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table, **kw)
            dt += time.perf_counter() - t0
            runs += 1
        flop, n = total_flop * runs, None
        sample = (f"whole {spec.name} wave (all {spec.total_tokens} tokens x {spec.num_q_heads} heads), "
                  f"{runs} run{'s' if runs > 1 else ''}")
    else:
        rng = np.random.default_rng(0)
        cu = spec.cu_tokens
        per_row = 2.0 * (spec.head_dim_qk + spec.head_dim_v)
        n = 16
        while True:
            toks = rng.integers(0, spec.total_tokens, n)
            heads = rng.integers(0, spec.num_q_heads, n)
            samples = np.stack([toks, heads], 1)
            qd = {int(t): wl.to_bits(tensors["q"][int(t)]) for t in set(toks.tolist())}
            r = np.searchsorted(cu, toks, side="right") - 1
            flop = float(np.sum(per_row * (spec.prefix_lens[r] + (toks - cu[r]) + 1)))
            t0 = time.perf_counter()
            oracle.chunked_prefill_rows(qd, k1, v1, spec.prefix_lens, spec.chunk_lens, spec.block_table,
                                        samples, **kw)
            dt = time.perf_counter() - t0
            if dt >= budget_s * 0.6 or n >= 1 << 16:
                break
            n = int(n * min(16.0, max(1.5, budget_s / max(dt, 1e-3))))
        sample = f"{n} random (token, head) rows of the {spec.name} wave, each over all its visible keys"
    return {"value": round(flop / dt / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": sample, "seconds": round(dt, 3), **host}


def host_cpu_info() -> dict:
    """The host the oracle runs on: logical CPUs, CPU model (lscpu) and the BLAS library's thread
    count (the numpy fp64 oracle's matrix products run on that pool)."""
    info = {"cpu_count": os.cpu_count(), "cpu_model": None, "blas_threads": None, "blas": None}
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.lower().startswith("model name"):
                info["cpu_model"] = line.split(":", 1)[1].strip()
                break
    except Exception:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if blas:
            info["blas_threads"] = int(max(i.get("num_threads", 1) for i in blas))
            info["blas"] = f"{blas[0].get('internal_api')} {blas[0].get('version')}"
    except Exception:
        pass
    return info


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: about one second of work)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps first (default: max(0.3 s, min(2 s, 300 steps)))")
    ap.add_argument("--config", default="5",
                    help="the headline wave (default 5: the latent-attention wave, the largest that fits one GPU)")
    ap.add_argument("--extras", default="3,4",
                    help="comma-separated waves also measured after the headline and reported under 'extra' "
                         "(each with the default warm-up and about one second of timed steps); 'none' for none")
    ap.add_argument("--max-splits", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (HBM counter calibration)")
    ap.add_argument("--measure-traffic", metavar="OUT_JSON", default=None,
                    help="run rocprofv3 FETCH_SIZE and WRITE_SIZE passes over this config and write the per-launch "
                         "HBM bytes of the attention kernel, calibrated against a plain copy, to OUT_JSON")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the attention path has no multi-GPU implementation",
              file=sys.stderr)
        sys.exit(2)
    if args.measure_traffic:
        sys.exit(measure_traffic(args.config, args.measure_traffic))
    if str(args.config).startswith("kda"):
        return main_kda(args)
    if str(args.config) == "mpu":
        return main_mpu(args)
    if str(args.config) == "hints":
        return main_hints(args)
    if str(args.config) == "peak":
        return main_peak(args)

    import torch
    import paper_2609_35263_amd as wp

    wp.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    res = measure_wave(str(args.config), dev, args.warmup, args.steps, args.max_splits,
                       calib_mib=args.copy_calibration_mib)
    # what the matrix cores sustain on this chip with random-bit operands (a power-limited clock), as
    # context for the nominal peak; run after the timed region
    p_tf, p_ghz = mfma_probe(torch)
    res["mfma_probe"] = {"tflops": round(p_tf, 1), "sclk_ghz": round(p_ghz, 3),
                         "attn_frac_of_probe": (round(res["roofline"]["achieved"] / p_tf, 4)
                                                if res["roofline"]["bound"] == "mfma" else None)}
    if res["roofline"]["bound"] == "hbm":
        r_gbs = hbm_read_probe(torch)
        res["hbm_read_probe"] = {"GBps": round(r_gbs, 1), "attn_frac_of_probe": round(res["roofline"]["achieved"] / r_gbs, 4)}
    extras = [] if args.extras.strip().lower() in ("", "none") else [e.strip() for e in args.extras.split(",")]
    if extras:
        res["extra"] = {}
        for name in extras:
            if name == str(args.config):
                continue
            x = measure_wave(name, dev, None, None, args.max_splits)
            res["extra"][x.pop("_name")] = {k: x[k] for k in ("value", "unit", "pct_peak", "ms_per_step", "steps",
                                                             "warmup", "new_tokens_per_s", "attn_kernel_ms",
                                                             "config", "roofline")}
    if not args.no_cpu_baseline:
        import workloads as wl
        progress("oracle baseline on the host cores")
        spec = res.pop("_spec")
        fresh = wl.make_tensors(spec, seed=res.pop("_seed"), device=dev, poison=False)
        res["cpu_baseline"] = cpu_baseline(spec, fresh)
        del fresh
    for k in [k for k in res if k.startswith("_")]:
        res.pop(k)
    print(json.dumps(res), flush=True)


SEEDS = {"1": 1000, "2": 2000, "3": 3000, "4": 4000, "5": 5000, "6p": 6000}


def progress(msg):
    """A progress line on stderr (the JSON line alone goes to stdout)."""
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def measure_wave(name, dev, warmup, steps, max_splits=0, calib_mib=0) -> dict:
    """Time whole steps (plan, upload, and per layer append + attention) of one wave and return the
    JSON fields of its line.  The attention launches are timed with events on the launch stream."""
    import numpy as np
    import torch
    import paper_2609_35263_amd as wp
    import workloads as wl

    spec = wl.config(name)
    layers = spec.layers
    seed = SEEDS.get(name, 7000)
    big = flops_alg(spec) > 1e12
    # layer tensors, resident in HBM; timing runs use zero-filled (not NaN) unused slots
    dl = []
    for l in range(layers):
        t = wl.make_tensors(spec, seed=seed, device=dev if big else "cpu", poison=False, layer=l)
        dl.append({k: (None if v is None else v.to(dev).contiguous()) for k, v in t.items()})
        del t
    T = spec.total_tokens
    outs = [torch.empty((T, spec.num_q_heads, spec.head_dim_v), dtype=torch.bfloat16, device=dev)
            for _ in range(layers)]
    lses = [torch.empty((T, spec.num_q_heads), dtype=torch.float32, device=dev) for _ in range(layers)]
    p0 = wp.plan_for(spec, max_splits=max_splits)
    ws = wp.new_workspace(p0, dev)
    info = p0.info()
    stream = torch.cuda.current_stream()

    attn_events = []

    def step(record=False):
        p = wp.plan_for(spec, max_splits=max_splits)
        wp.plan_upload(p, ws)
        for l in range(layers):
            d = dl[l]
            wp.append_kv(p, d["k_new"], d["v_new"], d["k_pool"], d["v_pool"], ws)
            if record:
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                wp.chunked_prefill(p, d["q"], d["k_pool"], d["v_pool"], outs[l], lses[l], ws)
                e1.record(stream)
                attn_events.append((e0, e1))
            else:
                wp.chunked_prefill(p, d["q"], d["k_pool"], d["v_pool"], outs[l], lses[l], ws)
        return p

    if calib_mib:
        n = calib_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    progress(f"{spec.name}: inputs resident, {info['num_items']} work items; warm-up and timed steps")
    warmup, steps, elapsed = run_timed(step, torch.cuda.synchronize, warmup, steps)
    ms_per_step = elapsed * 1e3 / steps
    progress(f"{spec.name}: {steps} timed steps after {warmup} warm-up, {ms_per_step:.3f} ms per step")
    attn_all = [a.elapsed_time(b) for a, b in attn_events]
    attn_ms = float(np.mean(attn_all))

    # append alone, for its HBM rate (outside the timed region)
    wp.plan_upload(p0, ws)
    torch.cuda.synchronize()
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record(stream)
    for _ in range(5):
        wp.append_kv(p0, dl[0]["k_new"], dl[0]["v_new"], dl[0]["k_pool"], dl[0]["v_pool"], ws)
    a1.record(stream)
    torch.cuda.synchronize()
    append_ms = a0.elapsed_time(a1) / 5
    del dl, outs, lses

    f_layer = flops_alg(spec)
    f_step = f_layer * layers
    value = f_step / (ms_per_step * 1e-3) / 1e12
    achieved = f_layer / (attn_ms * 1e-3) / 1e12
    traffic, counters = None, {}
    tfile = os.path.join(ROOT, "profiles", f"traffic_{spec.name}.json")
    if os.path.exists(tfile):
        try:
            tj = json.load(open(tfile))
            if tj.get("kernel_source_hash") == _kernel_hash():
                traffic = tj.get("bytes_per_launch")
                counters = {k: round(tj[k], 1) for k in ("mfma_util_pct", "l2_hit_pct") if k in tj}
        except Exception:
            traffic, counters = None, {}
    b_layer = bytes_alg(spec)
    kernel_name = "attn_gqa_kernel" if not spec.kv_shared else "attn_mla_kernel"
    if info.get("num_merge_items", 0) > 0:
        # key-range splits: the timed interval (one chunked_prefill call) also holds the merge kernel
        kernel_name += " + merge_kernel"
    if f_layer / b_layer >= RIDGE_FLOP_PER_BYTE:
        roofline = {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic, "kernel": kernel_name,
                    "alg_flop_per_launch": f_layer, "alg_bytes_per_launch": b_layer, **counters}
    else:
        gbps = b_layer / (attn_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(gbps, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(gbps / PEAK_HBM_GBS, 4), "traffic": traffic, "kernel": kernel_name,
                    "alg_flop_per_launch": f_layer, "alg_bytes_per_launch": b_layer, **counters}
    return {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{spec.name}: {spec.num_requests} requests, prefix {int(spec.prefix_lens.min())}-"
                               f"{int(spec.prefix_lens.max())}, chunks {int(spec.chunk_lens.min())}-"
                               f"{int(spec.chunk_lens.max())} ({T} new tokens), Hq {spec.num_q_heads}, "
                               f"Hkv {spec.num_kv_heads}, d {spec.head_dim_qk}/{spec.head_dim_v}, page "
                               f"{spec.page_size}, layers {layers}",
                   "global_batch": int(spec.num_requests), "new_tokens": int(T), "layers": int(layers),
                   "parallelism": "none (1 GPU)"},
        "new_tokens_per_s": round(T * layers / (ms_per_step * 1e-3) / layers, 1),
        "pct_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "attn_kernel_ms": round(attn_ms, 4),
        "attn_kernel_ms_median": round(float(np.median(attn_all)), 4),
        "append_ms": round(append_ms, 4),
        "append_GBps": round(append_bytes(spec) / (append_ms * 1e-3) / 1e9, 1),
        "attn_alg_GBps": round(bytes_alg(spec) / (attn_ms * 1e-3) / 1e9, 1),
        "work_items": info["num_items"],
        "roofline": roofline,
        "_name": spec.name, "_spec": spec, "_seed": seed,
    }


KDA_METRIC = "KDA chunked-prefill new tokens/s on 1 GPU; % of HBM peak"


def kda_bytes_alg(spec) -> float:
    """Algorithmic HBM bytes of one KDA layer: q, k, v (bf16), alpha (fp32), beta (fp32) read once, out
    (bf16) written once, and one fp32 snapshot per head read for each resumed request and written for
    each active one."""
    th = float(spec.total_tokens) * spec.num_heads
    per_th = 2 * spec.head_dim_k * 2 + spec.head_dim_v * 2 + spec.head_dim_k * 4 + 4 + spec.head_dim_v * 2
    active = spec.chunk_lens > 0
    snaps = int(np.sum(active & (spec.state_in >= 0))) + int(np.sum(active))
    return th * per_th + float(snaps) * spec.num_heads * spec.head_dim_k * spec.head_dim_v * 4


def kda_flops_alg(spec) -> float:
    """FLOP of the token-by-token recurrence per token and head: decay (d_k d_v), k^T S (2 d_k d_v), the
    rank-1 erase-and-write (2 d_k d_v) and the read-out (2 d_k d_v)."""
    return 7.0 * spec.head_dim_k * spec.head_dim_v * float(spec.total_tokens) * spec.num_heads


def kda_cpu_baseline(spec, tensors, budget_s=12.0):
    """Time the fp64 oracle (as it stands) on the host cores: the first n tokens of the first request,
    all heads, n grown until one run takes about `budget_s`.  Reported in new tokens/s of the whole layer."""
    import oracle.kda as okda
    import workloads as wl
    host = host_cpu_info()
    threads = host["blas_threads"] or host["cpu_count"]
    c0 = int(spec.chunk_lens[0])
    n = 8
    while True:
        n = min(n, c0)
        part = {k: tensors[k][:n].cpu() for k in ("q", "k", "v", "alpha", "beta")}
        bits = {k: wl.to_bits(part[k]) for k in ("q", "k", "v")}
        pool = tensors["state_pool"].cpu().numpy()
        t0 = time.perf_counter()
        okda.chunked_prefill(bits["q"], bits["k"], bits["v"], part["alpha"].numpy(), part["beta"].numpy(), pool,
                             [n], [int(spec.state_in[0])], [int(spec.state_out[0])])
        dt = time.perf_counter() - t0
        if dt >= budget_s * 0.6 or n >= c0:
            break
        n = int(n * min(16.0, max(1.5, budget_s / max(dt, 1e-3))))
    return {"value": round(n / dt, 3), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {n} tokens of request 0 of the {spec.name} wave, all {spec.num_heads} heads",
            "seconds": round(dt, 3)}


def main_kda(args):
    import torch
    import paper_2609_35263_amd as wp
    import workloads.kda as wk

    wp.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    spec = wk.config(args.config)
    t = wk.make_tensors(spec, seed=8000, device=dev, poison=False)
    T = spec.total_tokens
    out = torch.empty((T, spec.num_heads, spec.head_dim_v), dtype=torch.bfloat16, device=dev)
    pool = t["state_pool"]
    p0 = wp.kda_plan_for(spec)
    ws = wp.new_workspace(p0, dev)
    stream = torch.cuda.current_stream()
    kev = []

    def step(record=False):
        p = wp.kda_plan_for(spec)
        wp.kda_upload(p, ws)
        if record:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
        wp.kda_chunked_prefill(p, t["q"], t["k"], t["v"], t["alpha"], t["beta"], pool, out, ws)
        if record:
            e1.record(stream)
            kev.append((e0, e1))

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    warmup, steps, elapsed = run_timed(step, torch.cuda.synchronize, args.warmup, args.steps)
    ms_per_step = elapsed * 1e3 / steps
    kms = float(np.mean([a.elapsed_time(b) for a, b in kev]))
    b = kda_bytes_alg(spec)
    f = kda_flops_alg(spec)
    gbps = b / (kms * 1e-3) / 1e9
    traffic, counters = None, {}
    tfile = os.path.join(ROOT, "profiles", f"traffic_{spec.name}.json")
    if os.path.exists(tfile):
        try:
            tj = json.load(open(tfile))
            if tj.get("kernel_source_hash") == _kernel_hash("kda"):
                traffic = tj.get("bytes_per_launch")
                counters = {k: round(tj[k], 1) for k in ("mfma_util_pct", "l2_hit_pct") if k in tj}
        except Exception:
            traffic, counters = None, {}
    res = {
        "metric": KDA_METRIC,
        "value": round(T / (ms_per_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{spec.name}: {spec.num_requests} chunks of {int(spec.chunk_lens.min())}-"
                               f"{int(spec.chunk_lens.max())} tokens ({T} new tokens), "
                               f"{int(np.sum(spec.state_in >= 0))} resumed from snapshots, {spec.num_heads} heads, "
                               f"d_k {spec.head_dim_k}, d_v {spec.head_dim_v}",
                   "global_batch": int(spec.num_requests), "new_tokens": int(T), "layers": 1,
                   "parallelism": "none (1 GPU)"},
        "kda_kernel_ms": round(kms, 4),
        "alg_TFLOPs_recurrence": round(f / (kms * 1e-3) / 1e12, 3),
        "work_groups": int(p0.info()["num_items"]) * spec.num_heads,
        "roofline": {"bound": "hbm", "achieved": round(gbps, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(gbps / PEAK_HBM_GBS, 4), "traffic": traffic, "kernel": "kda_prefill_kernel",
                     "alg_bytes_per_launch": b, "alg_flop_per_launch": f, **counters},
    }
    r_gbs = hbm_read_probe(torch)
    res["hbm_read_probe"] = {"GBps": round(r_gbs, 1), "kda_frac_of_probe": round(gbps / r_gbs, 4)}
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = kda_cpu_baseline(spec, wk.make_tensors(spec, seed=8000, device=dev, poison=False))
    print(json.dumps(res), flush=True)


MPU_CONFIG = dict(max_budget=16384, min_budget=8192, block=64, stages=8, fills=1, max_lanes=64,
                  count_inflight=False)


def mfma_probe(torch, workgroups=1024, iters=20000, random_ops=1, launches=20):
    """Median TFLOP/s and shader clock (GHz) of the register-only MFMA probe over a few launches."""
    import ctypes
    import paper_2609_35263_amd as wp
    lib = wp.load_library()
    lib.wavepp_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
    lib.wavepp_probe_mfma.restype = ctypes.c_int
    sink = torch.empty(workgroups * 512, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(4, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream()
    ms = []
    for _ in range(launches):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st = lib.wavepp_probe_mfma(workgroups, iters, random_ops, ctypes.c_void_p(sink.data_ptr()),
                                   ctypes.c_void_p(clocks.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
        if st != 0:
            raise RuntimeError(f"probe failed: {st}")
        e1.record(stream)
        ms.append((e0, e1))
    torch.cuda.synchronize()
    t = float(np.median([a.elapsed_time(b) for a, b in ms[len(ms) // 2:]]))
    c = clocks.cpu().numpy().astype(np.float64)
    return workgroups * 8 * iters * 4 * 32768.0 / (t * 1e-3) / 1e12, float((c[2] - c[0]) / ((c[3] - c[1]) * 10.0))


def hbm_read_probe(torch, mib=4096, workgroups=8192, launches=12):
    """Median GB/s of the library's read-only streaming probe over a `mib` MiB device buffer: the rate
    plain streaming reads reach on this GPU, the practical ceiling of the gather-bound waves."""
    import ctypes
    import paper_2609_35263_amd as wp
    lib = wp.load_library()
    lib.wavepp_probe_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p]
    lib.wavepp_probe_hbm_read.restype = ctypes.c_int
    nbytes = mib << 20
    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    sink = torch.empty(workgroups * 256, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    ms = []
    for _ in range(launches):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st = lib.wavepp_probe_hbm_read(ctypes.c_void_p(src.data_ptr()), nbytes, workgroups,
                                       ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
        if st != 0:
            raise RuntimeError(f"read probe failed: {st}")
        e1.record(stream)
        ms.append((e0, e1))
    torch.cuda.synchronize()
    t = float(np.median([a.elapsed_time(b) for a, b in ms[len(ms) // 2:]]))
    del src, sink
    return nbytes / (t * 1e-3) / 1e9


def main_peak(args, workgroups=1024, iters=20000):
    """The dense bf16 matrix-core rate the chip sustains, and its shader clock meanwhile: the probe
    kernel of wavepp_probe.h (register operands only, four independent MFMA chains per wave)."""
    import ctypes
    import torch
    import paper_2609_35263_amd as wp
    lib = wp.load_library()
    lib.wavepp_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p]
    lib.wavepp_probe_mfma.restype = ctypes.c_int
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sink = torch.empty(workgroups * 512, dtype=torch.float32, device=dev)
    clocks = torch.zeros(4, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()
    events = []
    random_ops = 1

    def step(record=False):
        if record:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
        st = lib.wavepp_probe_mfma(workgroups, iters, random_ops, ctypes.c_void_p(sink.data_ptr()),
                                   ctypes.c_void_p(clocks.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
        if st != 0:
            raise RuntimeError(f"probe failed: {st}")
        if record:
            e1.record(stream)
            events.append((e0, e1))

    flop = workgroups * 8 * iters * 4 * 32768.0
    # small constant operands first (for the record), then random-bit ones (the reported value)
    random_ops = 0
    run_timed(step, torch.cuda.synchronize, 3, 20)
    c = clocks.cpu().numpy().astype(np.float64)
    quiet = {"tflops": round(flop / (float(np.median([a.elapsed_time(b) for a, b in events])) * 1e-3) / 1e12, 1),
             "sclk_ghz": round(float((c[2] - c[0]) / ((c[3] - c[1]) * 10.0)), 3)}
    events.clear()
    random_ops = 1
    warmup, steps, elapsed = run_timed(step, torch.cuda.synchronize, args.warmup, args.steps)
    ms = float(np.median([a.elapsed_time(b) for a, b in events]))
    tflops = flop / (ms * 1e-3) / 1e12
    c = clocks.cpu().numpy().astype(np.float64)
    sclk_ghz = (c[2] - c[0]) / ((c[3] - c[1]) * 10.0)          # s_memrealtime ticks at 100 MHz
    at_clk = 256 * sclk_ghz * 1e9 * 4096 / 1e12
    res = {
        "metric": "dense bf16 MFMA TFLOP/s sustained by a register-only probe (v_mfma_f32_32x32x16_bf16)",
        "value": round(tflops, 1),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(elapsed * 1e3 / steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{workgroups} workgroups x 8 waves x {iters} rounds x 4 MFMA chains, random-bit "
                               f"bf16 operands", "parallelism": "none (1 GPU)"},
        "small_constant_operands": quiet,
        "sclk_ghz_under_load": round(float(sclk_ghz), 3),
        "peak_at_measured_clock": round(at_clk, 1),
        "frac_of_nominal": round(tflops / PEAK_BF16_TFLOPS, 4),
        "frac_at_measured_clock": round(tflops / at_clk, 4),
        "roofline": None,
    }
    print(json.dumps(res), flush=True)


def mpu_trace(planner, n_requests=512, concurrency=64, seed=9000):
    """Drive a planner through one admission trace: requests with 10 % uncached suffixes of 65,536,
    131,072 or 262,144-token prompts (and a quarter cold), at most `concurrency` in the system; every
    proposed wave is accepted and the oldest wave retires when the ring is full.  Returns
    (decisions, waves, seconds spent inside plan + commit)."""
    rng = np.random.default_rng(seed)
    lengths = [65536, 131072, 262144]
    live, admitted, decisions, waves, spent = {}, 0, 0, 0, 0.0
    R = 2 * MPU_CONFIG["stages"]
    ring = 0
    while admitted < n_requests or live:
        while admitted < n_requests and len(live) < concurrency:
            L = int(rng.choice(lengths))
            cached = 0 if rng.random() < 0.25 else (L * 9 // 10) // 64 * 64
            planner.admit(admitted, cached, L)
            live[admitted] = L
            admitted += 1
        t0 = time.perf_counter()
        spans, _ = planner.plan(admission_pending=admitted < n_requests)
        if spans:
            planner.commit(spans)
        spent += time.perf_counter() - t0
        decisions += 1
        if spans:
            waves += 1
            ring += 1
            for rid, st, ln in spans:
                if st + ln >= live[rid]:
                    del live[rid]
        if ring >= R or not spans:
            if ring:
                planner.retire()
                ring -= 1
    return decisions, waves, spent


def main_mpu(args):
    import paper_2609_35263_amd as wp
    import oracle.mpu as omp
    wp.load_library()
    reps = max(1, 20 if args.steps is None else args.steps)
    warm = 3 if args.warmup is None else args.warmup
    for _ in range(warm):
        mpu_trace(wp.MpuPlanner(**MPU_CONFIG), n_requests=64)
    t0 = time.perf_counter()
    dec = spent = 0
    for _ in range(reps):
        d, w, s = mpu_trace(wp.MpuPlanner(**MPU_CONFIG))
        dec += d
        spent += s
    elapsed = time.perf_counter() - t0
    res = {
        "metric": "MPU wave-planner decisions/s on the host (plan + commit)",
        "value": round(dec / spent, 1),
        "unit": "decisions/s",
        "n_gpus": 1,
        "steps": reps,
        "warmup": warm,
        "ms_per_step": round(elapsed * 1e3 / reps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": "512 requests at concurrency 64: 10 % suffixes of 65,536 / 131,072 / 262,144-token "
                               "prompts (a quarter cold); P = 8 stages, M = 16,384, b_min = 8,192, F = 1, "
                               "unscheduled tokens only, up to 64 requests per wave",
                   "global_batch": 512, "parallelism": "none (host)"},
        "us_per_decision": round(spent / dec * 1e6, 3),
        "decisions_per_trace": dec // reps,
        "waves_per_trace": w,
        "roofline": None,
    }
    if not args.no_cpu_baseline:
        t1 = time.perf_counter()
        d, w2, s = mpu_trace(omp.Planner(**MPU_CONFIG))
        res["cpu_baseline"] = {"value": round(d / s, 1), "unit": "decisions/s", "cores": 1, "kind": "oracle",
                               "sample": "one full trace through the reference planner", "seconds": round(time.perf_counter() - t1, 3),
                               "same_waves": w2 == w}
    print(json.dumps(res), flush=True)


def main_hints(args, n_req=64, prompt=200_000, block=64, seed=9100):
    import paper_2609_35263_amd as wp
    import oracle.hints as ohi
    wp.load_library()
    rng = np.random.default_rng(seed)
    # 64 cached prompts of 200K tokens: groups of 8 share a common prefix of 0-100 % of the prompt
    bases = [rng.integers(0, 150_000, prompt) for _ in range(8)]
    idx = wp.HintIndex(num_shards=64)
    cached = []
    for i in range(n_req):
        b = bases[i % 8]
        cut = int(rng.integers(0, prompt // block + 1)) * block
        seq = np.concatenate([b[:cut], rng.integers(0, 150_000, prompt - cut)])
        _, keys = wp.block_hashes(seq, block)
        idx.add(0, keys)
        cached.append(keys)
    # requests: another 64 prompts over the same bases
    reqs = []
    t_hash = []
    for i in range(n_req):
        b = bases[i % 8]
        cut = int(rng.integers(0, prompt // block + 1)) * block
        seq = np.concatenate([b[:cut], rng.integers(0, 150_000, prompt - cut)]).astype(np.int32)
        t0 = time.perf_counter()
        _, keys = wp.block_hashes(seq, block)
        t_hash.append(time.perf_counter() - t0)
        reqs.append(keys)
    reps = max(1, 20 if args.steps is None else args.steps)
    warm = 3 if args.warmup is None else args.warmup
    gal, lin, probes_g, probes_l = [], [], [], []
    for _ in range(warm):
        for k in reqs:
            idx.probe_prefix(0, k)
    for _ in range(reps):
        for k in reqs:
            t0 = time.perf_counter()
            e, pg = idx.probe_prefix(0, k)
            gal.append(time.perf_counter() - t0)
            t0 = time.perf_counter()
            e2, pl = idx.probe_prefix_linear(0, k)
            lin.append(time.perf_counter() - t0)
            assert e == e2
            probes_g.append(pg)
            probes_l.append(pl)
    med = float(np.median(gal)) * 1e6
    res = {
        "metric": "reuse-hint prefix probe latency on the host (median, gallop + bisect)",
        "value": round(med, 3),
        "unit": "us",
        "n_gpus": 1,
        "steps": reps,
        "warmup": warm,
        "ms_per_step": round(float(np.sum(gal)) * 1e3 / reps, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "uint64",
        "data": "synthetic",
        "config": {"workload": f"{n_req} cached prompts of {prompt} tokens (blocks of {block}, 8 shared-prefix "
                               f"families) in a 64-shard index; {n_req} request prompts probed",
                   "global_batch": n_req, "parallelism": "none (host)"},
        "p99_us": round(float(np.percentile(gal, 99)) * 1e6, 3),
        "median_probes": int(np.median(probes_g)),
        "linear_scan_median_us": round(float(np.median(lin)) * 1e6, 3),
        "linear_scan_median_probes": int(np.median(probes_l)),
        "hash_ms_per_request": round(float(np.median(t_hash)) * 1e3, 3),
        "hash_MBps": round(prompt * 4 / float(np.median(t_hash)) / 1e6, 1),
        "index_entries": idx.size(),
        "roofline": None,
    }
    if not args.no_cpu_baseline:
        ref = ohi.HintIndex()
        for keys in cached:
            ref.add(0, [int(x) for x in keys])
        t0 = time.perf_counter()
        times = []
        for k in reqs:
            kl = [int(x) for x in k]
            t1 = time.perf_counter()
            ohi.prefix_endpoint(ref, 0, kl)
            times.append(time.perf_counter() - t1)
        res["cpu_baseline"] = {"value": round(float(np.median(times)) * 1e6, 3), "unit": "us", "cores": 1,
                               "kind": "oracle", "sample": f"the {n_req} request prompts, plain scan in the reference",
                               "seconds": round(time.perf_counter() - t0, 3)}
    print(json.dumps(res), flush=True)


def _pmc_pass(counters, config, calib_mib):
    """One rocprofv3 counter pass over a short child run of this config; returns the CSV rows."""
    import csv
    import subprocess
    import tempfile
    d = tempfile.mkdtemp(prefix=f"wavepp_{counters[0].lower()}_", dir=os.environ.get("TMPDIR", "/tmp"))
    cmd = ["rocprofv3", "--pmc", *counters, "-f", "csv", "-d", d, "-o", "run", "--",
           sys.executable, os.path.abspath(__file__), "--config", str(config), "--steps", "2", "--warmup", "1",
           "--no-cpu-baseline", "--extras", "none", "--copy-calibration-mib", str(calib_mib)]
    print("[traffic] " + " ".join(cmd), flush=True)
    res = subprocess.run(cmd, cwd=os.environ.get("TMPDIR", "/tmp"), timeout=300)
    rows = []
    for root, _, files in os.walk(d):
        for f in files:
            if f.endswith("counter_collection.csv"):
                rows += list(csv.DictReader(open(os.path.join(root, f))))
    if not rows:
        print(f"[traffic] no counter rows for {counters} (rc={res.returncode})", file=sys.stderr)
    return rows


def measure_traffic(config, out_json, calib_mib=1024):
    """rocprofv3 counter passes over a short run of this config: FETCH_SIZE, then WRITE_SIZE (HBM
    bytes), then MfmaUtil, then TCC_HIT_sum and TCC_MISS_sum (L2 hit rate), then SQ_LDS_BANK_CONFLICT
    and SQ_INSTS_LDS (LDS bank-conflict cycles and LDS instructions).

    Each byte counter is scaled by what it reads for one plain device copy of calib_mib MiB in the
    same process (known bytes / counted bytes), then averaged over the kernel's launches.  The GPU is
    not touched by this process itself: the profiled runs are child processes.
    """
    kind = "kda" if str(config).startswith("kda") else "attn"
    kname = "kda_prefill" if kind == "kda" else "attn_"
    out = {"config": str(config), "kernel_source_hash": _kernel_hash(kind), "calibration_copy_mib": calib_mib}
    known_kib = calib_mib * 1024.0
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        rows = _pmc_pass([counter], config, calib_mib)
        if not rows:
            return 1
        vals = [float(r["Counter_Value"]) for r in rows if kname in r["Kernel_Name"]]
        copy = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not vals or not copy:
            print("[traffic] kernel or calibration copy missing from the counter rows", file=sys.stderr)
            return 1
        calib = max(copy)          # the 1 GiB calibration copy; other device copies are far smaller
        factor = known_kib / calib
        out[counter] = {"kib_per_launch": sum(vals) / len(vals), "launches": len(vals),
                        "calibration_kib": calib, "factor": factor,
                        "bytes_per_launch": sum(vals) / len(vals) * factor * 1024.0}
    out["bytes_per_launch"] = out["FETCH_SIZE"]["bytes_per_launch"] + out["WRITE_SIZE"]["bytes_per_launch"]
    rows = _pmc_pass(["MfmaUtil"], config, calib_mib)
    util = [float(r["Counter_Value"]) for r in rows if kname in r["Kernel_Name"] and r["Counter_Name"] == "MfmaUtil"]
    if util:
        out["mfma_util_pct"] = sum(util) / len(util)
    rows = _pmc_pass(["TCC_HIT_sum", "TCC_MISS_sum"], config, calib_mib)
    hit = sum(float(r["Counter_Value"]) for r in rows if kname in r["Kernel_Name"] and r["Counter_Name"] == "TCC_HIT_sum")
    miss = sum(float(r["Counter_Value"]) for r in rows if kname in r["Kernel_Name"] and r["Counter_Name"] == "TCC_MISS_sum")
    if hit + miss > 0:
        out["l2_hit_pct"] = 100.0 * hit / (hit + miss)
    rows = _pmc_pass(["SQ_LDS_BANK_CONFLICT", "SQ_INSTS_LDS"], config, calib_mib)
    for cname, key in (("SQ_LDS_BANK_CONFLICT", "lds_bank_conflict_cycles_per_launch"),
                       ("SQ_INSTS_LDS", "lds_instructions_per_launch")):
        v = [float(r["Counter_Value"]) for r in rows if kname in r["Kernel_Name"] and r["Counter_Name"] == cname]
        if v:
            out[key] = sum(v) / len(v)
    out["command"] = (f"python bench.py --config {config} --measure-traffic <out.json>  (rocprofv3 --pmc passes "
                      f"FETCH_SIZE; WRITE_SIZE; MfmaUtil; TCC_HIT_sum TCC_MISS_sum; SQ_LDS_BANK_CONFLICT SQ_INSTS_LDS, each "
                      f"over: python3 bench.py --config {config} --steps 2 --warmup 1 --no-cpu-baseline --extras none "
                      f"--copy-calibration-mib {calib_mib})")
    with open(out_json, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out), flush=True)
    return 0


def _code_only(text: str) -> str:
    """C/C++ source without comments and with whitespace collapsed (string literals kept as they are)."""
    import re
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c == '"' or c == "'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return re.sub(r"\s+", " ", "".join(out)).strip()


def _kernel_hash(kind="attn", read=None):
    """Hash of the code (comments and layout ignored) that decides a kernel's memory traffic: its kernel
    file, its planner and the shared layout header."""
    import hashlib
    read = read or (lambda f: open(os.path.join(ROOT, "paper_2609_35263_amd", "csrc", f)).read())
    h = hashlib.sha256()
    files = ("kernels.hip", "host.cpp", "internal.h") if kind == "attn" else ("kda.hip", "kda_host.cpp", "internal.h")
    for f in files:
        h.update(_code_only(read(f)).encode())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
