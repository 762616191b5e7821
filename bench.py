"""Benchmark of the Speculative Rejection hot path on one MI355X.

One step = one sr_generate call: the whole hot path (prompt prefill of both
models, batched decode of N candidates, reward-model scoring at every
decision token, the rejection cuts and KV compaction, the final arg max) for
one prompt.  Default workload: the 8B-shaped generator and reward model
(32 layers, d=4096, 32/8 heads, hd=128, ffn 14336, vocab 128256; bf16,
random N(0, 0.02) weights), a 256-token random prompt, N=512, tau=128,
alpha=0.8, 1024 new tokens, temperature 1, no EOS.

Reports generator tokens/s (sampled response tokens / seconds per prompt),
seconds per prompt, the same for alpha=0 (Best-of-N at equal N) and the
speedup, the roofline of the dominant kernel class measured with HIP events
during the timed steps, and the CPU oracle on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "generator tokens/s and s/prompt at N, α (vs α=0 Best-of-N); % HBM/MFMA peak"
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
FP32_VECTOR_TFLOPS = 157.3
# kernel class -> (bound, unit) for the implementation in this library
BOUNDS = {
    "gen_gemm_mfma": ("mfma", "TFLOP/s"), "gen_gemm_hbm": ("hbm", "GB/s"), "decode_attn": ("hbm", "GB/s"),
    "rm_gemm": ("mfma", "TFLOP/s"), "prefill_attn": ("mfma", "TFLOP/s"), "sample": ("hbm", "GB/s"),
    "cut": ("hbm", "GB/s"), "other": ("hbm", "GB/s"),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def device_clocks(libhandle):
    """Peak engine and memory clocks the HIP runtime reports for device 0
    (MHz), with the engine clock the counters measured under the matrix-core
    bound reward-model GEMMs (profiles/mfma_batched_gemms.json) for context.
    The runtime is reached through the library's handle (its dependency
    scope), so the process keeps the one HIP runtime it already has."""
    import ctypes
    out = {}
    try:
        get = libhandle.hipDeviceGetAttribute
    except AttributeError:
        get = None
    if get is not None:
        v = ctypes.c_int()
        # hipDeviceAttributeClockRate = 5, hipDeviceAttributeMemoryClockRate = 60 (kHz)
        for key, attr in (("sclk_peak_mhz", 5), ("mclk_peak_mhz", 60)):
            if get(ctypes.byref(v), attr, 0) == 0:
                out[key] = v.value // 1000
    try:
        with open(os.path.join(ROOT, "profiles", "mfma_batched_gemms.json")) as f:
            d = json.load(f)
        out["sclk_under_mfma_load_ghz"] = d["reward_model_32768_rows"]["w13"]["sustained_clock_ghz"]
        out["sclk_under_mfma_load_source"] = "profiles/mfma_batched_gemms.json (GRBM_GUI_ACTIVE per XCD / launch time)"
    except (OSError, KeyError, ValueError):
        pass
    return out or None


def roofline_of(name, k, dtype):
    bound, unit = BOUNDS[name]
    if k["sec"] <= 0:
        return None
    if unit == "GB/s":
        achieved, peak = k["bytes"] / k["sec"] / 1e9, PEAK_HBM_GBS
    else:
        achieved = k["flops"] / k["sec"] / 1e12
        peak = FP32_VECTOR_TFLOPS if bound == "alu" else PEAK_TFLOPS[dtype]
    return {"kernel": name, "bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": None,
            "avg_launch_us": round(k["sec"] / max(1, k["launches"]) * 1e6, 2), "launches_timed": k["launches"]}


def load_traffic(kernel_class):
    """HBM traffic per launch of a kernel class from the committed PMC
    summary (profiles/traffic_*.json, written from rocprofv3 --pmc runs of
    FETCH_SIZE and WRITE_SIZE scaled by a copy of known size), if it was
    taken for this class; None otherwise."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    return {"bytes_per_launch": d["traffic_bytes_per_launch"], "source": os.path.relpath(path, ROOT)}


def _cpu_info():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count()
    try:
        from threadpoolctl import threadpool_info
        threads = max(i.get("num_threads", 1) for i in threadpool_info()) or 1
    except Exception:
        threads = nproc
    return model, nproc, threads


def cpu_baseline(cfg, gw, rw, kind, rows=4, steps=2, full_below=5e7):
    """The oracle on the host cores.  Small models: the oracle's whole
    Speculative Rejection run, timed end to end.  Large ones: a bounded
    sample, extrapolated to one prompt with the schedule's closed-form step
    counts -- the prompt forward of the generator (untimed weight widening
    beforehand), which gives the cost of a forward pass per token, and
    `steps` decode steps at `rows` candidates, which gives the cost of a
    decode step when the weights, not the rows, bound it; a decode step of
    b rows is charged max(that, b x the per-token forward cost), a reward
    round of b rows at length L b x (P + L) tokens of forward (the oracle
    scores every partial sequence from its first token, with the same-shape
    reward model, or with the generator for the mean log-probability)."""
    import numpy as np

    import synth
    from oracle import specrej
    from oracle.sampler import sample
    from oracle.transformer import Transformer

    model, nproc, threads = _cpu_info()
    m = cfg.model
    prompt = [int(x) for x in synth.prompt(cfg)]
    P = len(prompt)
    nparams = sum(int(np.prod(np.shape(v))) for v in gw.values())
    base = {"unit": "tokens/s", "cores": threads, "nproc": nproc, "cpu_model": model, "kind": "oracle"}
    if nparams < full_below:
        g = Transformer(m, gw, False)
        r = None if kind == "logprob" else Transformer(m, rw, True)
        lp = (lambda pr, toks: specrej.mean_logprob(g, pr, toks)) if kind == "logprob" else None
        t0 = time.perf_counter()
        out = specrej.speculative_rejection(g, r, prompt, cfg.n, cfg.alpha, cfg.tau, cfg.max_new_tokens,
                                            cfg.temperature, cfg.sample_seed, cfg.eos_id, cfg.max_rounds,
                                            score_fn=lp)
        dt = time.perf_counter() - t0
        return dict(base, value=round(out["generated"] / dt, 4), s_per_prompt=round(dt, 3),
                    sample=f"the oracle's whole run (float64 numpy), {out['generated']} tokens in {dt:.1f} s")
    g = Transformer(m, gw, False, cache_f64=True)
    for name in ("embed", "final_norm", "head"):
        g.w(name)
    for name in ("attn_norm", "wqkv", "wo", "ffn_norm", "w13", "w2"):
        for l in range(m.n_layers):
            g.w(name, l)
    t0 = time.perf_counter()
    state, l0 = g.start(prompt, rows, P + steps + 1)
    t_prompt = time.perf_counter() - t0
    toks = [sample(np.float32(l0), cfg.temperature, cfg.sample_seed, k, 0) for k in range(rows)]
    t0 = time.perf_counter()
    for s in range(1, steps + 1):
        lg = g.step(state, toks)
        toks = [sample(np.float32(lg[k]), cfg.temperature, cfg.sample_seed, k, s) for k in range(rows)]
    t_step = (time.perf_counter() - t0) / steps
    c_tok = t_prompt / P

    def extrapolate(alpha):
        rounds, total = specrej.schedule(cfg.n, alpha, cfg.tau, cfg.max_new_tokens, cfg.max_rounds)
        sec, b, L = t_prompt, cfg.n, 0
        for (Lr, br, K) in rounds + [(cfg.max_new_tokens, None, None)]:
            sec += (Lr - L) * max(t_step, b * c_tok)
            L = Lr
            if br is None:
                break
            sec += br * (P + Lr) * c_tok
            b = K
        sec += b * (P + cfg.max_new_tokens) * c_tok
        return sec, total

    sr_s, sr_tokens = extrapolate(cfg.alpha)
    bon_s, _ = extrapolate(0.0)
    return dict(base, value=round(sr_tokens / sr_s, 4), s_per_prompt=round(sr_s, 1),
                bon_s_per_prompt=round(bon_s, 1), extrapolated=True,
                sample=f"extrapolated: oracle (float64 numpy) prompt forward of {P} tokens {t_prompt:.1f} s and "
                       f"{steps} decode steps at {rows} candidates {t_step:.2f} s each, weights widened beforehand "
                       f"(untimed); a step of b rows costs max({t_step:.2f} s, b x {c_tok:.3f} s), a reward round "
                       f"b x (P + L) tokens x {c_tok:.3f} s, over the schedule's rounds")


def counter_workload(cfg, gen, rm, prompt, case="all"):
    """The hot path's kernels at the configuration's shapes in runs short
    enough for rocprofv3 --pmc (which does not complete a whole call of the
    8B-shaped pair on this software stack): one calibration kernel of known
    bytes; the generator's decode step (the library's own decode path, via
    sr_logits_teacher_forced) at every row count of the schedule; decode
    attention (sr_decode_attention) at each decode phase's row count and mean
    tail length; the reward model's four projections (sr_projection) at the
    row count of a scoring chunk.  `case` picks one group ("decode",
    "attention", "rm") or all; prints what ran, one line per case."""
    import numpy as np
    import torch

    import paper_2410_20290_amd as sr
    from oracle.specrej import schedule

    m = cfg.model
    dev = "cuda"
    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    del src, dst
    print(json.dumps({"case": "calibration", "read_bytes": 1 << 30, "write_bytes": 1 << 30}), flush=True)
    rounds, _ = schedule(cfg.n, cfg.alpha, cfg.tau, cfg.max_new_tokens, cfg.max_rounds)
    phases, L = [], 0
    b = cfg.n
    for (Lr, br, K) in rounds + [(cfg.max_new_tokens, None, None)]:
        phases.append((b, L, Lr))
        L = Lr
        if K is not None:
            b = K
    P = len(prompt)
    steps = 8
    for (rows, L0, L1) in (phases if case in ("all", "decode") else []):
        p = sr.make_params(rows, 0.0, steps, steps)
        ws = sr.Workspace(gen, rm, P, p)
        toks = torch.from_numpy(np.random.default_rng(0).integers(0, m.vocab, size=(rows, steps)).astype(np.int32))
        out = sr.logits_teacher_forced(gen, rm, prompt, p, toks.to(dev), ws)
        torch.cuda.synchronize()
        del out, ws
        torch.cuda.empty_cache()
        print(json.dumps({"case": "decode_step", "rows": rows, "steps": steps}), flush=True)
    bf = torch.bfloat16
    for (rows, L0, L1) in (phases if case in ("all", "attention") else []):
        lt = (L0 + L1) // 2
        cap = (lt + 63) // 64 * 64
        q = torch.randn(rows, m.n_heads, m.head_dim, device=dev)
        kp = torch.randn(m.n_kv_heads, P, m.head_dim, device=dev).to(bf).view(torch.int16)
        vp = torch.randn(m.n_kv_heads, P, m.head_dim, device=dev).to(bf).view(torch.int16)
        kt = torch.randn(rows, m.n_kv_heads, cap, m.head_dim, device=dev).to(bf).view(torch.int16)
        vt = torch.randn(rows, m.n_kv_heads, cap, m.head_dim, device=dev).to(bf).view(torch.int16)
        o = torch.empty(rows, m.n_heads * m.head_dim, dtype=torch.int16, device=dev)
        for _ in range(4):
            sr.decode_attention(q, kp, vp, kt, vt, lt, o)
        torch.cuda.synchronize()
        del q, kp, vp, kt, vt, o
        torch.cuda.empty_cache()
        print(json.dumps({"case": "decode_attention", "rows": rows, "P": P, "lt": lt, "launches": 4}), flush=True)
    if rm is not None and case in ("all", "rm"):
        M = min(32768, cfg.n * cfg.tau)
        x = torch.randn(M, m.d_model, device=dev).to(bf).view(torch.int16)
        u = torch.randn(M, m.ffn_dim, device=dev).to(bf).view(torch.int16)
        qkv_n = m.qkv_dim
        for name, (xin, N, K, mode) in {"qkv": (x, qkv_n, m.d_model, 0), "o": (x, m.d_model, m.d_model, 1),
                                        "w13": (x, m.ffn_dim, m.d_model, 2), "w2": (u, m.d_model, m.ffn_dim, 1)}.items():
            w = (torch.randn(2 if mode == 2 else 1, N, K, device=dev) * 0.02).to(bf).view(torch.int16)
            w = w if mode == 2 else w[0]
            out = torch.zeros(M, N, device=dev, dtype=torch.int16 if mode in (2, 3) else torch.float32)
            for _ in range(2):
                sr.projection(xin, w, mode, out)
            torch.cuda.synchronize()
            print(json.dumps({"case": "rm_projection", "name": name, "M": M, "N": N, "K": K, "mode": mode,
                              "launches": 2}), flush=True)
            del w, out
            torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="8b_bf16")
    ap.add_argument("--alpha", type=float, default=None)
    ap.add_argument("--tau", type=int, default=None)
    ap.add_argument("--profile-every", type=int, default=64)
    ap.add_argument("--no-bon", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--bon-runs", type=int, default=3, help="timed Best-of-N runs after one warm-up (median)")
    ap.add_argument("--cpu-rows", type=int, default=4)
    ap.add_argument("--cpu-steps", type=int, default=2)
    ap.add_argument("--max-new-tokens", type=int, default=None,
                    help="shorter responses (for counter runs of the same kernels; not a bench line)")
    ap.add_argument("--counter-workload", action="store_true",
                    help="run the hot path's kernels at this configuration's shapes in short runs for rocprofv3 "
                         "--pmc (see counter_workload) instead of the benchmark")
    ap.add_argument("--counter-case", default="all", choices=["all", "decode", "attention", "rm"])
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run one elementwise kernel that reads 1 GiB and writes 1 GiB, so a counter run can "
                         "scale FETCH_SIZE / WRITE_SIZE by what they read for a known byte count")
    ap.add_argument("--reward", choices=["model", "logprob"], default="model",
                    help="partial reward: the reward model, or the generator's mean log-probability "
                         "(section 5.3, no reward model)")
    ap.add_argument("--memory-plan", action="store_true",
                    help="take tau from the device's free memory (Algorithm 1, first step): the largest tau whose "
                         "workspace fits in the free HBM after the weights, less 4 GiB")
    ap.add_argument("--reward-recompute", action="store_true",
                    help="run whole responses through the reward model at every decision instead of keeping "
                         "the survivors' reward-model K/V across rounds")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}): the hot path is one GPU's batch of "
              "candidates; see the design notes for how it would shard", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    import paper_2410_20290_amd as sr

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    configs = dict(synth.CONFIGS, **{c.name: c for c in synth.SWEEP_8B_N1024})
    cfg = configs[args.config]
    if args.max_new_tokens is not None:
        cfg = cfg.with_(max_new_tokens=args.max_new_tokens)
    if args.alpha is not None:
        cfg = cfg.with_(alpha=args.alpha)
    if args.tau is not None:
        cfg = cfg.with_(tau=args.tau)
    m = cfg.model
    t = time.time()
    gw = synth.model_weights(m, cfg.gen_seed, False)
    rw = synth.model_weights(m, cfg.rm_seed, True)
    prompt = synth.prompt(cfg)
    log(f"[bench] weights generated in {time.time() - t:.1f}s")
    kind = sr.SR_REWARD_LOGPROB if args.reward == "logprob" else sr.SR_REWARD_MODEL
    gen = sr.DeviceModel.upload(m, gw, False)
    rm = sr.DeviceModel.upload(m, rw, True) if kind == sr.SR_REWARD_MODEL else None
    if sum(int(np.prod(np.shape(v))) for v in gw.values()) >= 5e7:
        rw = None   # the CPU leg runs the whole oracle only for small models
    torch.cuda.synchronize()
    log(f"[bench] weights uploaded ({time.time() - t:.1f}s)")
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()
        log("[bench] calibration kernel: 1 GiB read, 1 GiB written")

    if args.counter_workload:
        counter_workload(cfg, gen, rm, prompt, args.counter_case)
        return
    rrc = 1 if args.reward_recompute else 0
    if args.memory_plan:
        free, _ = torch.cuda.mem_get_info()
        cap = max(0, free - (4 << 30))
        q = sr.plan_for_memory(gen, rm, len(prompt), sr.make_params(cfg.n, cfg.alpha, cfg.tau, cfg.max_new_tokens,
                                                                     reward_kind=kind, reward_recompute=rrc), cap)
        log(f"[bench] memory plan: {free / 2**30:.1f} GiB free -> tau = {q.tau} at N = {q.n}")
        cfg = cfg.with_(tau=q.tau)
    p = sr.make_params(cfg.n, cfg.alpha, cfg.tau, cfg.max_new_tokens, cfg.temperature, cfg.sample_seed,
                       cfg.eos_id, 0, 0, kind, rrc)
    ws = sr.Workspace(gen, rm, len(prompt), p)
    log(f"[bench] workspace {ws.nbytes / 2**30:.2f} GiB")
    warm = None
    for i in range(args.warmup):
        o = sr.generate(gen, rm, prompt, p, ws, trace=i == 0)
        warm = warm or o
        log(f"[bench] warmup {i}: {o['sec_total']:.3f}s generated={o['generated_tokens']}")
    pp = sr.make_params(cfg.n, cfg.alpha, cfg.tau, cfg.max_new_tokens, cfg.temperature, cfg.sample_seed,
                        cfg.eos_id, 0, args.profile_every, kind, rrc)
    kern = {}
    gen_tokens = 0
    results = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        o = sr.generate(gen, rm, prompt, pp, ws)
        results.append(o)
        gen_tokens += o["generated_tokens"]
        for name, k in o["kernels"].items():
            a = kern.setdefault(name, {"sec": 0.0, "launches": 0, "bytes": 0.0, "flops": 0.0})
            for f in a:
                a[f] += k[f]
        log(f"[bench] step {i}: {o['sec_total']:.3f}s (prefill {o['sec_prefill']:.3f} decode {o['sec_decode']:.3f} "
            f"reward {o['sec_reward']:.3f} cut {o['sec_cut']:.3f}) best={o['best_index']} rounds={o['rounds']}")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    s_per_prompt = elapsed / args.steps
    value = gen_tokens / elapsed
    s_median = float(np.median([o["sec_total"] for o in results]))
    del ws
    torch.cuda.empty_cache()

    bon = None
    if not args.no_bon and cfg.alpha > 0:
        pb = sr.make_params(cfg.n, 0.0, cfg.tau, cfg.max_new_tokens, cfg.temperature, cfg.sample_seed,
                            cfg.eos_id, 0, 0, kind, rrc)
        wsb = sr.Workspace(gen, rm, len(prompt), pb)
        ob = sr.generate(gen, rm, prompt, pb, wsb, trace=True)   # warm-up (and the trace)
        log(f"[bench] best-of-N (alpha=0) warm-up: {ob['sec_total']:.3f}s")
        times = []
        for i in range(max(1, args.bon_runs)):
            torch.cuda.synchronize()
            tb = time.perf_counter()
            o = sr.generate(gen, rm, prompt, pb, wsb)
            torch.cuda.synchronize()
            times.append(time.perf_counter() - tb)
            assert o["best_index"] == ob["best_index"]
            log(f"[bench] best-of-N (alpha=0) run {i}: {times[-1]:.3f}s")
        tb = float(np.median(times))
        bon = {"s_per_prompt": round(tb, 4), "runs_s": [round(x, 4) for x in times], "warmup": 1,
               "tokens_per_s": round(ob["generated_tokens"] / tb, 1),
               "generated_tokens": ob["generated_tokens"], "best_index": ob["best_index"],
               "sr_best_index": results[-1]["best_index"]}
        if warm is not None and warm["trace"]["rounds"] > 0:
            # section 5 and Appendix B diagnostics: the first cut's partial
            # rewards against Best-of-N's final rewards of the same candidates
            # (the same seed draws the same responses), the answer's reward on
            # the range of Best-of-N's; values on random weights say nothing
            # about a trained reward model
            b0 = int(warm["trace"]["round_b"][0])
            cand0 = warm["trace"]["round_cand"][0, :b0]
            partial = warm["trace"]["round_scores"][0, :b0]
            final = ob["trace"]["final_scores"][cand0]
            pr, kd = sr.correlation(partial, final)
            bon["diagnostics"] = {
                "pearson_partial_final": round(pr, 4), "kendall_partial_final": round(kd, 4),
                "first_decision_token": int(warm["trace"]["round_L"][0]),
                "improvement_score": round(sr.improvement_score(ob["trace"]["final_scores"],
                                                                 results[-1]["best_score"]), 2),
                "relative_gpu_compute": round(s_per_prompt / tb, 4)}
        del wsb
        torch.cuda.empty_cache()

    # Decode-step launches are timed in 1 of every `profile_every` steps,
    # reward/prefill/cut launches always: scale to estimate each class's
    # share of the run when picking the dominant one.
    decode_classes = {"gen_gemm_mfma", "gen_gemm_hbm", "decode_attn", "sample"}
    kernels = {}
    for name, k in kern.items():
        r = roofline_of(name, k, m.dtype)
        if r:
            r["sec_timed"] = round(k["sec"], 4)
            r["sec_est_per_step"] = round(k["sec"] * (args.profile_every if name in decode_classes else 1)
                                          / args.steps, 4)
            kernels[name] = r
    roof = None
    if kernels:
        dominant = max(kernels, key=lambda n: kernels[n]["sec_est_per_step"])
        roof = dict(kernels[dominant])
        tr = load_traffic(dominant)
        if tr:
            roof["traffic"] = tr["bytes_per_launch"]
            roof["traffic_source"] = tr["source"]
    # the stated per-class goals at the 8B shape, with what this run reached
    targets = {}
    for name, goal in (("decode_attn", 0.70), ("gen_gemm_mfma", 0.50), ("rm_gemm", 0.50)):
        if name in kernels:
            targets[name] = {"frac": kernels[name]["frac"], "target": goal, "unit": kernels[name]["unit"],
                             "met": kernels[name]["frac"] >= goal}

    cpu = None
    if not args.no_cpu:
        del gen, rm
        torch.cuda.empty_cache()
        log("[bench] timing the CPU oracle")
        cpu = cpu_baseline(cfg, gw, rw, args.reward, args.cpu_rows, args.cpu_steps)
        log(f"[bench] CPU oracle: {cpu['sample']}")

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(s_per_prompt * 1e3, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": m.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {m.dtype} generator ({m.n_layers} layers, d {m.d_model}, "
                               f"{m.n_heads}/{m.n_kv_heads} heads x {m.head_dim}, ffn {m.ffn_dim}, vocab {m.vocab}) + "
                               + ("reward model of the same shape" if kind == sr.SR_REWARD_MODEL else
                                  "mean log-probability reward (no reward model)")
                               + f", prompt {cfg.prompt_len}, "
                               f"N={cfg.n}, tau={cfg.tau}, alpha={cfg.alpha}, {cfg.max_new_tokens} new tokens",
                   "reward": args.reward,
                   "tau_from": "free device memory" if args.memory_plan else "given",
                   "reward_kv": "recomputed each round" if (args.reward_recompute or kind != sr.SR_REWARD_MODEL)
                                else "cached across rounds",
                   "N": cfg.n, "alpha": cfg.alpha, "tau": cfg.tau, "max_new_tokens": cfg.max_new_tokens,
                   "prompt_len": cfg.prompt_len},
        "s_per_prompt": round(s_per_prompt, 4),
        "s_per_prompt_median": round(s_median, 4),
        "generated_tokens_per_prompt": results[-1]["generated_tokens"],
        "phases_s": {k: round(results[-1][k], 4) for k in ("sec_prefill", "sec_decode", "sec_reward", "sec_cut")},
        "best_of_n": bon,
        "speedup_vs_alpha0": round(bon["s_per_prompt"] / s_per_prompt, 3) if bon else None,
        "roofline": roof,
        "targets": targets,
        "kernels": kernels,
        "paper_context": "The paper reports Speculative Rejection as 16-32x more efficient than Best-of-N "
                         "(abstract; section 5.1): Best-of-N needs 16 to 32 GPUs to reach the reward Speculative "
                         "Rejection reaches on one, on a DGX node of H100 80 GB GPUs (Llama-3-8B generator, "
                         "Mistral-7B reward model, AlpacaFarm-Eval prompts).  That ratio compares against Best-of-N "
                         "at larger N on several GPUs and is not comparable to speedup_vs_alpha0 (alpha=0 at the "
                         "same N on one GPU).",
        "cpu_baseline": cpu,
        "clocks": device_clocks(sr.lib()),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
