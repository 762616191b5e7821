"""End-to-end parity of sr_generate against the oracle.

fp32 tiny configuration: the oracle runs the whole algorithm independently;
the GPU must return the same candidate, tokens, rounds and survivors, with
rewards within 1e-4 max|x|.  bf16 configurations: the GPU drives and the
oracle audits its trace -- the cut on the GPU's scores, the sampler on the
GPU's logits, the answer on the GPU's final rewards (all bit-exact), and
teacher-forced logits and rewards on the GPU's sequences (within 2e-2 max|x|).
"""
import numpy as np
import pytest

from gpu_util import check_trace_logic, device_models, need_gpu, oracle_models, say, tol, trace_rounds
from oracle import sampler as osamp
from oracle import specrej

pytestmark = pytest.mark.gpu

# A head-dim-128 pair small enough for the oracle: its first round (300 rows)
# runs the 32-key streaming decode attention with the batched prefix pass
# and the QKV finalize fused into it, the later rounds the 64-key form; two
# cuts compact the generator's and the reward model's caches.
import synth  # noqa: E402

synth.CONFIGS.setdefault(
    "hd128_bf16",
    synth.RunConfig("hd128_bf16", synth.ModelShape(2, 1024, 8, 2, 128, 512, 1000, "bf16", 500000.0),
                    40, 300, 16, 0.8, 128))


def gpu_run(name, reward_kind=0, reward_recompute=0, **over):
    torch, sr = need_gpu()
    c, gen, rm, prompt = device_models(name)
    c = c.with_(**over)
    p = sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens, c.temperature, c.sample_seed, c.eos_id, c.max_rounds,
                       reward_kind=reward_kind, reward_recompute=reward_recompute)
    out = sr.generate(gen, None if reward_kind else rm, prompt, p, trace=True)
    return c, prompt, out


@pytest.mark.parametrize("over", [{}, {"eos_id": 2}, {"max_rounds": 1}, {"alpha": 0.0},
                                  {"n": 40, "alpha": 0.1, "tau": 4, "max_new_tokens": 24}])
def test_tiny_fp32_matches_full_oracle(over):
    say(f"tiny_fp32 e2e {over}")
    c, prompt, out = gpu_run("tiny_fp32", **over)
    rounds = check_trace_logic(c, out)
    g, rm = oracle_models("tiny_fp32")
    ref = specrej.speculative_rejection(g, rm, prompt, c.n, c.alpha, c.tau, c.max_new_tokens, c.temperature,
                                        c.sample_seed, c.eos_id, c.max_rounds)
    t = out["trace"]
    # every candidate's tokens
    for k in range(c.n):
        assert t["all_tokens"][k, : t["all_len"][k]].tolist() == ref["responses"][k], k
    assert [(L, b, K) for (L, b, K, *_rest) in rounds] == [r[:3] for r in ref["rounds"]]
    for (L, b, K, cand, scores, acc), (rL, rb, rK, racc, rsc) in zip(rounds, ref["rounds"]):
        assert cand == sorted(rsc)
        want = np.array([rsc[k] for k in cand])
        assert np.abs(scores - want).max() <= 1e-4 * np.abs(want).max()
        assert sorted(k for k, a in zip(cand, acc) if a) == sorted(racc)
    assert out["best_index"] == ref["best"] and out["tokens"] == ref["tokens"]
    final = np.array(list(ref["final"].values()))
    assert abs(out["best_score"] - ref["score"]) <= 1e-4 * np.abs(final).max()
    fs = t["final_scores"]
    assert sorted(k for k in range(c.n) if not np.isnan(fs[k])) == sorted(ref["final"])
    got = np.array([fs[k] for k in ref["final"]])
    assert np.abs(got - final).max() <= 1e-4 * np.abs(final).max()
    assert out["generated_tokens"] == ref["generated"]
    if c.eos_id < 0:
        assert out["generated_tokens"] == specrej.schedule(c.n, c.alpha, c.tau, c.max_new_tokens, c.max_rounds)[1]


@pytest.mark.parametrize("name,over,rtol", [("tiny_fp32", {}, 1e-5), ("tiny_fp32", {"eos_id": 2}, 1e-5),
                                             ("small_bf16", {}, 2e-2), ("hd128_bf16", {}, 2e-2)])
def test_reward_cache_matches_recompute(name, over, rtol):
    """Scoring through the reward model's cached K/V of the survivors and
    re-running whole responses give the same first-round scores bit for bit
    (the same arithmetic), later-round scores within rounding, and the same
    run wherever the cuts agree."""
    say(f"{name} reward cache vs recompute {over}")
    c, _, a = gpu_run(name, **over)
    _, _, b = gpu_run(name, reward_recompute=1, **over)
    ra, rb = trace_rounds(a), trace_rounds(b)
    assert len(ra) >= 2
    assert np.array_equal(ra[0][4], rb[0][4])
    for x, y in zip(ra, rb):
        if x[:4] != y[:4]:
            break
        assert np.abs(x[4] - y[4]).max() <= rtol * np.abs(y[4]).max(), x[0]
    if [x[:4] for x in ra] == [y[:4] for y in rb] and all(np.array_equal(x[5], y[5]) for x, y in zip(ra, rb)):
        fa, fb = a["trace"]["final_scores"], b["trace"]["final_scores"]
        assert np.array_equal(np.isnan(fa), np.isnan(fb))
        m = ~np.isnan(fa)
        assert np.abs(fa[m] - fb[m]).max() <= rtol * np.abs(fb[m]).max()
        assert a["generated_tokens"] == b["generated_tokens"]
        # the answer agrees unless two members tie within rounding
        if a["best_index"] != b["best_index"]:
            assert abs(fb[a["best_index"]] - fb[b["best_index"]]) <= 2 * rtol * np.abs(fb[m]).max()


def test_diagnostics_against_best_of_n():
    """Section 5 / Appendix B diagnostics of a run against Best-of-N at the
    same seed.  Until the first cut both runs decode the same N rows through
    the same kernels, so every candidate's first tau tokens agree bit for bit
    and the first cut ranks partial rewards of exactly Best-of-N's prefixes.
    After a cut the batch shrinks and the kernels' summation order changes
    with it (split counts, row groups), so a survivor's continuation can leave
    Best-of-N's where a rounding difference moves a sampling decision (the
    oracle, in exact arithmetic, keeps them equal).  Where the answer's
    response is Best-of-N's response of the same candidate, its reward is
    Best-of-N's and the improvement score is at most 100."""
    torch, sr = need_gpu()
    say("small_bf16 diagnostics vs best-of-N")
    c, _, a = gpu_run("small_bf16")
    _, _, b = gpu_run("small_bf16", alpha=0.0)
    ta, tb = a["trace"], b["trace"]
    for k in range(c.n):
        la = min(int(ta["all_len"][k]), c.tau)
        assert ta["all_tokens"][k, :la].tolist() == tb["all_tokens"][k, :la].tolist(), k
    L0, b0, K0, cand0, partial, _ = trace_rounds(a)[0]
    assert L0 == c.tau and b0 == c.n and cand0 == list(range(c.n))
    final = tb["final_scores"]
    assert not np.isnan(final).any()
    pr, kd = sr.correlation(partial, final)
    from oracle import diagnostics as dg
    assert abs(pr - dg.pearson(partial, final)) < 1e-9 and abs(kd - dg.kendall(partial, final)) < 1e-12
    assert -1.0 <= pr <= 1.0 and -1.0 <= kd <= 1.0
    best = a["best_index"]
    n = int(ta["all_len"][best])
    if ta["all_tokens"][best, :n].tolist() == tb["all_tokens"][best, :int(tb["all_len"][best])].tolist():
        assert abs(a["best_score"] - final[best]) <= tol(c) * np.abs(final).max()
        score = sr.improvement_score(final, a["best_score"])
        assert score <= 100.0 + 100.0 * tol(c) * np.abs(final).max() / (final.max() - final.min())


def test_memory_planned_run_matches_given_budget():
    """Algorithm 1's memory-driven sizing on the device: with exactly the
    workspace of tau = 16 available, the planner picks tau = 16 and the run is
    the one with that budget given; with the device's free memory it picks the
    largest tau that fits, and the run completes within that workspace."""
    torch, sr = need_gpu()
    say("memory-planned tiny_fp32 run")
    c, gen, rm, prompt = device_models("tiny_fp32")
    p = sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens, c.temperature, c.sample_seed)
    need = sr.workspace_size(gen, rm, len(prompt), p)
    q = sr.plan_for_memory(gen, rm, len(prompt), p, need)
    assert (q.n, q.tau) == (c.n, c.tau)
    a = sr.generate(gen, rm, prompt, p)
    b = sr.generate(gen, rm, prompt, q)
    assert a["tokens"] == b["tokens"] and a["best_index"] == b["best_index"] and a["rounds"] == b["rounds"]
    free, _ = torch.cuda.mem_get_info()
    big = sr.plan_for_memory(gen, rm, len(prompt), p, free // 2)
    assert big.tau == c.max_new_tokens          # a tiny model fits every budget: one round, as Best-of-N
    o = sr.generate(gen, rm, prompt, big)
    assert o["rounds"] == 0 and o["generated_tokens"] == c.n * c.max_new_tokens


@pytest.mark.parametrize("name", ["small_bf16", "hd128_bf16"])
def test_bf16_audit(name):
    torch, sr = need_gpu()
    say(f"{name} e2e audit")
    c, prompt, out = gpu_run(name)
    rounds = check_trace_logic(c, out)
    sched, total = specrej.schedule(c.n, c.alpha, c.tau, c.max_new_tokens)
    assert [(L, b, K) for (L, b, K, *_rest) in rounds] == sched
    assert out["generated_tokens"] == total
    t = out["trace"]
    _, gen, rm, _ = device_models(name)
    g, orm = oracle_models(name)
    # (1) the sampler on the GPU's own first-round logits reproduces its tokens
    toks = t["all_tokens"][:, : c.tau].astype(np.int32)
    p = sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens)
    ws = sr.Workspace(gen, rm, len(prompt), p)
    lg = sr.logits_teacher_forced(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), ws).cpu().numpy()
    for k in range(c.n):
        for step in range(c.tau):
            assert osamp.sample(lg[k, step], c.temperature, c.sample_seed, k, step) == toks[k, step], (k, step)
    # (2) those logits match the float64 oracle on the same sequences
    for k in (0, c.n // 2, c.n - 1):
        ref = g.logits(list(prompt) + list(toks[k]))[len(prompt) - 1: len(prompt) - 1 + c.tau]
        assert np.abs(lg[k] - ref).max() <= tol(c) * np.abs(ref).max()
    # (3) partial rewards of every candidate at every cut, recomputed by the
    # oracle (the rounds after the first score through the reward model's
    # cached K/V), within the tolerance of the cut's whole reward vector
    assert len(rounds) >= 2
    for (L0, b0, K0, cand0, sc0, acc0) in rounds:
        refs = np.array([orm.score(list(prompt) + t["all_tokens"][cand0[j], :L0].tolist()) for j in range(b0)])
        err = np.abs(sc0 - refs)
        assert err.max() <= tol(c) * np.abs(refs).max(), (L0, int(err.argmax()))
    # (4) final rewards of I, recomputed by the oracle
    fs = t["final_scores"]
    mem = [k for k in range(c.n) if not np.isnan(fs[k])]
    refs = np.array([orm.score(list(prompt) + t["all_tokens"][k, : t["all_len"][k]].tolist()) for k in mem])
    assert np.abs(fs[mem] - refs).max() <= tol(c) * np.abs(refs).max()


@pytest.mark.parametrize("over", [{}, {"eos_id": 2}, {"n": 40, "alpha": 0.1, "tau": 4, "max_new_tokens": 24}])
def test_tiny_fp32_logprob_reward_matches_full_oracle(over):
    """Probability as the reward (section 5.3), no reward model: the GPU's
    candidates, cuts and answer equal the oracle's run with the mean
    log-probability score."""
    say(f"tiny_fp32 logprob e2e {over}")
    c, prompt, out = gpu_run("tiny_fp32", reward_kind=1, **over)
    rounds = check_trace_logic(c, out)
    g, _ = oracle_models("tiny_fp32")
    lp = lambda pr, toks: specrej.mean_logprob(g, pr, toks)
    ref = specrej.speculative_rejection(g, None, prompt, c.n, c.alpha, c.tau, c.max_new_tokens, c.temperature,
                                        c.sample_seed, c.eos_id, c.max_rounds, score_fn=lp)
    t = out["trace"]
    for k in range(c.n):
        assert t["all_tokens"][k, : t["all_len"][k]].tolist() == ref["responses"][k], k
    assert [(L, b, K) for (L, b, K, *_rest) in rounds] == [r[:3] for r in ref["rounds"]]
    for (L, b, K, cand, scores, acc), (rL, rb, rK, racc, rsc) in zip(rounds, ref["rounds"]):
        want = np.array([rsc[k] for k in cand])
        assert np.abs(scores - want).max() <= 1e-4 * np.abs(want).max()
        assert sorted(k for k, a in zip(cand, acc) if a) == sorted(racc)
    assert out["best_index"] == ref["best"] and out["tokens"] == ref["tokens"]
    final = np.array(list(ref["final"].values()))
    assert abs(out["best_score"] - ref["score"]) <= 1e-4 * np.abs(final).max()


def test_profiled_run_matches_unprofiled():
    """Event timing of the launches (profile_every > 0) changes no result,
    times every launch of the profiled decode steps (one decode-attention
    record per layer and step) plus every reward and cut launch, and reads
    its event batches back without loss."""
    torch, sr = need_gpu()
    c, gen, rm, prompt = device_models("hd128_bf16")
    say("hd128_bf16 profiled vs unprofiled")
    runs = []
    for every in (0, 3):
        p = sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens, c.temperature, c.sample_seed, c.eos_id,
                           c.max_rounds, profile_every=every)
        runs.append(sr.generate(gen, rm, prompt, p))
    a, b = runs
    assert a["tokens"] == b["tokens"]
    assert a["best_index"] == b["best_index"] and a["best_score"] == b["best_score"]
    assert all(k["launches"] == 0 for k in a["kernels"].values())
    kb = b["kernels"]
    profiled_steps = [s for s in range(1, c.max_new_tokens) if s % 3 == 0]
    assert kb["decode_attn"]["launches"] == c.model.n_layers * len(profiled_steps)
    # (300 rows and fewer: every decode projection is in the weight-bound class)
    assert kb["gen_gemm_mfma"]["launches"] == 0
    for name in ("gen_gemm_hbm", "decode_attn", "rm_gemm", "prefill_attn", "sample", "cut"):
        assert kb[name]["launches"] > 0 and kb[name]["sec"] > 0 and kb[name]["bytes"] > 0, name
