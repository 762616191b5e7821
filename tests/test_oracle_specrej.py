"""Speculative Rejection and Best-of-N in the oracle, pinned to what the paper
fixes: alpha = 0 is Best-of-N (section 5.1), survivors are the top
ceil((1 - alpha) b) by partial reward (section 4.2), the answer is the best
completed candidate (eq. output), the worked example of section 4.1, the
memory-budget schedule's closed forms, and brute force on a 2-token toy."""
import json
import math
import os
from collections import Counter

import numpy as np
import pytest
import torch
from scipy import stats

import synth
from oracle import specrej
from oracle.transformer import Transformer, softmax

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- keep count
def test_keep_count_table():
    for b, alpha, k in load("keep_count.json")["cases"]:
        assert specrej.keep_count(b, alpha) == k, (b, alpha)


def test_keep_count_is_ceil_of_kept_fraction():
    from fractions import Fraction
    for b in range(1, 300):
        for a in (0.0, 0.1, 0.25, 0.3, 0.5, 0.7, 0.75, 0.8, 0.9, 0.95, 0.999):
            exact = Fraction(specrej.alpha_ppm(a), specrej.PPM)
            kept = (1 - exact) * b
            ceil = -(-kept.numerator // kept.denominator)
            assert specrej.keep_count(b, a) == ceil
            assert specrej.keep_count(b, a) >= 1


# ------------------------------------------------- cut vs numpy's quantile
@pytest.mark.parametrize("b,alpha", [(10, 0.7), (16, 0.5), (64, 0.75), (103, 0.8), (512, 0.8), (37, 0.33)])
def test_cut_matches_lower_quantile_threshold(b, alpha):
    """eq. cutoff-threshold / accepted-set with numpy's inverted-CDF quantile:
    keep s >= q when alpha*b is fractional, s > q ("exceeds") when integral."""
    rng = np.random.default_rng(b)
    s = rng.normal(size=b)
    scores = {k: float(s[k]) for k in range(b)}
    K = specrej.keep_count(b, alpha)
    acc = set(specrej.top_k(list(range(b)), scores, K))
    q = np.quantile(s, specrej.alpha_ppm(alpha) / specrej.PPM, method="inverted_cdf")
    integral = (specrej.alpha_ppm(alpha) * b) % specrej.PPM == 0
    ref = {k for k in range(b) if (s[k] > q if integral else s[k] >= q)}
    assert acc == ref


def test_total_order_ties_and_nan():
    scores = {0: 1.0, 1: 2.0, 2: 2.0, 3: float("nan"), 4: -np.inf, 5: 2.0}
    assert specrej.top_k(list(scores), scores, 6) == [1, 2, 5, 0, 4, 3]
    assert specrej.arg_best(scores) == 1
    assert specrej.arg_best({7: float("nan"), 9: float("nan")}) == 7


# ------------------------------------------------------------- the schedule
def test_schedule_closed_forms():
    for c in load("schedule_closed_form.json")["cases"]:
        rounds, total = specrej.schedule(c["n"], c["alpha"], c["tau"], c["lmax"])
        assert [list(r) for r in rounds] == c["rounds"]
        assert total == c["tokens"]
        assert specrej.schedule(c["n"], 0.0, c["tau"], c["lmax"]) == ([], c["bon_tokens"])


def test_schedule_single_round_and_cascade():
    rounds, total = specrej.schedule(16, 0.5, 16, 64, max_rounds=1)
    assert rounds == [(16, 16, 8)] and total == 16 * 16 + 8 * 48
    # alpha small, tau small: after the first cut memory is still full
    # (floor(1600 / 95) = 16 = L), so a second cut follows at once.
    rounds, total = specrej.schedule(100, 0.05, 16, 64)
    assert rounds[0] == (16, 100, 95) and rounds[1] == (16, 95, 91) and rounds[2][:2] == (17, 91)
    L, b = 16, 91
    for (Lr, br, Kr) in rounds[2:]:
        assert Lr >= L and br == b and Kr < br
        assert Lr == L or Lr == min(64, 1600 // br)
        L, b = Lr, Kr


# ------------------------------------------------------------ tiny models
@pytest.fixture(scope="module")
def tiny():
    cfg = synth.CONFIGS["tiny_fp32"]
    g = Transformer(cfg.model, synth.model_weights(cfg.model, cfg.gen_seed, False), False)
    rm = Transformer(cfg.model, synth.model_weights(cfg.model, cfg.rm_seed, True), True)
    return cfg, g, rm, synth.prompt(cfg)


def run_sr(tiny, **kw):
    cfg, g, rm, pr = tiny
    args = dict(n=cfg.n, alpha=cfg.alpha, tau=cfg.tau, max_new=cfg.max_new_tokens,
                temperature=cfg.temperature, seed=cfg.sample_seed, eos_id=-1, max_rounds=0)
    args.update(kw)
    return specrej.speculative_rejection(g, rm, pr, **args)


def test_alpha_zero_is_best_of_n_bit_exact(tiny):
    cfg, g, rm, pr = tiny
    for eos in (-1, 2):
        sr = run_sr(tiny, alpha=0.0, eos_id=eos)
        bon = specrej.best_of_n(g, rm, pr, cfg.n, cfg.max_new_tokens, 1.0, cfg.sample_seed, eos_id=eos)
        assert sr["best"] == bon["best"] and sr["score"] == bon["score"]
        assert sr["responses"] == bon["responses"] and sr["final"] == bon["final"]
        assert sr["rounds"] == [] and sr["generated"] == bon["generated"]


def check_run_invariants(res, alpha, eos_id, bon):
    # survivors of every cut are the top K by partial reward
    for (L, b, K, acc, scores) in res["rounds"]:
        assert K == specrej.keep_count(b, alpha) and len(acc) == K
        order = sorted(scores, key=lambda k: (-scores[k], k))
        assert acc == order[:K]
    # the answer is the best member of I, ties to the lowest id
    best = max(res["final"], key=lambda k: (res["final"][k], -k))
    assert res["best"] == best and res["score"] == res["final"][best]
    # candidate invariance: SR's response of k is a prefix of BoN's (same seed)
    for k, toks in res["responses"].items():
        assert bon["responses"][k][:len(toks)] == toks
    # members of I are complete: EOS-terminated or at the maximum length
    for k in res["final"]:
        toks = res["responses"][k]
        assert (toks and toks[-1] == eos_id) or len(toks) == len(bon["responses"][k]) or \
            (eos_id in toks and toks.index(eos_id) == len(toks) - 1)


def test_sr_run_invariants_and_token_count(tiny):
    cfg, g, rm, pr = tiny
    bon = specrej.best_of_n(g, rm, pr, cfg.n, cfg.max_new_tokens, 1.0, cfg.sample_seed)
    res = run_sr(tiny)
    check_run_invariants(res, cfg.alpha, -1, bon)
    rounds, total = specrej.schedule(cfg.n, cfg.alpha, cfg.tau, cfg.max_new_tokens)
    assert [(L, b, K) for (L, b, K, _, _) in res["rounds"]] == rounds
    assert res["generated"] == total == 512
    assert len(res["final"]) == 4 and all(len(res["responses"][k]) == 64 for k in res["final"])


def test_sr_with_eos(tiny):
    cfg, g, rm, pr = tiny
    bon = specrej.best_of_n(g, rm, pr, cfg.n, cfg.max_new_tokens, 1.0, cfg.sample_seed, eos_id=2)
    res = run_sr(tiny, eos_id=2)
    check_run_invariants(res, cfg.alpha, 2, bon)
    done_early = [k for k, t in res["responses"].items() if t and t[-1] == 2]
    assert done_early, "the seed should produce some EOS-terminated candidates"
    # completed candidates scored at a cut join I whether accepted or not
    L1, b1, K1, acc1, sc1 = res["rounds"][0]
    for k in sc1:
        if res["responses"][k][-1] == 2 and len(res["responses"][k]) <= L1:
            assert k in res["final"] and res["final"][k] == sc1[k]


def test_sr_cascade_cut(tiny):
    cfg, g, rm, pr = tiny
    bon = specrej.best_of_n(g, rm, pr, 40, 24, 1.0, cfg.sample_seed)
    res = run_sr(tiny, n=40, alpha=0.1, tau=4, max_new=24)
    check_run_invariants(res, 0.1, -1, bon)
    rounds, total = specrej.schedule(40, 0.1, 4, 24)
    assert [(L, b, K) for (L, b, K, _, _) in res["rounds"]] == rounds
    assert res["generated"] == total
    assert any(r1[0] == r2[0] for r1, r2 in zip(rounds, rounds[1:])), "expected a cascaded cut"


def test_sr_single_round(tiny):
    cfg, g, rm, pr = tiny
    res = run_sr(tiny, max_rounds=1)
    assert len(res["rounds"]) == 1 and len(res["final"]) == 8
    assert res["generated"] == 16 * 16 + 8 * 48


# ------------------------------------------------------- worked example 4.1
class ScriptedGenerator:
    """Greedy toy generator: every row first emits token 0, then keeps
    emitting 1 + its candidate id."""

    def __init__(self, vocab):
        self.vocab = vocab

    def start(self, prompt, rows, capacity):
        l0 = np.full(self.vocab, -50.0)
        l0[0] = 0.0
        return {"rows": np.arange(rows)}, l0

    def select_rows(self, state, idx):
        return {"rows": state["rows"][np.asarray(idx, dtype=np.int64)]}

    def step(self, state, tokens):
        out = np.full((len(tokens), self.vocab), -50.0)
        out[np.arange(len(tokens)), state["rows"] + 1] = 0.0
        return out


def test_paper_worked_example():
    ex = load("paper_example_sec41.json")
    tau, lmax = 4, 8

    def score(prompt, toks):
        cand = toks[1] - 1
        return ex["final_scores"][cand] if len(toks) == lmax else ex["partial_scores"][cand]

    gen = ScriptedGenerator(8)
    res = specrej.speculative_rejection(gen, None, [1, 2, 3], 2, ex["alpha"], tau, lmax, 0.0, 0,
                                        score_fn=score)
    (L, b, K, acc, scores), = res["rounds"]
    assert (L, b, K) == (tau, 2, ex["keep"])
    assert acc == [0] and min(scores[k] for k in acc) == pytest.approx(ex["c_star"], abs=1e-6)
    assert res["best"] == ex["returned"] and res["score"] == pytest.approx(ex["final_scores"][0], abs=1e-6)
    bon = specrej.best_of_n(gen, None, [1, 2, 3], 2, lmax, 0.0, 0, score_fn=score)
    assert bon["best"] == res["best"]
    # tokens generated: 2 x tau before the cut, then one candidate to the end
    assert res["generated"] == 2 * tau + (lmax - tau)


# -------------------------------------------------- brute force, V = 2 toy
TOY = synth.ModelShape(1, 16, 2, 2, 8, 32, 2, "f32", 10000.0)
TOY_LMAX = 8


@pytest.fixture(scope="module")
def toy():
    g = Transformer(TOY, synth.model_weights(TOY, 0, False, std=0.6), False)
    rm = Transformer(TOY, synth.model_weights(TOY, 1, True, std=0.6), True)
    prompt = [0, 1, 1]
    paths = [tuple((i >> (TOY_LMAX - 1 - t)) & 1 for t in range(TOY_LMAX)) for i in range(2 ** TOY_LMAX)]
    prob, logp = {}, {}
    for p in paths:
        lg = g.logits(prompt + list(p))[len(prompt) - 1:len(prompt) - 1 + TOY_LMAX]
        pr = softmax(lg)[np.arange(TOY_LMAX), list(p)]
        prob[p] = float(np.prod(pr))
        logp[p] = float(np.mean(np.log(pr)))
    reward = {p: rm.score(prompt + list(p)) for p in paths}
    return g, rm, prompt, prob, logp, reward


@pytest.mark.slow
def test_toy_enumeration(toy):
    g, rm, prompt, prob, logp, reward = toy
    assert abs(sum(prob.values()) - 1.0) < 1e-9
    # greedy decoding equals the stepwise arg max of the enumeration
    res = specrej.best_of_n(g, rm, prompt, 1, TOY_LMAX, 0.0, 0)
    path = []
    for t in range(TOY_LMAX):
        lg = g.logits(prompt + path)[-1]
        path.append(int(np.argmax(lg)))
    assert res["tokens"] == path


@pytest.mark.slow
def test_toy_best_of_n_distribution_and_answer(toy):
    g, rm, prompt, prob, logp, reward = toy
    n = 4096
    bon = specrej.best_of_n(g, rm, prompt, n, TOY_LMAX, 1.0, 7)
    sampled = Counter(tuple(t) for t in bon["responses"].values())
    # path frequencies follow the enumerated probabilities (cells with small
    # expectation pooled)
    exp = np.array([prob[p] * n for p in prob])
    obs = np.array([sampled.get(p, 0) for p in prob])
    big = exp >= 5
    e = np.append(exp[big], exp[~big].sum())
    o = np.append(obs[big], obs[~big].sum())
    chi2 = ((o - e) ** 2 / e).sum()
    assert chi2 < stats.chi2.ppf(0.999, len(e) - 1)
    # each sampled path's reward is its enumerated reward; the answer is the
    # best sampled path
    for k, t in bon["responses"].items():
        assert bon["final"][k] == np.float32(reward[tuple(t)])
    best_path = max(sampled, key=lambda p: reward[p])
    assert tuple(bon["tokens"]) == best_path
    # probability-as-reward (section 5.3): the global optimum is the most
    # likely path; Best-of-N finds it whenever it was sampled
    opt = max(logp, key=logp.get)
    lp = lambda pr, toks: logp[tuple(toks)] if len(toks) == TOY_LMAX else 0.0
    bon_lp = specrej.best_of_n(g, rm, prompt, 256, TOY_LMAX, 1.0, 7, score_fn=lp)
    if opt in {tuple(t) for t in bon_lp["responses"].values()}:
        assert tuple(bon_lp["tokens"]) == opt


@pytest.mark.slow
def test_toy_speculative_rejection(toy):
    g, rm, prompt, prob, logp, reward = toy
    n = 512
    res = specrej.speculative_rejection(g, rm, prompt, n, 0.5, 2, TOY_LMAX, 1.0, 7)
    bon = specrej.best_of_n(g, rm, prompt, n, TOY_LMAX, 1.0, 7)
    check_run_invariants(res, 0.5, -1, bon)
    assert [r[:3] for r in res["rounds"]] == [r for r in specrej.schedule(n, 0.5, 2, TOY_LMAX)[0]]
    # every member of I is a full path whose final reward is the enumerated one
    for k in res["final"]:
        assert res["final"][k] == np.float32(reward[tuple(res["responses"][k])])


@pytest.mark.slow
def test_toy_mean_logprob_is_normalised_and_matches_cached_decode(toy):
    """Section 5.3 score: exp(len * score) over all 2^8 full paths sums to
    one; the score of every prefix equals the per-step log-probabilities
    from the KV-cached decode path (a separate code path of the oracle);
    and one step matches torch's log_softmax."""
    g, rm, prompt, prob, logp, reward = toy
    paths = list(prob)
    total = sum(math.exp(TOY_LMAX * specrej.mean_logprob(g, prompt, list(p))) for p in paths)
    assert abs(total - 1.0) < 1e-9
    for p in paths[::37]:
        state, l0 = g.start(prompt, 1, len(prompt) + TOY_LMAX + 1)
        lg, acc = l0, 0.0
        for t, tok in enumerate(p):
            row = np.asarray(lg).reshape(-1)
            acc += row[tok] - (row.max() + math.log(np.exp(row - row.max()).sum()))
            assert specrej.mean_logprob(g, prompt, list(p[:t + 1])) == pytest.approx(acc / (t + 1), abs=1e-12)
            lg = g.step(state, [tok])[0]
    lg = g.logits(prompt + [1, 0])[len(prompt) + 1]
    ref = torch.log_softmax(torch.from_numpy(lg), dim=0).numpy()
    got = specrej.mean_logprob(g, prompt, [1, 0, 1]) * 3 - specrej.mean_logprob(g, prompt, [1, 0]) * 2
    assert got == pytest.approx(ref[1], abs=1e-12)
