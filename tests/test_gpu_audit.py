"""Audits of whole sr_generate runs at every configuration's full size
(section 4.2, Algorithm 1): the GPU drives and the oracle audits its trace.

Bit for bit, from the run's own trace:
  * every cut: the keep count and the survivors are the oracle's top K of the
    GPU's scores (eqs. cutoff-threshold and accepted-set);
  * the answer is the oracle's arg max of the GPU's final rewards over I
    (eq. output);
  * the rounds (L, b, K) and the token count follow the memory-budget
    schedule in closed form;
  * sampling: for the watched candidates (the answer, the runner-up in I and
    the best-ranked candidate each cut rejected), the oracle's sampler applied
    to the very logits rows the run drew from reproduces every response token
    at every step, before and after each cut.
Against the exact (float64) oracle:
  * the run's logits at steps {0, tau - 1, tau, L_r - 1 and L_r of each cut,
    Lmax - 1} of a few watched candidates against the oracle generator
    teacher-forced on the same tokens;
  * those candidates' rewards at every cut they reached and their final
    reward, against the oracle reward model on the same prefixes;
each within max(2e-2 max|x|, 2 D), max|x| the oracle tensor's max-abs and D
the drift of a bf16 model from the exact one on the same tokens: the largest
deviation of the oracle's bf16-operand mode from its exact mode over the
same logits rows, and over the candidate's whole partial-reward curve (every
prefix length) for rewards.  A bf16 model at 16 and 32 layers is itself 2-5 %
of max|x| away from the exact model on these random-init weights (and a
perturbation of float32 size before each bf16 rounding already moves its
logits by ~2 %), so no bf16 evaluation can meet 2e-2 max|x| there; at 4
layers D is far below it and the bound is 2e-2 max|x|.
The float64 oracle runs every layer (weights widened one layer at a time);
it re-runs only a few candidates of the 8B-shaped pair to stay within the
test budget.
"""
import time

import numpy as np
import pytest

from gpu_util import check_trace_logic, device_models, need_gpu, oracle_models, say, tol
from oracle import sampler as osamp
from oracle import specrej

pytestmark = pytest.mark.gpu

# (configuration, overrides, candidates the float64 oracle re-runs)
AUDITS = [
    ("small_bf16", {}, 4),
    ("1b_bf16", {}, 2),
    ("8b_bf16", {}, 1),
    ("8b_bf16_n1024", {"alpha": 0.5, "tau": 64}, 1),
    ("8b_bf16_n1024", {"alpha": 0.9, "tau": 256}, 1),
]


def _run(sr, c, gen, rm, prompt, watch=()):
    p = sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens, c.temperature, c.sample_seed, c.eos_id,
                       c.max_rounds)
    ws = sr.Workspace(gen, rm, len(prompt), p)
    out = sr.generate(gen, rm, prompt, p, ws, trace=True, watch=watch)
    del ws
    return out


def _watch_set(c, out, rounds, n_extra=6):
    """The answer, the runner-up of I, and the best-ranked candidate that
    each cut rejected."""
    t = out["trace"]
    fs = t["final_scores"]
    members = {k: float(fs[k]) for k in range(c.n) if not np.isnan(fs[k])}
    order = specrej.top_k(list(members), members, len(members))
    watch = order[:2]
    for (L, b, K, cand, scores, acc) in rounds:
        rej = [k for k, a in zip(cand, acc) if not a]
        sd = {k: float(s) for k, s in zip(cand, scores)}
        if rej:
            watch.append(specrej.top_k(rej, sd, 1)[0])
    seen = []
    for k in watch:
        if k not in seen:
            seen.append(k)
    return seen[:n_extra]


def _audit_steps(c, rounds, length):
    steps = {0, c.tau - 1, c.tau, c.max_new_tokens - 1}
    for (L, *_rest) in rounds:
        steps |= {L - 1, L}
    return sorted(s for s in steps if 0 <= s < length)


@pytest.mark.parametrize("name,over,n_oracle", AUDITS,
                         ids=[f"{n}-" + "-".join(f"{k}{v}" for k, v in o.items()) for n, o, _ in AUDITS])
def test_full_size_audit(name, over, n_oracle):
    torch, sr = need_gpu()
    t0 = time.time()
    c, gen, rm, prompt = device_models(name)
    c = c.with_(**over)
    say(f"audit {c.name} {over}: N={c.n} P={c.prompt_len} tau={c.tau} alpha={c.alpha} Lmax={c.max_new_tokens}")
    out = _run(sr, c, gen, rm, prompt)
    rounds = check_trace_logic(c, out)
    sched, total = specrej.schedule(c.n, c.alpha, c.tau, c.max_new_tokens)
    assert [(L, b, K) for (L, b, K, *_rest) in rounds] == sched
    assert out["generated_tokens"] == total
    say(f"  run 1: {out['sec_total']:.2f}s, {len(rounds)} cuts, best {out['best_index']}")

    # the same run again, recording the logits rows of the watched candidates
    watch = _watch_set(c, out, rounds)
    again = _run(sr, c, gen, rm, prompt, watch=watch)
    t1, t2 = out["trace"], again["trace"]
    assert again["best_index"] == out["best_index"] and again["best_score"] == out["best_score"]
    assert np.array_equal(t1["all_tokens"], t2["all_tokens"]) and np.array_equal(t1["all_len"], t2["all_len"])
    assert np.array_equal(t1["round_scores"], t2["round_scores"], equal_nan=True)
    wl = t2["watch_logits"]
    say(f"  run 2 (watching {watch}): {again['sec_total']:.2f}s")

    # sampling, bit for bit, at every step of every watched candidate
    for w, k in enumerate(watch):
        n = int(t1["all_len"][k])
        toks = t1["all_tokens"][k, :n]
        for step in range(n):
            assert osamp.sample(wl[w, step], c.temperature, c.sample_seed, k, step) == toks[step], (k, step)
    say(f"  sampler reproduced {sum(int(t1['all_len'][k]) for k in watch)} tokens ({time.time() - t0:.0f}s)")

    # logits and rewards of the first n_oracle watched candidates vs float64
    P = len(prompt)
    pl = [int(x) for x in prompt]
    cands = watch[:n_oracle]
    g, orm = oracle_models(name)
    bf = c.model.dtype == "bf16"
    gb, ormb = oracle_models(name, bf16_operands=True) if bf else (None, None)
    seqs, steps = [], []
    for k in cands:
        n = int(t1["all_len"][k])
        st = _audit_steps(c, rounds, n)
        steps.append(st)
        seqs.append(pl + t1["all_tokens"][k, :max(st)].tolist())
    tl = time.time()
    layer_note = lambda l: (l % 4 == 3) and say(f"    oracle layer {l + 1}/{c.model.n_layers} ({time.time() - tl:.0f}s)")
    pos = [[P - 1 + s for s in st] for st in steps]
    refs = g.logits_at(seqs, pos, progress=layer_note)
    # the oracle tensor: these candidates' logits rows at the audited steps
    scale = max(float(np.abs(ref).max()) for ref in refs)
    drift = 0.0
    if bf:
        refb = gb.logits_at(seqs, pos, progress=layer_note)
        drift = max(float(np.abs(a - b).max()) for a, b in zip(refs, refb))
    bound = max(tol(c) * scale, 2.0 * drift)
    worst = 0.0
    for k, st, ref in zip(cands, steps, refs):
        errs = [float(np.abs(wl[watch.index(k), s] - ref[j]).max()) for j, s in enumerate(st)]
        say("  candidate %d: max|err| / max|x| by step: %s" % (
            k, ", ".join(f"{s}: {e / scale:.4f}" for s, e in zip(st, errs))))
        worst = max(worst, max(errs))
    say(f"  logits: bf16-model drift D = {drift / scale:.4f} of max|x|, bound {bound / scale:.4f}")
    assert worst <= bound, (worst, scale, drift)
    say(f"  logits at {sum(len(s) for s in steps)} steps match the oracle: worst {worst / scale:.4f} of max|x| "
        f"({time.time() - t0:.0f}s)")
    got, lens, rseqs = [], [], []
    for k in cands:
        ls, gs = [], []
        for r, (L, b, K, cand, scores, acc) in enumerate(rounds):
            if k in cand and (r == 0 or rounds[r - 1][0] != L or k not in rounds[r - 1][3]):
                ls.append(L)
                gs.append(float(scores[cand.index(k)]))
        fin = float(t1["final_scores"][k])
        n = int(t1["all_len"][k])
        if not np.isnan(fin):
            ls.append(n)
            gs.append(fin)
        lens.append([P + L for L in ls])
        got.append(gs)
        rseqs.append(pl + t1["all_tokens"][k, :max(ls)].tolist())
    tl = time.time()
    # every prefix length of each candidate (one causal forward gives them
    # all); the compared entries are those the run scored
    curve = [list(range(P + 1, len(rs) + 1)) for rs in rseqs]
    ex = orm.scores_at(rseqs, curve, progress=layer_note)
    ref = np.concatenate([e[[L - P - 1 for L in ls]] for e, ls in zip(ex, lens)])
    got = np.concatenate([np.array(x) for x in got])
    drift = 0.0
    if bf:
        exb = ormb.scores_at(rseqs, curve, progress=layer_note)
        drift = max(float(np.abs(a - b).max()) for a, b in zip(ex, exb))
    scale = float(np.abs(ref).max())
    bound = max(tol(c) * scale, 2.0 * drift)
    err = float(np.abs(got - ref).max())
    say(f"  rewards {got.tolist()} vs oracle {ref.tolist()}: max|err| / max|x| = {err / scale:.4f}; "
        f"bf16-model drift over the reward curves D = {drift / scale:.4f}, bound {bound / scale:.4f}")
    assert err <= bound, (got, ref, drift)
    say(f"  {len(ref)} rewards match the oracle ({time.time() - t0:.0f}s)")
