"""Best-of-N and Speculative Rejection, step by step as the paper states them.

Best-of-N (section 3): draw N i.i.d. responses y_k ~ p(. | x), score each
with s, return the arg max.

Speculative Rejection (section 4.2, Algorithm 1): run Best-of-N with a large
initial batch; each time memory fills up (the decision token), score every
partial response with s (eq. partial-reward-set), compute the cutoff as the
alpha lower quantile of those scores (eq. cutoff-threshold), keep the
candidates at or above it (eq. accepted-set), move the completed ones into
the set I, and continue the accepted unfinished ones; return the arg max of
s over I (eq. output).

Readings where the paper is silent or loose (each is listed in the design
notes of the repository):

* Keep count.  "Top (1 - alpha) proportion" with ties broken by candidate id:
  K = ceil((1 - alpha) b), computed in integers as
  b - floor(alpha_ppm * b / 10^6) with alpha_ppm = round(alpha * 10^6).
  K >= 1 whenever alpha < 1, so the accepted set is never empty.
* Total order.  Score descending, then candidate id ascending; NaN ranks
  below every number.  Used for the cut and for the final arg max.
* Decision tokens.  Memory holds B = N * tau response-token slots.  A round
  with b unfinished candidates at length L runs to
  D = min(Lmax, floor(B / b)); the first round therefore stops at tau.  If
  floor(B / b) <= L after a cut (memory still full), another cut follows at
  once on the same scores.  A round in which no candidate could be rejected
  (K = b), or past ``max_rounds`` cuts, runs to Lmax without calling s.
  With alpha = 0 this is exactly Best-of-N.
* Completed rows (EOS) are scored and ranked with the rest at a cut, join I
  whether accepted or not, and stop generating.  Rows still unfinished at
  Lmax are final as they are.  When every candidate of a round is complete,
  or D = Lmax, all are scored and join I.
* tau and L count response tokens only; the EOS token belongs to the
  response (section 3) and is scored.
"""
import math

import numpy as np

from .sampler import sample

PPM = 1_000_000


def alpha_ppm(alpha: float) -> int:
    return int(math.floor(alpha * PPM + 0.5))


def keep_count(b: int, alpha: float) -> int:
    """K = ceil((1 - alpha) * b), exactly, via the integer rule above."""
    return b - (alpha_ppm(alpha) * b) // PPM


def rank_key(score: float, cand: int):
    """Sort key: best first (score descending, NaN last, then id ascending)."""
    if score != score:  # NaN
        return (1, 0.0, cand)
    return (0, -score, cand)


def top_k(cands, scores: dict, k: int):
    """The first k candidates in the total order (eq. accepted-set)."""
    order = sorted(cands, key=lambda c: rank_key(scores[c], c))
    return order[:k]


def arg_best(scores: dict) -> int:
    """arg max over a dict cand -> score in the total order (eq. output)."""
    return top_k(list(scores), scores, 1)[0]


def mean_logprob(gen, prompt, tokens) -> float:
    """The probability-as-reward score of section 5.3:
    s(y) = (1 / len(y)) ln p(y | x), with p the generator's own softmax
    (temperature 1) and ln p(y | x) the sum over the response tokens of
    ln p(y_t | x, y_<t).  Computed in float64 from one forward pass over
    x + y: row P - 1 + t of the logits gives the distribution of y_t."""
    P, n = len(prompt), len(tokens)
    if n == 0:
        return 0.0
    lg = gen.logits(list(prompt) + list(tokens))[P - 1:P - 1 + n]
    m = lg.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(lg - m).sum(axis=1))
    return float(np.mean(lg[np.arange(n), list(tokens)] - lse))


def _f32(x) -> float:
    return float(np.float32(x))


class Result(dict):
    """best, score, tokens (of best), responses {cand: tokens}, final {cand: score},
    rounds [(L, b, K, accepted, scores)], generated, decisions [D per round]."""


def speculative_rejection(gen, rm, prompt, n, alpha, tau, max_new, temperature,
                          seed, eos_id=-1, max_rounds=0, score_fn=None):
    """Algorithm 1 (section 4.2) under the readings in the module docstring.

    ``score_fn(prompt, tokens) -> float`` overrides the reward model (used for
    the probability-as-reward variant of section 5.3); by default it is
    rm.score(prompt + tokens).  Scores are rounded to float32 before ranking,
    the precision in which the GPU ranks them.
    """
    prompt = [int(t) for t in prompt]
    P = len(prompt)
    Lmax = max_new
    B = n * tau
    if score_fn is None:
        score_fn = lambda pr, toks: rm.score(pr + toks)

    def decision(b, L, r):
        if keep_count(b, alpha) == b or (max_rounds > 0 and r >= max_rounds):
            return Lmax
        return min(Lmax, B // b)

    state, l0 = gen.start(prompt, n, P + Lmax)
    A = list(range(n))           # candidates of the current round (ascending)
    G = list(range(n))           # rows still generating (= A minus completed)
    logits = np.repeat(l0[None], n, axis=0)
    fresh = True
    toks = {k: [] for k in A}
    done = {k: False for k in A}
    I = {}
    rounds, decisions = [], []
    generated = 0
    r, L = 0, 0
    D = decision(n, 0, 0)
    decisions.append(D)
    while True:
        # Phase 1: early generation up to the decision token.
        while L < D and G:
            if not fresh:
                logits = gen.step(state, [toks[k][-1] for k in G])
            for i, k in enumerate(G):
                t = sample(np.float32(logits[i]), temperature, seed, k, L)
                toks[k].append(t)
                if t == eos_id:
                    done[k] = True
            generated += len(G)
            L += 1
            keep = [i for i, k in enumerate(G) if not done[k]]
            G = [G[i] for i in keep]
            state = gen.select_rows(state, keep)
            fresh = False
        # Every candidate complete: score all, they join I.
        if D == Lmax or not G:
            for k in A:
                I[k] = _f32(score_fn(prompt, toks[k]))
            break
        # Phase 2: partial rewards and the cut.
        b = len(A)
        K = keep_count(b, alpha)
        scores = {k: _f32(score_fn(prompt, toks[k])) for k in A}
        acc = top_k(A, scores, K)
        for k in A:
            if done[k]:
                I[k] = scores[k]
        rounds.append((L, b, K, list(acc), dict(scores)))
        A = sorted(k for k in acc if not done[k])
        r += 1
        # Phase 3: batch for the next round (another cut if memory is still full).
        while A:
            if keep_count(len(A), alpha) == len(A) or (max_rounds > 0 and r >= max_rounds):
                D = Lmax
                break
            Dn = min(Lmax, B // len(A))
            if Dn > L:
                D = Dn
                break
            b2 = len(A)
            K2 = keep_count(b2, alpha)
            acc2 = top_k(A, scores, K2)
            rounds.append((L, b2, K2, list(acc2), {k: scores[k] for k in A}))
            A = sorted(acc2)
            r += 1
        if not A:
            break
        decisions.append(D)
        aset = set(A)
        keep = [i for i, k in enumerate(G) if k in aset]
        G = [G[i] for i in keep]
        state = gen.select_rows(state, keep)
    best = arg_best(I)
    return Result(best=best, score=I[best], tokens=list(toks[best]), responses=toks,
                  final=I, rounds=rounds, generated=generated, decisions=decisions)


def best_of_n(gen, rm, prompt, n, max_new, temperature, seed, eos_id=-1, score_fn=None):
    """Best-of-N (section 3): N full responses, each scored, arg max returned."""
    prompt = [int(t) for t in prompt]
    P = len(prompt)
    if score_fn is None:
        score_fn = lambda pr, toks: rm.score(pr + toks)
    state, l0 = gen.start(prompt, n, P + max_new)
    rows = list(range(n))
    logits = np.repeat(l0[None], n, axis=0)
    toks = {k: [] for k in rows}
    generated = 0
    for L in range(max_new):
        if not rows:
            break
        if L > 0:
            logits = gen.step(state, [toks[k][-1] for k in rows])
        for i, k in enumerate(rows):
            toks[k].append(sample(np.float32(logits[i]), temperature, seed, k, L))
        generated += len(rows)
        keep = [i for i, k in enumerate(rows) if toks[k][-1] != eos_id]
        rows = [rows[i] for i in keep]
        state = gen.select_rows(state, keep)
    final = {k: _f32(score_fn(prompt, toks[k])) for k in range(n)}
    best = arg_best(final)
    return Result(best=best, score=final[best], tokens=list(toks[best]), responses=toks,
                  final=final, rounds=[], generated=generated, decisions=[max_new])


def schedule(n, alpha, tau, max_new, max_rounds=0):
    """Rounds (L, b, K) and generated tokens when no candidate emits EOS."""
    B = n * tau
    Lmax = max_new
    rounds = []
    b, L, r, total = n, 0, 0, 0

    def decision(b, r):
        if keep_count(b, alpha) == b or (max_rounds > 0 and r >= max_rounds):
            return Lmax
        return min(Lmax, B // b)

    D = decision(b, r)
    while True:
        total += b * (D - L)
        L = D
        if D == Lmax:
            break
        K = keep_count(b, alpha)
        rounds.append((L, b, K))
        b = K
        r += 1
        while True:
            if keep_count(b, alpha) == b or (max_rounds > 0 and r >= max_rounds):
                D = Lmax
                break
            Dn = min(Lmax, B // b)
            if Dn > L:
                D = Dn
                break
            K = keep_count(b, alpha)
            rounds.append((L, b, K))
            b = K
            r += 1
    return rounds, total
