"""Model-level parity: teacher-forced generator logits through the decode
path and reward-model scores, against the oracle's float64 transformer,
within 1e-4 max|x| (fp32 model) or 2e-2 max|x| (bf16 model)."""
import numpy as np
import pytest

from gpu_util import device_models, need_gpu, oracle_models, say, tol

pytestmark = pytest.mark.gpu


def run_tf(name, rows, length, seed):
    torch, sr = need_gpu()
    c, gen, rm, prompt = device_models(name)
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, c.model.vocab, size=(rows, length)).astype(np.int32)
    p = sr.make_params(max(rows, c.n), c.alpha, max(c.tau, length), max(length, c.max_new_tokens))
    ws = sr.Workspace(gen, rm, len(prompt), p)
    out = sr.logits_teacher_forced(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), ws).cpu().numpy()
    return c, prompt, toks, out


@pytest.mark.parametrize("name,rows,length", [("tiny_fp32", 5, 24), ("small_bf16", 3, 40)])
def test_teacher_forced_logits(name, rows, length):
    say(f"teacher-forced {name} rows={rows} len={length}")
    c, prompt, toks, got = run_tf(name, rows, length, 1)
    g, _ = oracle_models(name)
    for r in range(rows):
        ref = g.logits(list(prompt) + list(toks[r]))[len(prompt) - 1: len(prompt) - 1 + length]
        err = np.abs(got[r] - ref).max()
        assert err <= tol(c) * np.abs(ref).max(), (r, err, np.abs(ref).max())


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16"])
def test_reward_scores(name):
    torch, sr = need_gpu()
    say(f"reward scores {name}")
    c, gen, rm, prompt = device_models(name)
    rng = np.random.default_rng(3)
    rows, max_len = 9, 37
    toks = rng.integers(0, c.model.vocab, size=(rows, max_len)).astype(np.int32)
    lens = np.array([1, 2, 37, 36, 16, 17, 5, 30, 33], dtype=np.int32)
    p = sr.make_params(max(rows, c.n), c.alpha, c.tau, max(max_len, c.max_new_tokens))
    ws = sr.Workspace(gen, rm, len(prompt), p)
    got = sr.reward_scores(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda(),
                           ws).cpu().numpy()
    _, orm = oracle_models(name)
    ref = np.array([orm.score(list(prompt) + list(toks[r, :lens[r]])) for r in range(rows)])
    assert np.abs(got - ref).max() <= tol(c) * np.abs(ref).max(), (got, ref)
