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


def _hd128_shape(g):
    import synth
    hkv = 2
    return synth.ModelShape(2, 128 * hkv * g if g > 1 else 256, hkv * g, hkv, 128, 512, 1000, "bf16", 500000.0)


@pytest.mark.parametrize("g", [1, 2, 4, 8])
def test_reward_and_logits_head_dim_128(g):
    """head_dim 128 paths (MFMA prefill attention, 128-wide decode) for every
    GQA group size, on small random bf16 models."""
    import synth
    from oracle.transformer import Transformer
    torch, sr = need_gpu()
    shape = _hd128_shape(g)
    say(f"hd128 g={g} shape={shape}")
    gw, rw = synth.model_weights(shape, 0, False), synth.model_weights(shape, 1, True)
    gen, rm = sr.DeviceModel.upload(shape, gw, False), sr.DeviceModel.upload(shape, rw, True)
    prompt = synth.tokens(37, shape.vocab, 5)
    rng = np.random.default_rng(g)
    rows, max_len = 5, 45
    toks = rng.integers(0, shape.vocab, size=(rows, max_len)).astype(np.int32)
    lens = np.array([45, 1, 17, 33, 44], dtype=np.int32)
    p = sr.make_params(8, 0.5, 45, 48)
    ws = sr.Workspace(gen, rm, len(prompt), p)
    got = sr.reward_scores(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda(),
                           ws).cpu().numpy()
    orm = Transformer(shape, rw, True)
    ref = np.array([orm.score(list(prompt) + list(toks[r, :lens[r]])) for r in range(rows)])
    assert np.abs(got - ref).max() <= 2e-2 * np.abs(ref).max(), (got, ref)
    lg = sr.logits_teacher_forced(gen, rm, prompt, p, torch.from_numpy(toks[:3, :20].copy()).cuda(), ws).cpu().numpy()
    og = Transformer(shape, gw, False)
    for r in range(3):
        refl = og.logits(list(prompt) + list(toks[r, :20]))[len(prompt) - 1: len(prompt) - 1 + 20]
        assert np.abs(lg[r] - refl).max() <= 2e-2 * np.abs(refl).max()


def test_teacher_forced_many_rows_head_dim_128():
    """Decode with enough rows for the 32-key streaming attention, the
    batched prefix pass and the QKV finalize fused into the attention (head
    dim 128, 4 query heads per KV head), checked on a few rows against the
    oracle."""
    import synth
    from oracle.transformer import Transformer
    torch, sr = need_gpu()
    shape = _hd128_shape(4)
    say(f"hd128 many rows shape={shape}")
    gw, rw = synth.model_weights(shape, 2, False), synth.model_weights(shape, 3, True)
    gen, rm = sr.DeviceModel.upload(shape, gw, False), sr.DeviceModel.upload(shape, rw, True)
    prompt = synth.tokens(37, shape.vocab, 6)
    rows, length = 260, 12
    toks = np.random.default_rng(7).integers(0, shape.vocab, size=(rows, length)).astype(np.int32)
    p = sr.make_params(rows, 0.5, length, length)
    ws = sr.Workspace(gen, rm, len(prompt), p)
    lg = sr.logits_teacher_forced(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), ws).cpu().numpy()
    og = Transformer(shape, gw, False)
    for r in (0, 131, rows - 1):
        refl = og.logits(list(prompt) + list(toks[r]))[len(prompt) - 1: len(prompt) - 1 + length]
        assert np.abs(lg[r] - refl).max() <= 2e-2 * np.abs(refl).max(), r


def test_8b_layer_shapes_at_run_row_counts():
    """The 8B shape's layers (d 4096, 32 query / 8 KV heads of 128, ffn
    14336, vocab 128256, RoPE theta 5e5, prompt 256) with two of them, so the
    float64 oracle stays quick, at the row counts of the 8B run's rounds:
    512 rows (256 x 256 and 256 x 128 projection tiles, 32-key streaming
    attention with the batched prefix pass, fused QKV finalize), 103 rows
    (112-row streaming tiles, 32-key streaming attention over prefix and
    tail), 21 rows (32-row streaming tiles, 64-key attention split and
    merged) and the first cut's reward-model prefill of 512 x 128 tokens
    (256 x 256 tiles).  Sampled rows against the oracle."""
    import synth
    from oracle.transformer import Transformer
    torch, sr = need_gpu()
    shape = synth.ModelShape(2, 4096, 32, 8, 128, 14336, 128256, "bf16", 500000.0)
    say(f"8B layer shapes {shape}")
    gw, rw = synth.model_weights(shape, 0, False), synth.model_weights(shape, 1, True)
    gen, rm = sr.DeviceModel.upload(shape, gw, False), sr.DeviceModel.upload(shape, rw, True)
    prompt = synth.tokens(256, shape.vocab, 5)
    rng = np.random.default_rng(8)
    length = 3
    og = Transformer(shape, gw, False)
    for rows in (512, 103, 21):
        toks = rng.integers(0, shape.vocab, size=(rows, length)).astype(np.int32)
        p = sr.make_params(rows, 0.8, length, length)
        ws = sr.Workspace(gen, rm, len(prompt), p)
        lg = sr.logits_teacher_forced(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), ws).cpu().numpy()
        for r in (0, rows // 2, rows - 1):
            refl = og.logits(list(prompt) + list(toks[r]))[len(prompt) - 1: len(prompt) - 1 + length]
            assert np.abs(lg[r] - refl).max() <= 2e-2 * np.abs(refl).max(), (rows, r)
        del ws
    # the first cut's reward-model prefill: 512 responses of 128 tokens
    # (65 536 tokens, as in the 8B run), a few rows of ragged length
    rows, rl = 512, 128
    toks = rng.integers(0, shape.vocab, size=(rows, rl)).astype(np.int32)
    lens = np.full(rows, rl, dtype=np.int32)
    lens[1], lens[rows - 2] = 77, 1
    p = sr.make_params(rows, 0.8, rl, rl)
    ws = sr.Workspace(gen, rm, len(prompt), p)
    got = sr.reward_scores(gen, rm, prompt, p, torch.from_numpy(toks).cuda(), torch.from_numpy(lens).cuda(),
                           ws).cpu().numpy()
    orm = Transformer(shape, rw, True)
    sel = [0, 1, rows - 2, rows - 1]
    ref = np.array([orm.score(list(prompt) + list(toks[r, :lens[r]])) for r in sel])
    assert np.abs(got[sel] - ref).max() <= 2e-2 * np.abs(ref).max(), (got[sel], ref)
