"""The oracle's generator and reward model, pinned to an independent
implementation of the same architecture (HuggingFace transformers' Llama), to
torch's float64 library routines for the numerically delicate pieces, and to
invariants of causal decoding.

HF's Llama evaluates RMSNorm statistics, the attention softmax and the rotary
angles in float32 even in a float64 model, so the whole-model comparison
holds to ~1e-6 relative; 1e-5 is used, far below what any structural mistake
(wrong head mapping, RoPE pairing, eps, scale, transposed weight) produces.
RMSNorm and causal grouped-query attention are pinned exactly (1e-12) to
torch.nn.functional.rms_norm and scaled_dot_product_attention in float64."""
import numpy as np
import pytest
import torch

import synth
from oracle.transformer import Transformer, causal_attention, decode_attention, rmsnorm, rope, rope_cos_sin, widen

transformers = pytest.importorskip("transformers")


def hf_model(shape, w, reward):
    from transformers import LlamaConfig, LlamaForCausalLM, LlamaModel
    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model,
                      intermediate_size=shape.ffn_dim, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, max_position_embeddings=4096,
                      rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta,
                      tie_word_embeddings=False, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    m = (LlamaModel if reward else LlamaForCausalLM)(cfg).double().eval()
    base = m if reward else m.model
    T = lambda a: torch.from_numpy(widen(a))
    nq, nk = shape.n_heads * shape.head_dim, shape.n_kv_heads * shape.head_dim
    with torch.no_grad():
        base.embed_tokens.weight.copy_(T(w["embed"]))
        for l, layer in enumerate(base.layers):
            qkv = widen(w["wqkv"][l])
            layer.self_attn.q_proj.weight.copy_(torch.from_numpy(qkv[:nq]))
            layer.self_attn.k_proj.weight.copy_(torch.from_numpy(qkv[nq:nq + nk]))
            layer.self_attn.v_proj.weight.copy_(torch.from_numpy(qkv[nq + nk:]))
            layer.self_attn.o_proj.weight.copy_(T(w["wo"][l]))
            layer.mlp.gate_proj.weight.copy_(T(w["w13"][l][0]))
            layer.mlp.up_proj.weight.copy_(T(w["w13"][l][1]))
            layer.mlp.down_proj.weight.copy_(T(w["w2"][l]))
            layer.input_layernorm.weight.copy_(T(w["attn_norm"][l]))
            layer.post_attention_layernorm.weight.copy_(T(w["ffn_norm"][l]))
        base.norm.weight.copy_(T(w["final_norm"]))
        if not reward:
            m.lm_head.weight.copy_(T(w["head"]))
    return m


SHAPES = [
    synth.ModelShape(2, 64, 4, 2, 16, 96, 50, "f32", 10000.0),     # GQA, fp32 weights
    synth.ModelShape(2, 64, 4, 4, 16, 96, 50, "bf16", 500000.0),   # MHA, bf16 weights
    synth.ModelShape(1, 48, 6, 2, 8, 80, 33, "f32", 10000.0),      # group of 3, odd sizes
]


@pytest.mark.parametrize("shape", SHAPES)
def test_generator_logits_match_hf_llama(shape):
    w = synth.model_weights(shape, 0, False, std=0.2)
    toks = synth.tokens(23, shape.vocab, 9)
    ours = Transformer(shape, w, False).logits(toks)
    ref = hf_model(shape, w, False)(torch.from_numpy(toks.astype(np.int64))[None]).logits[0].detach().numpy()
    assert np.abs(ours - ref).max() <= 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("shape", SHAPES)
def test_reward_score_matches_hf_llama_last_state(shape):
    w = synth.model_weights(shape, 1, True, std=0.2)
    toks = synth.tokens(17, shape.vocab, 4)
    ours = Transformer(shape, w, True).score(toks)
    hs = hf_model(shape, w, True)(torch.from_numpy(toks.astype(np.int64))[None]).last_hidden_state[0].detach().numpy()
    ref = float(hs[-1] @ widen(w["head"]))
    assert abs(ours - ref) <= 1e-5 * max(1.0, abs(ref))


def test_cached_decode_equals_full_recompute():
    shape = SHAPES[0]
    g = Transformer(shape, synth.model_weights(shape, 0, False, std=0.2), False)
    prompt = synth.tokens(9, shape.vocab, 1)
    cont = [[3, 7, 1, 0], [4, 4, 2, 9], [0, 1, 2, 3]]
    st, l0 = g.start(prompt, 3, 9 + 4)
    full0 = g.logits(prompt)
    assert np.abs(l0 - full0[-1]).max() < 1e-12
    for t in range(4):
        lg = g.step(st, [c[t] for c in cont])
        for r in range(3):
            full = g.logits(list(prompt) + cont[r][:t + 1])
            assert np.abs(lg[r] - full[-1]).max() < 1e-12


def test_rows_are_independent_after_selection():
    shape = SHAPES[0]
    g = Transformer(shape, synth.model_weights(shape, 0, False, std=0.2), False)
    prompt = synth.tokens(5, shape.vocab, 2)
    st, _ = g.start(prompt, 3, 8)
    g.step(st, [1, 2, 3])
    st = g.select_rows(st, [2, 0])
    lg = g.step(st, [5, 6])
    assert np.abs(lg[0] - g.logits(list(prompt) + [3, 5])[-1]).max() < 1e-12
    assert np.abs(lg[1] - g.logits(list(prompt) + [1, 6])[-1]).max() < 1e-12


def test_rope_identity_at_zero_and_norm_preserving():
    x = np.random.default_rng(0).normal(size=(3, 16))
    c, s = rope_cos_sin(np.zeros(1), 16, 10000.0)
    assert np.array_equal(rope(x, c, s), x)
    c, s = rope_cos_sin(np.array([37.0]), 16, 10000.0)
    assert np.allclose(np.linalg.norm(rope(x, c, s), axis=-1), np.linalg.norm(x, axis=-1))


def test_rope_frequencies_match_hf_float32_table():
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding
    cfg = LlamaConfig(hidden_size=64, num_attention_heads=4, head_dim=16, rope_theta=500000.0,
                      max_position_embeddings=4096)
    emb = LlamaRotaryEmbedding(cfg)
    pos = torch.arange(0, 2000, 7)[None]
    cos, sin = emb(torch.zeros(1, dtype=torch.float32), pos)
    c, s = rope_cos_sin(pos[0].numpy(), 16, 500000.0)
    assert np.abs(cos[0, :, :8].numpy() - c).max() < 5e-4
    assert np.abs(sin[0, :, 8:].numpy() - s).max() < 5e-4


def test_rmsnorm_matches_torch_float64():
    x = np.random.default_rng(3).normal(0, 0.05, size=(7, 64))
    g = np.random.default_rng(4).normal(1, 0.1, size=64)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=1e-5).numpy()
    assert np.abs(rmsnorm(x, g, 1e-5) - ref).max() < 1e-12


@pytest.mark.parametrize("hq,hkv", [(4, 4), (4, 2), (8, 2), (6, 3), (4, 1)])
def test_causal_gqa_attention_matches_torch_sdpa(hq, hkv):
    rng = np.random.default_rng(hq * 10 + hkv)
    T, hd = 13, 16
    q, k, v = rng.normal(size=(T, hq, hd)), rng.normal(size=(T, hkv, hd)), rng.normal(size=(T, hkv, hd))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q.transpose(1, 0, 2))[None], torch.from_numpy(k.transpose(1, 0, 2))[None],
        torch.from_numpy(v.transpose(1, 0, 2))[None], is_causal=True, enable_gqa=True)[0].numpy()
    assert np.abs(causal_attention(q, k, v, hkv) - ref.transpose(1, 0, 2)).max() < 1e-12


@pytest.mark.parametrize("hq,hkv,T", [(4, 4, 1), (8, 2, 9), (32, 8, 40)])
def test_decode_attention_is_last_causal_row_and_sdpa(hq, hkv, T):
    """One new query over a cached sequence: the last row of causal
    attention, and torch's (non-causal) SDPA of that single query."""
    rng = np.random.default_rng(hq + 100 * T)
    hd = 16
    q, k, v = rng.normal(size=(T, hq, hd)), rng.normal(size=(T, hkv, hd)), rng.normal(size=(T, hkv, hd))
    got = decode_attention(q[-1], k, v, hkv)
    assert np.abs(got - causal_attention(q, k, v, hkv)[-1]).max() < 1e-12
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q[-1:].transpose(1, 0, 2))[None], torch.from_numpy(k.transpose(1, 0, 2))[None],
        torch.from_numpy(v.transpose(1, 0, 2))[None], enable_gqa=True)[0].numpy()
    assert np.abs(got - ref[:, 0, :]).max() < 1e-12


@pytest.mark.parametrize("cache", [True, False])
def test_forward_many_equals_forward_of_each(cache):
    """Sequences of different lengths through one stacked pass (weights
    widened once per layer) give each sequence's own forward; prefix scores
    from one pass equal the scores of the prefixes run on their own (the
    causal mask), and logits at chosen positions equal those rows of the
    full logits."""
    shape = SHAPES[1]
    gw, rw = synth.model_weights(shape, 0, False, std=0.2), synth.model_weights(shape, 1, True, std=0.2)
    g, r = Transformer(shape, gw, False, cache_f64=cache), Transformer(shape, rw, True, cache_f64=cache)
    seqs = [synth.tokens(n, shape.vocab, 10 + n).tolist() for n in (17, 1, 9)]
    hs = g.forward_many(seqs)
    for s, h in zip(seqs, hs):
        assert h.shape == (len(s), shape.d_model)
        assert np.abs(h - g.forward(s)).max() < 1e-12
    pos = [[0, 5, 16], [0], [8, 3]]
    for s, p, lg in zip(seqs, pos, g.logits_at(seqs, pos)):
        assert np.abs(lg - g.logits(s)[p]).max() < 1e-12
    lens = [[1, 9, 17], [1], [4, 9]]
    for s, ls, sc in zip(seqs, lens, r.scores_at(seqs, lens)):
        assert np.abs(sc - np.array([r.score(s[:L]) for L in ls])).max() < 1e-12


def test_threaded_widen_is_exact():
    rng = np.random.default_rng(11)
    a = rng.integers(0, 1 << 16, size=(5, 1 << 20), dtype=np.uint16)
    a[(a & 0x7F80) == 0x7F80] = 0   # no NaN patterns, so equality is well defined
    got = widen(a)
    ref = (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert got.shape == a.shape and np.array_equal(got, ref)
    f = rng.normal(size=(3, 1 << 21)).astype(np.float32)
    assert np.array_equal(widen(f), f.astype(np.float64))


def test_to_bf16_rounds_like_torch():
    """The bf16 rounding of the oracle's bf16-operand mode equals torch's
    float32 -> bfloat16 conversion (round to nearest even), specials included."""
    from oracle.transformer import to_bf16
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([0.0, -0.0, np.inf, -np.inf, 3.3895313892515355e38, -3.4e38, 1e-40, -1e-45])])
    x = x.astype(np.float32)
    # exact ties: low 16 bits 0x8000 with even and odd kept parts
    ties = (np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00018000], dtype=np.uint32)).view(np.float32)
    x = np.concatenate([x, ties])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = to_bf16(x)
    assert np.array_equal(got, ref) and np.array_equal(np.signbit(got), np.signbit(ref))
    assert np.isnan(to_bf16(np.array([np.nan]))[0])
    # float64 input is held as float32 first
    y = rng.standard_normal(1000)
    assert np.array_equal(to_bf16(y), torch.from_numpy(y).float().to(torch.bfloat16).double().numpy())


def test_bf16_operands_drift_is_bf16_sized_and_like_hf_autocast():
    """The bf16-operand mode is a bf16 model: on a 4-layer model its logits
    leave the exact model's by a bf16-sized amount (not zero, well below 5 %),
    of the same size as HF Llama's under torch's bf16 autocast (an independent
    bf16 evaluation, within a factor of 3)."""
    shape = synth.ModelShape(4, 256, 8, 2, 32, 512, 500, "bf16", 10000.0)
    w = synth.model_weights(shape, 0, False, std=0.05)
    toks = synth.tokens(96, shape.vocab, 3)
    ex = Transformer(shape, w, False).logits(toks)
    bm = Transformer(shape, w, False, bf16_operands=True).logits(toks)
    m = hf_model(shape, w, False).float()
    with torch.no_grad(), torch.autocast("cpu", dtype=torch.bfloat16):
        hf = m(torch.from_numpy(np.asarray(toks, dtype=np.int64))[None]).logits[0].float().numpy()
    sc = np.abs(ex).max()
    ours, theirs = np.abs(bm - ex).max() / sc, np.abs(hf - ex).max() / sc
    assert 2.0 ** -12 < ours < 5e-2, ours
    assert 1 / 3 < ours / theirs < 3, (ours, theirs)
    # scores too, through the same mode
    rw = synth.model_weights(shape, 1, True, std=0.05)
    se = Transformer(shape, rw, True).scores_at([toks], [[10, 50, 96]])[0]
    sb = Transformer(shape, rw, True, bf16_operands=True).scores_at([toks], [[10, 50, 96]])[0]
    assert 0 < np.abs(sb - se).max() < 5e-2 * np.abs(se).max()
