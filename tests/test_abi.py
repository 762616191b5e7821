"""The C interface on the CPU: every symbol the header declares is exported,
the keep count matches the paper's rule, and invalid arguments are rejected
with the documented status before any device work."""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import paper_2410_20290_amd as sr
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sr.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return sr.lib()


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "specrej.h")).read()
    return sorted(set(re.findall(r"^\s*(?:sr_status|int32_t|size_t|const char \*)\s*\*?(sr_\w+)\(", text, re.M)))


def test_header_symbols_exported(L):
    names = declared_symbols()
    assert len(names) == 20, names
    for n in names:
        assert hasattr(L, n), n


def test_keep_count_table(L):
    with open(os.path.join(ROOT, "tests", "golden", "keep_count.json")) as f:
        for b, a, k in json.load(f)["cases"]:
            assert sr.keep_count(b, a) == k
    assert sr.keep_count(10, 1.0) == -1 and sr.keep_count(10, -0.1) == -1 and sr.keep_count(-1, 0.5) == -1


def fake_model(shape, reward, dtype=None):
    cfg = sr.sr_model_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                             shape.ffn_dim, shape.vocab, shape.rope_theta, shape.rms_eps,
                             dtype if dtype is not None else (sr.SR_BF16 if shape.dtype == "bf16" else sr.SR_F32),
                             1 if reward else 0)
    w = sr.sr_weights(*([0x1000] * 9))  # never dereferenced: validation fails or sizes only
    return sr.sr_model(cfg, w)


def ws_size(L, gen, rm, P, p):
    out = ctypes.c_size_t(0)
    st = L.sr_workspace_size(ctypes.byref(gen), ctypes.byref(rm), P, ctypes.byref(p), ctypes.byref(out))
    return st, out.value


@pytest.mark.parametrize("name", list(synth.CONFIGS))
def test_workspace_size_of_every_config(L, name):
    c = synth.CONFIGS[name]
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    st, n = ws_size(L, gen, rm, c.prompt_len, sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens))
    assert st == sr.SR_OK and n > 0
    st0, n0 = ws_size(L, gen, rm, c.prompt_len, sr.make_params(c.n, 0.0, c.tau, c.max_new_tokens))
    assert st0 == sr.SR_OK
    if name.startswith("8b"):
        # the KV pools dominate: Best-of-N holds N * Lmax response tokens
        kvb = 2 * 32 * 8 * 128 * 2
        assert n0 >= c.n * c.max_new_tokens * kvb
        assert n0 < 300 * 2**30


def test_reward_cache_size():
    """The reward model's cache of the 8B-shaped pair adds two pools of the
    generator pools' slot counts (N * tau = 65536 slots each at N=512,
    tau=128, alpha=0.8) and nothing when it cannot be used."""
    c = synth.CONFIGS["8b_bf16"]
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    kvb = 2 * 32 * 8 * 128 * 2
    sizes = {}
    for rc in (0, 1):
        st, sizes[rc] = ws_size(sr.lib(), gen, rm, c.prompt_len,
                                sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens, reward_recompute=rc))
        assert st == sr.SR_OK
    assert abs(sizes[0] - sizes[1] - 2 * c.n * c.tau * kvb) <= 4096
    # Best-of-N scores once: no cache whatever the flag
    b = [ws_size(sr.lib(), gen, rm, c.prompt_len, sr.make_params(c.n, 0.0, c.tau, c.max_new_tokens,
                                                                 reward_recompute=rc))[1] for rc in (0, 1)]
    assert b[0] == b[1]
    # the log-probability reward has no reward model to cache
    b = [ws_size(sr.lib(), gen, rm, c.prompt_len, sr.make_params(c.n, c.alpha, c.tau, c.max_new_tokens,
                                                                 reward_kind=sr.SR_REWARD_LOGPROB,
                                                                 reward_recompute=rc))[1] for rc in (0, 1)]
    assert b[0] == b[1]


def plan(L, gen, rm, P, p, cap):
    out = sr.sr_params()
    st = L.sr_plan_for_memory(ctypes.byref(gen), ctypes.byref(rm), P, ctypes.byref(p), cap, ctypes.byref(out))
    return st, out


@pytest.mark.parametrize("name,alpha", [("tiny_fp32", 0.5), ("small_bf16", 0.75), ("8b_bf16", 0.8),
                                        ("8b_bf16", 0.0), ("8b_bf16_n1024", 0.5)])
def test_plan_for_memory_is_maximal(L, name, alpha):
    """Algorithm 1's memory-driven sizing: the chosen tau (n given) or n (tau
    given) is the largest whose workspace fits the capacity."""
    c = synth.CONFIGS[name]
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    p = sr.make_params(c.n, alpha, c.tau, c.max_new_tokens)
    base = ws_size(L, gen, rm, c.prompt_len, p)[1]
    for cap in (base, base + 1, base * 3 // 2, base * 4, 288 * 10**9):
        st, out = plan(L, gen, rm, c.prompt_len, p, cap)
        assert st == sr.SR_OK, sr.last_error()
        assert out.n == c.n and out.alpha == alpha and out.max_new_tokens == c.max_new_tokens
        fit = lambda tau: ws_size(L, gen, rm, c.prompt_len, sr.make_params(c.n, alpha, tau, c.max_new_tokens))[1]
        assert fit(out.tau) <= cap
        assert out.tau == c.max_new_tokens or fit(out.tau + 1) > cap
        if cap == base:
            assert out.tau >= c.tau
    # n from memory at the given tau
    q = sr.make_params(0, alpha, c.tau, c.max_new_tokens)
    for cap in (base, base * 2, 288 * 10**9):
        st, out = plan(L, gen, rm, c.prompt_len, q, cap)
        assert st == sr.SR_OK, sr.last_error()
        fitn = lambda n: ws_size(L, gen, rm, c.prompt_len, sr.make_params(n, alpha, c.tau, c.max_new_tokens))[1]
        assert out.tau == c.tau and fitn(out.n) <= cap and (out.n == 4096 or fitn(out.n + 1) > cap)
        if cap == base:
            assert out.n >= c.n
    # too little memory for anything
    st, _ = plan(L, gen, rm, c.prompt_len, p, 1 << 20)
    assert st == sr.SR_ERR_WORKSPACE_TOO_SMALL and sr.last_error()


def test_plan_for_memory_rejects_bad_input(L):
    c = synth.CONFIGS["tiny_fp32"]
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    assert plan(L, gen, rm, 32, sr.make_params(16, 1.5, 16, 64), 1 << 40)[0] == sr.SR_ERR_INVALID_ARG
    assert plan(L, gen, rm, 0, sr.make_params(16, 0.5, 16, 64), 1 << 40)[0] == sr.SR_ERR_INVALID_ARG
    assert L.sr_plan_for_memory(ctypes.byref(gen), ctypes.byref(rm), 32, None, 1 << 40, None) == \
        sr.SR_ERR_INVALID_ARG


BAD_PARAMS = [
    dict(n=0), dict(n=5000), dict(alpha=1.0), dict(alpha=-0.1), dict(alpha=float("nan")), dict(tau=0),
    dict(max_new_tokens=0), dict(temperature=-1.0), dict(temperature=float("inf")), dict(eos_id=512),
    dict(eos_id=-2), dict(max_rounds=-1), dict(reward_kind=2), dict(reward_recompute=2),
    dict(reward_recompute=-1),
]


@pytest.mark.parametrize("bad", BAD_PARAMS)
def test_invalid_params_rejected(L, bad):
    c = synth.CONFIGS["tiny_fp32"]
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    args = dict(n=16, alpha=0.5, tau=16, max_new_tokens=64, temperature=1.0)
    args.update(bad)
    st, _ = ws_size(L, gen, rm, 32, sr.make_params(**args))
    assert st == sr.SR_ERR_INVALID_ARG
    assert sr.last_error()


def test_invalid_models_rejected(L):
    c = synth.CONFIGS["small_bf16"]
    p = sr.make_params(64, 0.75, 32, 256)
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    assert ws_size(L, rm, rm, 128, p)[0] == sr.SR_ERR_INVALID_ARG          # reward model as generator
    assert ws_size(L, gen, gen, 128, p)[0] == sr.SR_ERR_INVALID_ARG        # generator as reward model
    assert ws_size(L, gen, fake_model(c.model, True, sr.SR_F32), 128, p)[0] == sr.SR_ERR_INVALID_ARG
    odd = synth.ModelShape(4, 512, 8, 2, 48, 1536, 8192, "bf16", 1e4)
    assert ws_size(L, fake_model(odd, False), fake_model(odd, True), 128, p)[0] == sr.SR_ERR_UNSUPPORTED
    odd = synth.ModelShape(4, 500, 8, 2, 64, 1536, 8192, "bf16", 1e4)
    assert ws_size(L, fake_model(odd, False), fake_model(odd, True), 128, p)[0] == sr.SR_ERR_UNSUPPORTED
    odd = synth.ModelShape(4, 512, 6, 4, 64, 1536, 8192, "bf16", 1e4)
    assert ws_size(L, fake_model(odd, False), fake_model(odd, True), 128, p)[0] == sr.SR_ERR_INVALID_ARG
    assert ws_size(L, gen, rm, 0, p)[0] == sr.SR_ERR_INVALID_ARG
    g0 = fake_model(c.model, False)
    g0.w.wqkv = None
    assert ws_size(L, g0, rm, 128, p)[0] == sr.SR_ERR_INVALID_ARG


def test_generate_rejects_before_device_work(L):
    c = synth.CONFIGS["tiny_fp32"]
    gen, rm = fake_model(c.model, False), fake_model(c.model, True)
    p = sr.make_params(16, 0.5, 16, 64)
    prompt = np.arange(32, dtype=np.int32)
    out = np.zeros(64, np.int32)
    res = sr.sr_result()
    call = lambda prm, pl, ws, nb: L.sr_generate(ctypes.byref(gen), ctypes.byref(rm), prm.ctypes.data, pl,
                                                 ctypes.byref(p), ws, nb, None, out.ctypes.data,
                                                 ctypes.byref(res), None)
    assert call(prompt, 32, 0x10000, 0) == sr.SR_ERR_WORKSPACE_TOO_SMALL
    assert "workspace" in sr.last_error()
    assert call(prompt, 32, 0x10001, 1 << 40) == sr.SR_ERR_INVALID_ARG      # misaligned
    bad = prompt.copy()
    bad[3] = 512
    assert call(bad, 32, 0x10000, 1 << 40) == sr.SR_ERR_INVALID_ARG          # token out of range
    assert call(prompt, 0, 0x10000, 1 << 40) == sr.SR_ERR_INVALID_ARG


def test_kernel_entries_reject_bad_arguments(L):
    assert L.sr_select(0x1000, 0x1000, 0, 1, 0x1000, None) == sr.SR_ERR_INVALID_ARG
    assert L.sr_select(0x1000, 0x1000, 5000, 1, 0x1000, None) == sr.SR_ERR_INVALID_ARG
    assert L.sr_select(0x1000, 0x1000, 4, 5, 0x1000, None) == sr.SR_ERR_INVALID_ARG
    assert L.sr_sample(0x1000, 2, 0, 0x1000, 0, 1.0, 1, 0x1000, None) == sr.SR_ERR_INVALID_ARG
    assert L.sr_sample(0x1000, 2, 10, 0x1000, 0, -1.0, 1, 0x1000, None) == sr.SR_ERR_INVALID_ARG
    assert L.sr_philox_fill(1, 0, 4, 0, None) == sr.SR_ERR_INVALID_ARG
    # compaction: len beyond capacity, blocks too small, overlap
    a = lambda **k: L.sr_compact(k.get("src", 0x100000), k.get("sb", 4096), k.get("dst", 0x900000), k.get("db", 4096),
                                 0x1000, k.get("b", 2), 1, 1, 64, 2, k.get("cs", 8), k.get("cd", 8), k.get("len", 4),
                                 0x2000, 0x3000, None)
    assert a(len=9) == sr.SR_ERR_INVALID_ARG
    assert a(sb=64) == sr.SR_ERR_INVALID_ARG
    assert a(dst=0x100100) == sr.SR_ERR_INVALID_ARG
    assert a(b=0) == sr.SR_ERR_INVALID_ARG
    # prefill attention: cached + new positions beyond the row capacity, shapes
    pa = lambda **k: L.sr_prefill_attention(k.get("dt", sr.SR_BF16), k.get("hd", 128), k.get("hq", 8),
                                            k.get("hkv", 2), k.get("rows", 2), k.get("lr", 4), 0x1000, 0x2000,
                                            0x3000, 16, 0x4000, 0x5000, k.get("cap", 8), k.get("t0", 4), 0x6000,
                                            None)
    assert pa(t0=5) == sr.SR_ERR_INVALID_ARG
    assert pa(t0=-1) == sr.SR_ERR_INVALID_ARG
    assert pa(hd=48) == sr.SR_ERR_UNSUPPORTED
    assert pa(hq=6, hkv=4) == sr.SR_ERR_INVALID_ARG
    assert pa(hq=6, hkv=2) == sr.SR_ERR_UNSUPPORTED
    assert pa(dt=7) == sr.SR_ERR_INVALID_ARG
    assert pa(rows=0) == sr.SR_OK and pa(lr=0) == sr.SR_OK
