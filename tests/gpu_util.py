"""Shared helpers of the GPU parity tests."""
import functools
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2410_20290_amd as sr
    if not os.path.exists(sr.LIB_PATH):
        pytest.fail("libspecrej.so is not built (run __graft_entry__.build())")
    return torch, sr


def say(*a):
    print(*a, flush=True)


@functools.lru_cache(maxsize=2)
def host_weights(model, gen_seed, rm_seed):
    """Generator and reward-model weights of one shape (shared by every
    configuration of that shape and seeds)."""
    import synth
    return synth.model_weights(model, gen_seed, False), synth.model_weights(model, rm_seed, True)


def host_models(name):
    import synth
    c = synth.CONFIGS[name]
    gw, rw = host_weights(c.model, c.gen_seed, c.rm_seed)
    return c, gw, rw, synth.prompt(c)


_dev = {}


def device_models(name):
    """(config, gen, rm, prompt) with each shape's weights uploaded once per
    process (at most two shapes resident)."""
    torch, sr = need_gpu()
    c, gw, rw, pr = host_models(name)
    key = (c.model, c.gen_seed, c.rm_seed)
    if key not in _dev:
        if len(_dev) >= 2:
            _dev.pop(next(iter(_dev)))
            torch.cuda.empty_cache()
        _dev[key] = (sr.DeviceModel.upload(c.model, gw, False), sr.DeviceModel.upload(c.model, rw, True))
    return (c,) + _dev[key] + (pr,)


def oracle_models(name, bf16_operands=False):
    from oracle.transformer import Transformer
    c, gw, rw, pr = host_models(name)
    return (Transformer(c.model, gw, False, bf16_operands=bf16_operands),
            Transformer(c.model, rw, True, bf16_operands=bf16_operands))


def tol(cfg):
    """Max-abs tolerance factor relative to max|x| of the oracle tensor."""
    return 1e-4 if cfg.model.dtype == "f32" else 2e-2


def trace_rounds(out):
    """(L, b, K, candidates, scores, accept flags) of every cut of a traced run."""
    t = out["trace"]
    rounds = []
    for r in range(t["rounds"]):
        b = int(t["round_b"][r])
        cand = t["round_cand"][r, :b].tolist()
        rounds.append((int(t["round_L"][r]), b, int(t["round_keep"][r]), cand,
                       t["round_scores"][r, :b].copy(), t["round_accept"][r, :b].copy()))
    return rounds


def check_trace_logic(c, out):
    """What must hold of any run, whatever the model numerics, bit for bit:
    the keep count of every cut, the survivors = the oracle's top K on the
    GPU's own scores (eqs. cutoff-threshold and accepted-set), the answer =
    the oracle's arg max over the GPU's final rewards of I (eq. output), and
    the token accounting."""
    from oracle import specrej
    t = out["trace"]
    rounds = trace_rounds(out)
    for (L, b, K, cand, scores, acc) in rounds:
        assert K == specrej.keep_count(b, c.alpha)
        assert cand == sorted(cand)
        sd = {k: float(s) for k, s in zip(cand, scores)}
        kept = set(specrej.top_k(cand, sd, K))
        assert [int(a) for a in acc] == [1 if k in kept else 0 for k in cand]
    fs = t["final_scores"]
    members = {k: float(fs[k]) for k in range(c.n) if not np.isnan(fs[k])}
    assert out["best_index"] == specrej.arg_best(members)
    assert out["best_score"] == np.float32(members[out["best_index"]])
    lens = t["all_len"]
    assert out["generated_tokens"] == int(lens.sum())
    assert out["tokens"] == t["all_tokens"][out["best_index"], : lens[out["best_index"]]].tolist()
    return rounds
