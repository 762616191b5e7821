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


@functools.lru_cache(maxsize=4)
def host_models(name):
    import synth
    c = synth.CONFIGS[name]
    return (c, synth.model_weights(c.model, c.gen_seed, False), synth.model_weights(c.model, c.rm_seed, True),
            synth.prompt(c))


_dev = {}


def device_models(name):
    """(config, gen, rm, prompt) with weights uploaded once per process."""
    torch, sr = need_gpu()
    if name not in _dev:
        if len(_dev) >= 2:          # keep at most two configurations resident
            _dev.pop(next(iter(_dev)))
            torch.cuda.empty_cache()
        c, gw, rw, pr = host_models(name)
        _dev[name] = (c, sr.DeviceModel.upload(c.model, gw, False), sr.DeviceModel.upload(c.model, rw, True), pr)
    return _dev[name]


def oracle_models(name):
    from oracle.transformer import Transformer
    c, gw, rw, pr = host_models(name)
    return Transformer(c.model, gw, False), Transformer(c.model, rw, True)


def tol(cfg):
    """Max-abs tolerance factor relative to max|x| of the oracle tensor."""
    return 1e-4 if cfg.model.dtype == "f32" else 2e-2
