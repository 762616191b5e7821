"""Seeded synthetic inputs for the Speculative Rejection hot path.

Both sides of every parity test (the CPU oracle and the GPU library) receive
their inputs from here: random-init model weights shaped like the paper's
workloads (Llama-3-8B-like generator and reward model, section 5) and uniform
random prompts standing in for AlpacaFarm-Eval prompts, which are not
available.  The module holds none of the method's arithmetic.

Weights of bf16 models are returned as ``uint16`` arrays of bf16 bit
patterns; fp32 models as ``float32``.  All norm gains are 1.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build() -> str:
    """Compile the generator with gcc (CPU only)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", "-o", _LIB_PATH, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        u16p = ctypes.POINTER(ctypes.c_uint16)
        f32p = ctypes.POINTER(ctypes.c_float)
        i32p = ctypes.POINTER(ctypes.c_int32)
        u32p = ctypes.POINTER(ctypes.c_uint32)
        lib.synth_normal_bf16.argtypes = [u16p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_double]
        lib.synth_normal_f32.argtypes = [f32p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_double]
        lib.synth_tokens.argtypes = [i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32]
        lib.synth_philox.argtypes = [u32p, u32p, u32p]
        _lib = lib
    return _lib


def philox(ctr, key):
    """Philox4x32-10 of the generator (used only by its known-answer test)."""
    lib = _load()
    c = (ctypes.c_uint32 * 4)(*[int(x) & 0xFFFFFFFF for x in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(x) & 0xFFFFFFFF for x in key])
    o = (ctypes.c_uint32 * 4)()
    lib.synth_philox(c, k, o)
    return tuple(int(x) for x in o)


def normal(shape, seed: int, tensor_id: int, std: float, dtype: str) -> np.ndarray:
    """Array of N(0, std) draws; element i depends only on (seed, tensor_id, i)."""
    lib = _load()
    n = int(np.prod(shape))
    if dtype == "bf16":
        out = np.empty(n, dtype=np.uint16)
        lib.synth_normal_bf16(out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16)), n, seed, tensor_id, std)
    elif dtype == "f32":
        out = np.empty(n, dtype=np.float32)
        lib.synth_normal_f32(out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), n, seed, tensor_id, std)
    else:
        raise ValueError(dtype)
    return out.reshape(shape)


def tokens(n: int, vocab: int, seed: int) -> np.ndarray:
    """n uniform random token ids in [0, vocab)."""
    lib = _load()
    out = np.empty(n, dtype=np.int32)
    lib.synth_tokens(out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n, vocab, seed)
    return out


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str  # "f32" or "bf16"
    rope_theta: float
    rms_eps: float = 1e-5

    @property
    def qkv_dim(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim


@dataclass(frozen=True)
class RunConfig:
    name: str
    model: ModelShape
    prompt_len: int
    n: int
    tau: int
    alpha: float
    max_new_tokens: int
    temperature: float = 1.0
    sample_seed: int = 42
    gen_seed: int = 0
    rm_seed: int = 1
    prompt_seed: int = 2
    eos_id: int = -1
    max_rounds: int = 0

    def with_(self, **kw) -> "RunConfig":
        return replace(self, **kw)


_TINY = ModelShape(2, 128, 4, 4, 32, 512, 512, "f32", 10000.0)
_SMALL = ModelShape(4, 512, 8, 2, 64, 1536, 8192, "bf16", 10000.0)
_ONE_B = ModelShape(16, 2048, 32, 8, 64, 8192, 32000, "bf16", 10000.0)
_EIGHT_B = ModelShape(32, 4096, 32, 8, 128, 14336, 128256, "bf16", 500000.0)

CONFIGS = {
    "tiny_fp32": RunConfig("tiny_fp32", _TINY, 32, 16, 16, 0.5, 64),
    "small_bf16": RunConfig("small_bf16", _SMALL, 128, 64, 32, 0.75, 256),
    "1b_bf16": RunConfig("1b_bf16", _ONE_B, 256, 256, 128, 0.8, 1024),
    "8b_bf16": RunConfig("8b_bf16", _EIGHT_B, 256, 512, 128, 0.8, 1024),
    "8b_bf16_n1024": RunConfig("8b_bf16_n1024", _EIGHT_B, 512, 1024, 64, 0.8, 1024),
}
# The N=1024 sweep over alpha and tau on the 8B-shaped pair.
SWEEP_8B_N1024 = [CONFIGS["8b_bf16_n1024"].with_(alpha=a, tau=t, name=f"8b_bf16_n1024_a{a}_t{t}")
                  for a in (0.5, 0.8, 0.9) for t in (64, 256)]

_TENSOR_IDS = {"embed": 1, "wqkv": 2, "wo": 3, "w13": 4, "w2": 5, "head": 6}


def weight_shapes(m: ModelShape, reward: bool) -> dict:
    """Shapes of the packed weight arrays (rows are output features)."""
    nl, d = m.n_layers, m.d_model
    return {
        "embed": (m.vocab, d),
        "attn_norm": (nl, d),
        "wqkv": (nl, m.qkv_dim, d),
        "wo": (nl, d, m.n_heads * m.head_dim),
        "ffn_norm": (nl, d),
        "w13": (nl, 2, m.ffn_dim, d),   # [gate; up]
        "w2": (nl, d, m.ffn_dim),
        "final_norm": (d,),
        "head": (d,) if reward else (m.vocab, d),
    }


def model_weights(m: ModelShape, seed: int, reward: bool, std: float = 0.02) -> dict:
    """Random-init weights: N(0, std) matrices, unit norm gains."""
    out = {}
    for name, shape in weight_shapes(m, reward).items():
        if name.endswith("norm"):
            if m.dtype == "bf16":
                out[name] = np.full(shape, 0x3F80, dtype=np.uint16)
            else:
                out[name] = np.ones(shape, dtype=np.float32)
        else:
            out[name] = normal(shape, seed, _TENSOR_IDS[name], std, m.dtype)
    return out


def prompt(cfg: RunConfig) -> np.ndarray:
    return tokens(cfg.prompt_len, cfg.model.vocab, cfg.prompt_seed)


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float32 exactly."""
    return (a.astype(np.uint32) << 16).view(np.float32)
