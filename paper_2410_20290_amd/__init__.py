"""Python binding of libspecrej (Speculative Rejection on MI355X / gfx950).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  torch provides device memory and streams.  The names follow the
C interface in include/specrej.h.  Importing this module does not need a GPU;
calling anything that launches work does, and fails loudly if the library is
not built.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspecrej.so")

SR_OK, SR_ERR_INVALID_ARG, SR_ERR_WORKSPACE_TOO_SMALL, SR_ERR_UNSUPPORTED, SR_ERR_DEVICE, SR_ERR_INTERNAL = range(6)
SR_F32, SR_BF16 = 0, 1

_i32, _i64, _u64, _f32, _f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float, ctypes.c_double
_vp = ctypes.c_void_p


class sr_model_config(ctypes.Structure):
    _fields_ = [("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32), ("n_kv_heads", _i32),
                ("head_dim", _i32), ("ffn_dim", _i32), ("vocab", _i32), ("rope_theta", _f32),
                ("rms_eps", _f32), ("dtype", _i32), ("is_reward", _i32)]


class sr_weights(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ("embed", "attn_norm", "wqkv", "wo", "ffn_norm", "w13", "w2",
                                   "final_norm", "head")]


class sr_model(ctypes.Structure):
    _fields_ = [("cfg", sr_model_config), ("w", sr_weights)]


NCLASS = 8
KERNEL_CLASSES = ["gen_gemm_mfma", "gen_gemm_hbm", "decode_attn", "rm_gemm", "prefill_attn", "sample", "cut",
                  "other"]


class sr_params(ctypes.Structure):
    _fields_ = [("n", _i32), ("alpha", _f64), ("tau", _i32), ("max_new_tokens", _i32),
                ("temperature", _f32), ("seed", _u64), ("eos_id", _i32), ("max_rounds", _i32),
                ("profile_every", _i32), ("reward_kind", _i32), ("reward_recompute", _i32)]


class sr_result(ctypes.Structure):
    _fields_ = [("best_index", _i32), ("best_score", _f32), ("n_tokens", _i32), ("rounds", _i32),
                ("generated_tokens", _i64), ("sec_total", _f64), ("sec_prefill", _f64),
                ("sec_decode", _f64), ("sec_reward", _f64), ("sec_cut", _f64),
                ("kernel_sec", _f64 * NCLASS), ("kernel_launches", _i64 * NCLASS),
                ("kernel_bytes", _f64 * NCLASS), ("kernel_flops", _f64 * NCLASS)]


class sr_trace(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ("round_L", "round_b", "round_keep", "round_cand", "round_scores",
                                   "round_accept", "all_tokens", "all_len", "final_scores")] + \
               [("max_rounds_cap", _i32), ("watch_cand", _vp), ("n_watch", _i32), ("watch_logits", _vp)]


_lib = None


class SpecRejError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"specrej status {status}: {msg}")
        self.status = status


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.sr_last_error.restype = ctypes.c_char_p
        L.sr_keep_count.argtypes = [_i32, _f64]
        L.sr_keep_count.restype = _i32
        L.sr_workspace_size.argtypes = [P(sr_model), P(sr_model), _i32, P(sr_params), P(ctypes.c_size_t)]
        L.sr_plan_for_memory.argtypes = [P(sr_model), P(sr_model), _i32, P(sr_params), ctypes.c_size_t,
                                         P(sr_params)]
        L.sr_generate.argtypes = [P(sr_model), P(sr_model), _vp, _i32, P(sr_params), _vp, ctypes.c_size_t,
                                  _vp, _vp, P(sr_result), P(sr_trace)]
        L.sr_philox_fill.argtypes = [_u64, _vp, _i32, _vp, _vp]
        L.sr_sample.argtypes = [_vp, _i32, _i32, _vp, _i32, _f32, _u64, _vp, _vp]
        L.sr_select.argtypes = [_vp, _vp, _i32, _i32, _vp, _vp]
        L.sr_compact.argtypes = [_vp, _i64, _vp, _i64, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32,
                                 _vp, _vp, _vp]
        L.sr_logits_teacher_forced.argtypes = [P(sr_model), P(sr_model), _vp, _i32, P(sr_params), _vp, _i32,
                                               _i32, _vp, _vp, ctypes.c_size_t, _vp]
        L.sr_reward_scores.argtypes = [P(sr_model), P(sr_model), _vp, _i32, P(sr_params), _vp, _vp, _i32,
                                       _i32, _vp, _vp, ctypes.c_size_t, _vp]
        L.sr_projection.argtypes = [_i32, _vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp, ctypes.c_size_t, _vp]
        L.sr_projection_scratch.argtypes = [_i32, _i32, _i32, _i32, _i32]
        L.sr_projection_scratch.restype = ctypes.c_size_t
        L.sr_decode_attention.argtypes = [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _i32, _i32,
                                          _vp, _vp, ctypes.c_size_t, _vp]
        L.sr_decode_attention_scratch.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32]
        L.sr_decode_attention_scratch.restype = ctypes.c_size_t
        L.sr_decode_attention_noalloc.argtypes = [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _i32,
                                                  _i32, _vp, _vp]
        L.sr_decode_attention_noalloc_limit.argtypes = []
        L.sr_decode_attention_noalloc_limit.restype = ctypes.c_size_t
        L.sr_prefill_attention.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _i32,
                                           _i32, _vp, _vp]
        L.sr_correlation.argtypes = [_vp, _vp, _i32, P(ctypes.c_double), P(ctypes.c_double)]
        L.sr_improvement_score.argtypes = [_vp, _i32, _f32, P(ctypes.c_double)]
        for f in ("sr_projection", "sr_decode_attention", "sr_decode_attention_noalloc", "sr_prefill_attention", "sr_plan_for_memory",
                  "sr_correlation", "sr_improvement_score", "sr_workspace_size", "sr_generate", "sr_philox_fill", "sr_sample", "sr_select", "sr_compact",
                  "sr_logits_teacher_forced", "sr_reward_scores"):
            getattr(L, f).restype = _i32
        _lib = L
    return _lib


def _mref(m):
    """Pointer to a model descriptor, or NULL for None (a reward model is not
    needed when the reward is the generator's own log-probability)."""
    return None if m is None else ctypes.byref(m.desc)


def last_error() -> str:
    return lib().sr_last_error().decode()


def _check(status):
    if status != SR_OK:
        raise SpecRejError(status, last_error())


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream=None) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def keep_count(b: int, alpha: float) -> int:
    return int(lib().sr_keep_count(b, alpha))


# ---------------------------------------------------------------- models
@dataclass
class DeviceModel:
    """Weights of one model on the device plus its C descriptor."""
    shape: object           # synth.ModelShape-like (fields of sr_model_config)
    reward: bool
    tensors: dict           # name -> torch tensor on the device
    desc: sr_model

    @staticmethod
    def upload(shape, weights: dict, reward: bool, device="cuda") -> "DeviceModel":
        import torch
        ts = {}
        for name, a in weights.items():
            a = np.ascontiguousarray(a)
            if a.dtype == np.uint16:
                t = torch.from_numpy(a.view(np.int16)).to(device)
            else:
                t = torch.from_numpy(a.astype(np.float32, copy=False)).to(device)
            ts[name] = t
        cfg = sr_model_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                              shape.ffn_dim, shape.vocab, shape.rope_theta, shape.rms_eps,
                              SR_BF16 if shape.dtype == "bf16" else SR_F32, 1 if reward else 0)
        w = sr_weights(*[_ptr(ts[n]) for n in ("embed", "attn_norm", "wqkv", "wo", "ffn_norm", "w13", "w2",
                                               "final_norm", "head")])
        return DeviceModel(shape, reward, ts, sr_model(cfg, w))


SR_REWARD_MODEL, SR_REWARD_LOGPROB = 0, 1


def make_params(n, alpha, tau, max_new_tokens, temperature=1.0, seed=42, eos_id=-1, max_rounds=0,
                profile_every=0, reward_kind=SR_REWARD_MODEL, reward_recompute=0) -> sr_params:
    return sr_params(n, alpha, tau, max_new_tokens, temperature, seed, eos_id, max_rounds, profile_every,
                     reward_kind, reward_recompute)


def workspace_size(gen: DeviceModel, rm: DeviceModel, prompt_len: int, p: sr_params) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().sr_workspace_size(ctypes.byref(gen.desc), _mref(rm), prompt_len, ctypes.byref(p),
                                   ctypes.byref(out)))
    return int(out.value)


def plan_for_memory(gen: DeviceModel, rm: DeviceModel, prompt_len: int, p: sr_params, capacity_bytes: int) -> sr_params:
    """sr_plan_for_memory: p with the largest tau (p.n >= 1) or n (p.n == 0)
    whose workspace fits in capacity_bytes."""
    out = sr_params()
    _check(lib().sr_plan_for_memory(ctypes.byref(gen.desc), _mref(rm), prompt_len, ctypes.byref(p),
                                    int(capacity_bytes), ctypes.byref(out)))
    return out


def correlation(x, y):
    """sr_correlation: (Pearson, Kendall) of the paired host arrays x, y."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    y = np.ascontiguousarray(np.asarray(y, dtype=np.float32))
    if x.shape != y.shape or x.ndim != 1:
        raise ValueError("x and y must be 1-D arrays of one length")
    pr, kd = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(lib().sr_correlation(x.ctypes.data, y.ctypes.data, len(x), ctypes.byref(pr), ctypes.byref(kd)))
    return pr.value, kd.value


def improvement_score(bon_rewards, sr_reward: float) -> float:
    """sr_improvement_score over the Best-of-N rewards (host array)."""
    z = np.ascontiguousarray(np.asarray(bon_rewards, dtype=np.float32))
    out = ctypes.c_double(0.0)
    _check(lib().sr_improvement_score(z.ctypes.data, len(z), float(sr_reward), ctypes.byref(out)))
    return out.value


def alloc_workspace(nbytes: int, device="cuda"):
    import torch
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws, ws.data_ptr() + off, nbytes


class Workspace:
    """A device buffer sized for (gen, rm, prompt_len, params)."""

    def __init__(self, gen, rm, prompt_len, p, device="cuda"):
        self.nbytes = workspace_size(gen, rm, prompt_len, p)
        self.tensor, self.ptr, _ = alloc_workspace(self.nbytes, device)


def generate(gen: DeviceModel, rm: DeviceModel, prompt, p: sr_params, ws: Workspace = None, trace=False,
             max_rounds_cap=64, stream=None, watch=()) -> dict:
    """sr_generate; returns the answer, result summary and (optionally) the
    trace.  ``watch``: candidates whose sampled-from logits rows the trace
    records (out["trace"]["watch_logits"] [len(watch)][max_new_tokens][vocab];
    implies trace=True)."""
    prompt = np.ascontiguousarray(np.asarray(prompt, dtype=np.int32))
    if ws is None:
        ws = Workspace(gen, rm, len(prompt), p)
    out_tokens = np.zeros(max(1, p.max_new_tokens), dtype=np.int32)
    res = sr_result()
    tr = None
    arrays = {}
    watch = np.ascontiguousarray(np.asarray(list(watch), dtype=np.int32))
    trace = trace or len(watch) > 0
    if trace:
        n, R = p.n, max_rounds_cap
        arrays = dict(round_L=np.zeros(R, np.int32), round_b=np.zeros(R, np.int32),
                      round_keep=np.zeros(R, np.int32), round_cand=np.zeros((R, n), np.int32),
                      round_scores=np.zeros((R, n), np.float32), round_accept=np.zeros((R, n), np.int32),
                      all_tokens=np.zeros((n, p.max_new_tokens), np.int32), all_len=np.zeros(n, np.int32),
                      final_scores=np.zeros(n, np.float32))
        tr = sr_trace(*[a.ctypes.data for a in arrays.values()], R)
        if len(watch):
            wl = np.full((len(watch), p.max_new_tokens, gen.shape.vocab), np.nan, dtype=np.float32)
            arrays["watch_logits"] = wl
            tr.watch_cand, tr.n_watch, tr.watch_logits = watch.ctypes.data, len(watch), wl.ctypes.data
    st = lib().sr_generate(ctypes.byref(gen.desc), _mref(rm), prompt.ctypes.data, len(prompt),
                           ctypes.byref(p), ws.ptr, ws.nbytes, _stream(stream), out_tokens.ctypes.data,
                           ctypes.byref(res), ctypes.byref(tr) if tr is not None else None)
    _check(st)
    out = {f: getattr(res, f) for f, _ in sr_result._fields_ if not f.startswith("kernel_")}
    out["kernels"] = {name: {"sec": res.kernel_sec[i], "launches": int(res.kernel_launches[i]),
                             "bytes": res.kernel_bytes[i], "flops": res.kernel_flops[i]}
                      for i, name in enumerate(KERNEL_CLASSES)}
    out["tokens"] = out_tokens[:res.n_tokens].tolist()
    if trace:
        R = res.rounds
        out["trace"] = {k: v for k, v in arrays.items()}
        out["trace"]["rounds"] = R
    return out


# ------------------------------------------------- kernel-level entry points
def philox_fill(seed: int, ctr, out, stream=None):
    _check(lib().sr_philox_fill(seed, _ptr(ctr), ctr.shape[0], _ptr(out), _stream(stream)))


def sample(logits, cand, step: int, temperature: float, seed: int, tokens, stream=None):
    rows, vocab = logits.shape
    _check(lib().sr_sample(_ptr(logits), rows, vocab, _ptr(cand), step, temperature, seed, _ptr(tokens),
                           _stream(stream)))


def select(scores, cand, keep: int, accept, stream=None):
    _check(lib().sr_select(_ptr(scores), _ptr(cand), scores.shape[0], keep, _ptr(accept), _stream(stream)))


def compact(src, src_block, dst, dst_block, keep_flag, n_layers, n_kv_heads, head_dim, elem_bytes, cap_src,
            cap_dst, length, src_row, new_count, stream=None):
    _check(lib().sr_compact(_ptr(src), src_block, _ptr(dst), dst_block, _ptr(keep_flag), keep_flag.shape[0],
                            n_layers, n_kv_heads, head_dim, elem_bytes, cap_src, cap_dst, length, _ptr(src_row),
                            _ptr(new_count), _stream(stream)))


def projection(x, w, mode: int, out, stream=None):
    """sr_projection: x [M][K], w [N][K] (mode 2: [2][N][K]), see the header."""
    import torch
    dtype = SR_BF16 if x.dtype in (torch.int16, torch.bfloat16) else SR_F32
    M, K = x.shape
    N = w.shape[-2]
    need = int(lib().sr_projection_scratch(dtype, M, N, K, mode))
    part = torch.empty(max(need, 1), dtype=torch.float32, device=x.device)
    _check(lib().sr_projection(dtype, _ptr(x), _ptr(w), M, N, K, mode, _ptr(out), _ptr(part), need,
                               _stream(stream)))
    return part


def decode_attention(q, kpre, vpre, ktail, vtail, lt: int, out, stream=None):
    """sr_decode_attention: q float [rows][hq][hd]; kpre/vpre [hkv][P][hd]
    (or None when P = 0); ktail/vtail [rows][hkv][cap][hd]; out [rows][hq*hd]
    in the model dtype (bf16 tensors travel as int16).  See the header."""
    import torch
    rows, hq, hd = q.shape
    hkv, cap = ktail.shape[1], ktail.shape[2]
    P = 0 if kpre is None else kpre.shape[1]
    dtype = SR_BF16 if ktail.dtype in (torch.int16, torch.bfloat16) else SR_F32
    need = int(lib().sr_decode_attention_scratch(hd, hq, hkv, rows, P, lt))
    part = torch.empty(max(need, 1), dtype=torch.float32, device=q.device)
    _check(lib().sr_decode_attention(dtype, hd, hq, hkv, rows, _ptr(q), _ptr(kpre), _ptr(vpre), P, _ptr(ktail),
                                     _ptr(vtail), cap, lt, _ptr(out), _ptr(part), need, _stream(stream)))
    return part


def decode_attention_noalloc(q, kpre, vpre, ktail, vtail, lt: int, out, stream=None):
    """sr_decode_attention_noalloc: as decode_attention, with the split
    partials in the library's static device scratch (no buffer allocated)."""
    import torch
    rows, hq, hd = q.shape
    hkv, cap = ktail.shape[1], ktail.shape[2]
    P = 0 if kpre is None else kpre.shape[1]
    dtype = SR_BF16 if ktail.dtype in (torch.int16, torch.bfloat16) else SR_F32
    _check(lib().sr_decode_attention_noalloc(dtype, hd, hq, hkv, rows, _ptr(q), _ptr(kpre), _ptr(vpre), P,
                                             _ptr(ktail), _ptr(vtail), cap, lt, _ptr(out), _stream(stream)))


def decode_attention_noalloc_limit() -> int:
    """Bytes of the static scratch behind sr_decode_attention_noalloc."""
    return int(lib().sr_decode_attention_noalloc_limit())


def prefill_attention(q, kpre, vpre, kown, vown, t0: int, out, stream=None):
    """sr_prefill_attention: q float [rows][lr][hq][hd]; kpre/vpre [hkv][P][hd]
    (or None when P = 0); kown/vown [rows][hkv][cap][hd] holding each row's
    positions 0..t0+lr-1; out [rows][lr][hq*hd] in the model dtype (bf16
    tensors travel as int16).  See the header."""
    import torch
    rows, lr, hq, hd = q.shape
    hkv, cap = kown.shape[1], kown.shape[2]
    P = 0 if kpre is None else kpre.shape[1]
    dtype = SR_BF16 if kown.dtype in (torch.int16, torch.bfloat16) else SR_F32
    _check(lib().sr_prefill_attention(dtype, hd, hq, hkv, rows, lr, _ptr(q), _ptr(kpre), _ptr(vpre), P, _ptr(kown),
                                      _ptr(vown), cap, t0, _ptr(out), _stream(stream)))


def logits_teacher_forced(gen: DeviceModel, rm: DeviceModel, prompt, p: sr_params, tokens, ws: Workspace,
                          stream=None):
    """Logits [rows][len][V] of every response position, through the decode path."""
    import torch
    prompt = np.ascontiguousarray(np.asarray(prompt, dtype=np.int32))
    rows, length = tokens.shape
    out = torch.empty((rows, length, gen.shape.vocab), dtype=torch.float32, device=tokens.device)
    _check(lib().sr_logits_teacher_forced(ctypes.byref(gen.desc), _mref(rm), prompt.ctypes.data,
                                          len(prompt), ctypes.byref(p), _ptr(tokens), rows, length, _ptr(out),
                                          ws.ptr, ws.nbytes, _stream(stream)))
    return out


def reward_scores(gen: DeviceModel, rm: DeviceModel, prompt, p: sr_params, tokens, lens, ws: Workspace,
                  stream=None):
    """Reward of each response row (tokens [rows][max_len], lens [rows])."""
    import torch
    prompt = np.ascontiguousarray(np.asarray(prompt, dtype=np.int32))
    rows, max_len = tokens.shape
    out = torch.empty(rows, dtype=torch.float32, device=tokens.device)
    _check(lib().sr_reward_scores(ctypes.byref(gen.desc), _mref(rm), prompt.ctypes.data,
                                  len(prompt), ctypes.byref(p), _ptr(tokens), _ptr(lens), rows, max_len, _ptr(out),
                                  ws.ptr, ws.nbytes, _stream(stream)))
    return out
