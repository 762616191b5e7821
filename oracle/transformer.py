"""The generator p and the reward model s of section 3, in float64.

The paper treats both as black boxes: p is sampled auto-regressively
(eq. auto-regressive), s maps prompt and response to a real number (section 3,
"Inference-time Alignment"), evaluated on the concatenation of the prompt and
a (partial) response (section 4.2, eq. partial-reward-set).  Its models are
Llama-3-8B and Mistral-7B-shaped decoders (section 5), so both are written
here as a pre-norm Llama-style decoder:

* h_0 = E[token]
* per layer: a = RMSNorm(h) * g_attn;  q, k, v = a Wq^T, a Wk^T, a Wv^T;
  rotate-half RoPE on q and k at the token's absolute position;
  causal attention with grouped KV heads (query head j reads KV head
  floor(j * hkv / hq)), scale 1/sqrt(hd);  h += o Wo^T;
  f = RMSNorm(h) * g_ffn;  h += (silu(f W1^T) * (f W3^T)) W2^T
* out = RMSNorm(h) * g_final.
* generator: logits = out W_head^T (untied head);
  reward model: s = w_head . out[last token] (a scalar head, no bias).

RMSNorm(x) = x / sqrt(mean(x^2) + eps).  RoPE frequency i is
theta^(-2i/hd); pair (x_i, x_{i+hd/2}) rotates by position * frequency.

Weights come in the packed layout of the C interface: wqkv [nl][(hq+2hkv)hd][d]
(q rows, then k, then v), wo [nl][d][hq hd], w13 [nl][2][ff][d] (gate, up),
w2 [nl][d][ff]; bf16 weights as uint16 bit patterns, widened exactly.

The per-candidate decode state keeps a private KV cache for every row,
prompt included: nothing is shared between candidates here.

bf16 operands (``bf16_operands=True``): the same model as a bf16 model
computes it in mixed precision -- the operands of every matrix product are
rounded to bf16 (round to nearest even): the normalised activations entering
a projection, the attention output entering Wo, the SwiGLU product entering
W2, the final normalised state entering the head, and in attention q, k (the
score product) and the softmax probabilities and v (the value product);
products accumulate, and everything else is computed, in float32.  The paper fixes no
precision; this mode exists to measure how far a bf16 model drifts from the
exact one on given inputs (the scale a bf16 implementation is compared at),
never as the reference itself.
"""
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np


def to_bf16(x, dtype=np.float64) -> np.ndarray:
    """Round to the nearest bf16 value, ties to even (via float32: float64
    values are first rounded to float32, as a float32 pipeline holds them),
    returned as `dtype`.  NaN stays NaN, infinities stay infinite, values
    beyond the largest bf16 round to infinity."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    out = np.where(np.isnan(f), np.float32(np.nan), out)
    return out.astype(dtype)


def _to_bf16_f32(x) -> np.ndarray:
    return to_bf16(x, np.float32)


def _same(x):
    return x


def _widen_block(a, dtype=np.float64) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(dtype)
    return a.astype(dtype)


def widen(a, dtype=np.float64) -> np.ndarray:
    """Weights as float64 (or `dtype`; bf16 bit patterns are widened
    exactly).  Large arrays are widened in row blocks on several threads
    (numpy's casts run without the interpreter lock); the result is the
    same."""
    a = np.asarray(a)
    if a.ndim == 0 or a.size < (1 << 22):
        return _widen_block(a, dtype)
    out = np.empty(a.shape, dtype=dtype)
    flat_in, flat_out = a.reshape(-1), out.reshape(-1)
    n = flat_in.size
    parts = min(32, os.cpu_count() or 1)
    step = -(-n // parts)

    def one(i):
        flat_out[i * step:(i + 1) * step] = _widen_block(flat_in[i * step:(i + 1) * step], dtype)

    with ThreadPoolExecutor(parts) as ex:
        list(ex.map(one, range(parts)))
    return out


def rmsnorm(x, g, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x):
    return x / (1.0 + np.exp(-x))


def rope_cos_sin(positions, head_dim, theta):
    half = head_dim // 2
    freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[..., None] * freq
    return np.cos(ang), np.sin(ang)


def rope(x, cos, sin):
    """Rotate-half RoPE on the last axis; cos/sin broadcast over heads."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def softmax(x, axis=-1):
    m = np.max(x, axis=axis, keepdims=True)
    e = np.exp(x - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def causal_attention(q, k, v, n_kv_heads, operand=_same):
    """Causal attention of one sequence: q [T][hq][hd], k, v [T][hkv][hd].

    Query head j reads KV head floor(j * hkv / hq); query i sees keys 0..i.
    ``operand`` is applied to the operands of the two matrix products.
    """
    T, hq, hd = q.shape
    mask = np.triu(np.ones((T, T), dtype=bool), k=1)
    q, k, v = operand(q), operand(k), operand(v)
    o = np.empty_like(q)
    for j in range(hq):
        kh = (j * n_kv_heads) // hq
        sc = (q[:, j, :] @ k[:, kh, :].T) / math.sqrt(hd)
        sc[mask] = -np.inf
        o[:, j, :] = operand(softmax(sc)) @ v[:, kh, :]
    return o


def decode_attention(q, k, v, n_kv_heads):
    """Attention of one new query per head over a cached sequence (the decode
    step of section 4.2): q [hq][hd]; k, v [T][hkv][hd], the query being the
    newest position, so it sees all T keys.  Equals the last row of
    ``causal_attention`` over the same keys."""
    hq, hd = q.shape
    o = np.empty_like(q)
    for j in range(hq):
        kh = (j * n_kv_heads) // hq
        sc = (k[:, kh, :] @ q[j]) / np.sqrt(hd)
        o[j] = softmax(sc) @ v[:, kh, :]
    return o


class Transformer:
    """A decoder given by a shape (see ``synth.ModelShape``) and weights."""

    def __init__(self, shape, weights: dict, reward: bool, cache_f64: bool = None, bf16_operands: bool = False):
        self.s = shape
        self.reward = reward
        self.raw = weights
        self.bf16_operands = bf16_operands
        self.op = _to_bf16_f32 if bf16_operands else _same
        self.ft = np.float32 if bf16_operands else np.float64   # arithmetic type
        nparams = sum(int(np.prod(np.shape(v))) for v in weights.values())
        self.cache_f64 = (nparams * 8 < (4 << 30)) if cache_f64 is None else cache_f64
        self._c = {}

    # -- weight access -------------------------------------------------
    def w(self, name, layer=None):
        key = (name, layer)
        if key in self._c:
            return self._c[key]
        a = self.raw[name] if layer is None else self.raw[name][layer]
        a = widen(a, self.ft)
        if self.cache_f64:
            self._c[key] = a
        return a

    def _split_qkv(self, qkv):
        s = self.s
        nq, nk = s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
        q = qkv[..., :nq].reshape(qkv.shape[:-1] + (s.n_heads, s.head_dim))
        k = qkv[..., nq:nq + nk].reshape(qkv.shape[:-1] + (s.n_kv_heads, s.head_dim))
        v = qkv[..., nq + nk:].reshape(qkv.shape[:-1] + (s.n_kv_heads, s.head_dim))
        return q, k, v

    def _ffn(self, h, l):
        s = self.s
        f = self.op(rmsnorm(h, self.w("ffn_norm", l), s.rms_eps))
        w13 = self.w("w13", l)
        gate = f @ w13[0].T
        up = f @ w13[1].T
        return self.op(silu(gate) * up) @ self.w("w2", l).T

    def kv_head_of(self, j):
        return (j * self.s.n_kv_heads) // self.s.n_heads

    # -- full causal forward over one sequence ---------------------------
    def forward(self, tokens):
        """Final normalised hidden states [T][d] of one token sequence."""
        s = self.s
        tokens = np.asarray(tokens, dtype=np.int64)
        T = len(tokens)
        h = self.w("embed")[tokens] if self.cache_f64 else widen(self.raw["embed"][tokens], self.ft)
        cos, sin = rope_cos_sin(np.arange(T), s.head_dim, s.rope_theta)
        cos, sin = cos[:, None, :].astype(self.ft), sin[:, None, :].astype(self.ft)
        for l in range(s.n_layers):
            a = self.op(rmsnorm(h, self.w("attn_norm", l), s.rms_eps))
            q, k, v = self._split_qkv(a @ self.w("wqkv", l).T)
            q, k = rope(q, cos, sin), rope(k, cos, sin)
            o = causal_attention(q, k, v, s.n_kv_heads, self.op)
            h = h + self.op(o.reshape(T, -1)) @ self.w("wo", l).T
            h = h + self._ffn(h, l)
        return rmsnorm(h, self.w("final_norm"), s.rms_eps)

    def forward_many(self, seqs, progress=None):
        """``forward`` of several token sequences at once: the final
        normalised hidden states [T_i][d] of each.  The sequences share each
        layer's projections (their rows stacked) and attend only to
        themselves, so every layer's weights are widened once for all of
        them (for models too large to keep widened).  ``progress(l)`` is
        called after layer l when given."""
        s = self.s
        seqs = [np.asarray(t, dtype=np.int64) for t in seqs]
        lens = [len(t) for t in seqs]
        ends = np.cumsum(lens)
        starts = ends - np.asarray(lens)
        allt = np.concatenate(seqs)
        h = self.w("embed")[allt] if self.cache_f64 else widen(self.raw["embed"][allt], self.ft)
        pos = np.concatenate([np.arange(T) for T in lens])
        cos, sin = rope_cos_sin(pos, s.head_dim, s.rope_theta)
        cos, sin = cos[:, None, :].astype(self.ft), sin[:, None, :].astype(self.ft)
        for l in range(s.n_layers):
            a = self.op(rmsnorm(h, self.w("attn_norm", l), s.rms_eps))
            q, k, v = self._split_qkv(a @ self.w("wqkv", l).T)
            q, k = rope(q, cos, sin), rope(k, cos, sin)
            o = np.empty_like(q)
            for b, e in zip(starts, ends):
                o[b:e] = causal_attention(q[b:e], k[b:e], v[b:e], s.n_kv_heads, self.op)
            h = h + self.op(o.reshape(len(allt), -1)) @ self.w("wo", l).T
            h = h + self._ffn(h, l)
            if progress:
                progress(l)
        out = rmsnorm(h, self.w("final_norm"), s.rms_eps)
        return [out[b:e] for b, e in zip(starts, ends)]

    def logits_at(self, seqs, positions, progress=None):
        """Generator logits at chosen positions of several sequences:
        for sequence i, rows [len(positions[i])][V] with row j the
        distribution of token positions[i][j] + 1 (as ``logits``)."""
        assert not self.reward
        hs = self.forward_many(seqs, progress)
        head = self.w("head")
        return [self.op(h[np.asarray(p, dtype=np.int64)]) @ head.T for h, p in zip(hs, positions)]

    def scores_at(self, seqs, lengths, progress=None):
        """Reward-model scores of prefixes: for sequence i and each length L
        in lengths[i], s(first L tokens) = w_head . out[L - 1].  Under the
        causal mask the state at position L - 1 depends only on the first L
        tokens, so one forward over the whole sequence serves every prefix."""
        assert self.reward
        hs = self.forward_many(seqs, progress)
        head = self.w("head")
        return [np.array([float(self.op(h[L - 1]) @ head) for L in ls]) for h, ls in zip(hs, lengths)]

    def logits(self, tokens):
        """Generator logits [T][V]: row t is the distribution of token t+1."""
        assert not self.reward
        return self.op(self.forward(tokens)) @ self.w("head").T

    def score(self, tokens) -> float:
        """Reward model s(x, y): scalar head on the last token's state."""
        assert self.reward
        out = self.forward(tokens)
        return float(self.op(out[-1]) @ self.w("head"))

    # -- batched incremental decoding with private caches ---------------
    def start(self, prompt, rows: int, capacity: int):
        """Decode state for ``rows`` candidates that all begin with ``prompt``.

        Every row gets its own copy of the prompt's keys and values (the
        prompt forward is deterministic, so it is evaluated once and copied).
        ``capacity`` bounds prompt plus response length.
        Returns (state, logits of the last prompt position [V]).
        """
        assert not self.bf16_operands, "bf16 operands: whole-sequence forwards only"
        s = self.s
        prompt = np.asarray(prompt, dtype=np.int64)
        P = len(prompt)
        h = widen(self.raw["embed"][prompt])
        cos, sin = rope_cos_sin(np.arange(P), s.head_dim, s.rope_theta)
        cos, sin = cos[:, None, :], sin[:, None, :]
        state = {"k": [], "v": [], "pos": P}
        for l in range(s.n_layers):
            a = rmsnorm(h, self.w("attn_norm", l), s.rms_eps)
            q, k, v = self._split_qkv(a @ self.w("wqkv", l).T)
            q, k = rope(q, cos, sin), rope(k, cos, sin)
            o = causal_attention(q, k, v, s.n_kv_heads)
            h = h + o.reshape(P, -1) @ self.w("wo", l).T
            h = h + self._ffn(h, l)
            # private per-row caches [rows][kvh][capacity][hd]
            kc = np.zeros((rows, s.n_kv_heads, capacity, s.head_dim))
            vc = np.zeros((rows, s.n_kv_heads, capacity, s.head_dim))
            kc[:, :, :P] = k.transpose(1, 0, 2)[None]
            vc[:, :, :P] = v.transpose(1, 0, 2)[None]
            state["k"].append(kc)
            state["v"].append(vc)
        out = rmsnorm(h, self.w("final_norm"), s.rms_eps)
        return state, out[-1] @ self.w("head").T

    @staticmethod
    def select_rows(state, idx):
        """Keep only the rows ``idx`` of a decode state."""
        idx = np.asarray(idx, dtype=np.int64)
        return {"k": [k[idx] for k in state["k"]], "v": [v[idx] for v in state["v"]],
                "pos": state["pos"]}

    def step(self, state, tokens):
        """Append one token per row at position state['pos']; return logits [rows][V]."""
        assert not self.bf16_operands, "bf16 operands: whole-sequence forwards only"
        s = self.s
        tokens = np.asarray(tokens, dtype=np.int64)
        rows = len(tokens)
        pos = state["pos"]
        h = widen(self.raw["embed"][tokens])
        cos, sin = rope_cos_sin(np.array([pos]), s.head_dim, s.rope_theta)
        scale = 1.0 / np.sqrt(s.head_dim)
        for l in range(s.n_layers):
            a = rmsnorm(h, self.w("attn_norm", l), s.rms_eps)
            q, k, v = self._split_qkv(a @ self.w("wqkv", l).T)   # [rows][heads][hd]
            q, k = rope(q, cos, sin), rope(k, cos, sin)
            state["k"][l][:, :, pos] = k
            state["v"][l][:, :, pos] = v
            K = state["k"][l][:, :, :pos + 1]                     # [rows][kvh][T][hd]
            V = state["v"][l][:, :, :pos + 1]
            o = np.empty((rows, s.n_heads, s.head_dim))
            for j in range(s.n_heads):
                kh = self.kv_head_of(j)
                sc = np.einsum("rd,rtd->rt", q[:, j, :], K[:, kh]) * scale
                o[:, j, :] = np.einsum("rt,rtd->rd", softmax(sc), V[:, kh])
            h = h + o.reshape(rows, -1) @ self.w("wo", l).T
            h = h + self._ffn(h, l)
        state["pos"] = pos + 1
        out = rmsnorm(h, self.w("final_norm"), s.rms_eps)
        return out @ self.w("head").T
