"""Next-token sampling, eq. (auto-regressive) of section 3.

The paper samples y^{k+1} ~ p(. | x, y^{<=k}) and names no temperature,
top-k or top-p, so p is the plain softmax of the logits divided by the
temperature T.  To make a token a function of the logits alone (so that the
CPU and the GPU agree on every draw given the same logits), the draw is an
integer inverse CDF:

1. m = max_i l_i;  z_i = (l_i - m) * (1/T), two float32 roundings, where
   1/T is rounded to float32 from T taken as a float32.
2. p_i = exp_sr(z_i), a fully specified float32 exponential (below).
3. w_i = trunc(p_i * 2^32) as an unsigned 64-bit integer; W = sum_i w_i.
4. x = word 0 of Philox4x32-10(counter = (step, candidate, 0, 0),
   key = (seed mod 2^32, seed div 2^32)).
5. t = floor(x * W / 2^32), computed exactly.
6. token = min { i : w_0 + ... + w_i > t }.

Since x < 2^32, t < W, so some token is always drawn, and a token with
w_i = 0 never is.  T = 0 means greedy decoding (first index of the maximum).
A row with no positive weight (every logit -inf or NaN) has no distribution;
it yields token 0.

exp_sr follows Cody and Waite's range reduction (Software Manual for the
Elementary Functions, 1980): n = rint(z * log2 e), r = z - n*ln2_hi - n*ln2_lo
with ln2_hi carrying few enough bits that n*ln2_hi is exact, then the
degree-7 Taylor polynomial of e^r (coefficients 1/j! in float32) by Horner's
rule, then scaling by 2^n.  Every operation is a separately rounded float32
multiply or add (no fused multiply-add), in the order written here.
Inputs below -24 give 0 (their weight would truncate to 0 anyway); NaN
logits are ignored by the maximum and get weight 0.
"""
import numpy as np

from .philox import philox4x32_10

F32 = np.float32
LOG2E = F32(1.4426950408889634)
LN2_HI = F32(0.693145751953125)            # 0x3F317200: 15 significant bits
LN2_LO = F32(0.6931471805599453 - 0.693145751953125)
COEF = [F32(1.0), F32(1.0), F32(1.0 / 2), F32(1.0 / 6), F32(1.0 / 24),
        F32(1.0 / 120), F32(1.0 / 720), F32(1.0 / 5040)]
EXP_CUTOFF = F32(-24.0)
TWO32 = F32(4294967296.0)


def exp_sr(z):
    """float32 e^z for z <= 0, elementwise, as specified above."""
    z = np.asarray(z, dtype=F32)
    below = ~(z >= EXP_CUTOFF)                 # below the cutoff, -inf or NaN
    with np.errstate(invalid="ignore", over="ignore"):
        zc = np.where(below, F32(0.0), z).astype(F32)
        t = (zc * LOG2E).astype(F32)
        n = np.rint(t).astype(F32)
        r = (zc - (n * LN2_HI).astype(F32)).astype(F32)
        r = (r - (n * LN2_LO).astype(F32)).astype(F32)
        p = COEF[7]
        for j in range(6, -1, -1):
            p = ((p * r).astype(F32) + COEF[j]).astype(F32)
        out = np.ldexp(p, n.astype(np.int32)).astype(F32)
    return np.where(below, F32(0.0), out).astype(F32)


def uniform_word(seed: int, cand: int, step: int) -> int:
    """The 32-bit uniform keyed by (seed, candidate, step)."""
    return philox4x32_10((step, cand, 0, 0), (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF))[0]


def inverse_temperature(temperature: float):
    """1/T rounded to float32, from T as a float32 (the interface's type)."""
    return F32(1.0 / float(F32(temperature)))


def weights(logits, temperature: float):
    """Integer weights w_i (uint64) of one row of float32 logits (NaN -> 0)."""
    l = np.asarray(logits, dtype=F32)
    m = np.nanmax(l)
    inv_t = inverse_temperature(temperature)
    z = ((l - m).astype(F32) * inv_t).astype(F32)
    p = exp_sr(z)
    return (p * TWO32).astype(F32).astype(np.uint64)


def draw_threshold(x: int, total: int) -> int:
    """floor(x * W / 2^32) for x < 2^32, W < 2^64, without overflow."""
    return x * (total >> 32) + ((x * (total & 0xFFFFFFFF)) >> 32)


def sample(logits, temperature: float, seed: int, cand: int, step: int) -> int:
    """Token drawn for candidate ``cand`` at generation step ``step``."""
    l = np.asarray(logits, dtype=F32)
    if np.isnan(l).all() or (l[~np.isnan(l)] == -np.inf).all():
        return 0
    if temperature == 0.0:
        return int(np.flatnonzero(l == np.nanmax(l))[0])
    w = weights(l, temperature)
    total = int(w.sum(dtype=np.uint64))
    if total == 0:
        return 0
    t = draw_threshold(uniform_word(seed, cand, step), total)
    return inverse_cdf(w, t)


def inverse_cdf(w, t: int) -> int:
    """Step 6: the first index i whose cumulative weight w_0 + ... + w_i
    exceeds t strictly (a t equal to a cumulative weight falls to the next
    token with positive weight)."""
    cum = np.cumsum(np.asarray(w, dtype=np.uint64), dtype=np.uint64)
    return int(np.searchsorted(cum, np.uint64(t), side="right"))
