"""Decode attention (sr_decode_attention) and prefill attention
(sr_prefill_attention) against the oracle's float64 attention on the same
bf16 / fp32 inputs: shared prefix plus each row's own keys, ragged tails, no
prefix, prefix only, cached history before the new tokens, every query-group
size and head size the kernels take.  Each row's max-abs error is bounded
relative to the max-abs of that row of the oracle's output: 1e-2 for bf16,
1e-5 for fp32."""
import numpy as np
import pytest

from gpu_util import need_gpu, say
from oracle.transformer import causal_attention, decode_attention

pytestmark = pytest.mark.gpu


def bf16_round(a):
    u = a.astype(np.float32).view(np.uint32)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.view(np.float32)


def to_dev(torch, a, bf16):
    if bf16:
        return torch.from_numpy((a.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).cuda()
    return torch.from_numpy(a.astype(np.float32)).cuda()


CASES = [
    # dtype, hd, hq, hkv, rows, P, lt, cap
    ("bf16", 128, 32, 8, 103, 256, 300, 320),
    ("bf16", 128, 32, 8, 21, 256, 700, 704),
    ("bf16", 128, 32, 8, 40, 256, 1, 128),
    ("bf16", 128, 32, 8, 128, 256, 50, 64),
    ("bf16", 128, 32, 8, 160, 256, 20, 32),
    ("bf16", 128, 32, 8, 512, 256, 127, 128),     # first round of the 8B schedule
    ("bf16", 128, 32, 8, 512, 256, 1, 128),
    ("bf16", 128, 32, 8, 1024, 256, 33, 40),      # largest row count of the MFMA streaming form
    ("bf16", 128, 64, 8, 300, 256, 0, 16),
    ("bf16", 128, 16, 8, 129, 40, 300, 320),
    ("bf16", 128, 8, 8, 130, 70, 33, 40),         # one query head per KV head; prefix not a multiple of 64
    ("bf16", 128, 32, 8, 160, 600, 10, 16),       # prefix longer than the stage ring
    ("bf16", 128, 64, 8, 12, 100, 90, 96),
    ("bf16", 128, 32, 8, 17, 0, 77, 80),
    ("bf16", 128, 32, 8, 5, 256, 0, 16),
    ("bf16", 128, 8, 8, 3, 31, 5, 8),
    ("bf16", 128, 16, 2, 9, 64, 130, 130),
    ("bf16", 64, 32, 8, 33, 256, 129, 130),
    ("bf16", 64, 8, 2, 7, 128, 33, 40),
    # row groups sharing the prefix: head_dim 64 at the 1B run's rows, four
    # and eight query heads per KV head, a partial last group
    ("bf16", 64, 32, 8, 256, 256, 129, 130),
    ("bf16", 64, 32, 8, 66, 256, 500, 512),
    ("bf16", 64, 8, 2, 64, 128, 33, 40),
    ("bf16", 128, 64, 8, 101, 256, 77, 80),
    ("bf16", 128, 32, 8, 64, 33, 1, 8),
    ("f32", 32, 4, 4, 16, 32, 17, 64),
    ("f32", 32, 8, 1, 6, 5, 3, 3),
]


@pytest.mark.parametrize("dtype,hd,hq,hkv,rows,P,lt,cap", CASES)
def test_decode_attention(dtype, hd, hq, hkv, rows, P, lt, cap):
    torch, sr = need_gpu()
    say(f"decode attention {dtype} hd={hd} hq={hq} hkv={hkv} rows={rows} P={P} lt={lt} cap={cap}")
    bf16 = dtype == "bf16"
    rng = np.random.default_rng(hd + hq + rows + P + lt)
    q = rng.normal(size=(rows, hq, hd)).astype(np.float32)
    kp, vp = rng.normal(size=(2, hkv, P, hd)).astype(np.float32)
    kt, vt = rng.normal(size=(2, rows, hkv, cap, hd)).astype(np.float32)
    if bf16:
        kp, vp, kt, vt = (bf16_round(a) for a in (kp, vp, kt, vt))
    out = torch.zeros((rows, hq * hd), dtype=torch.int16 if bf16 else torch.float32, device="cuda")
    qd = torch.from_numpy(q).cuda()
    kpd = to_dev(torch, kp, bf16) if P else None
    vpd = to_dev(torch, vp, bf16) if P else None
    sr.decode_attention(qd, kpd, vpd, to_dev(torch, kt, bf16), to_dev(torch, vt, bf16), lt, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    if bf16:
        got = (got.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    got = got.reshape(rows, hq, hd)
    worst = 0.0
    for r in range(rows):
        k = np.concatenate([kp.transpose(1, 0, 2), kt[r, :, :lt].transpose(1, 0, 2)], axis=0).astype(np.float64)
        v = np.concatenate([vp.transpose(1, 0, 2), vt[r, :, :lt].transpose(1, 0, 2)], axis=0).astype(np.float64)
        ref = decode_attention(q[r].astype(np.float64), k, v, hkv)
        worst = max(worst, float(np.abs(got[r] - ref).max() / np.abs(ref).max()))
    tol = 1e-2 if bf16 else 1e-5
    assert worst <= tol, worst


PREFILL_CASES = [
    # dtype, hd, hq, hkv, rows, P, t0, lr, cap
    ("bf16", 128, 32, 8, 3, 40, 37, 29, 70),      # matrix-core kernel, ragged tiles
    ("bf16", 128, 32, 8, 2, 256, 128, 100, 636),  # 8B shapes: second scoring round
    ("bf16", 128, 32, 8, 2, 256, 0, 128, 128),    # 8B shapes: first scoring round (two 16-query blocks a work-group)
    ("bf16", 128, 32, 8, 2, 7, 45, 130, 200),     # ragged last block, last work-group with one block
    ("bf16", 64, 32, 8, 2, 30, 3, 150, 160),      # head_dim 64
    ("bf16", 128, 16, 8, 2, 20, 5, 70, 80),       # 2 query heads per KV head: 4 blocks a work-group, 5 blocks
    ("bf16", 128, 8, 8, 2, 0, 16, 33, 49),
    ("bf16", 128, 16, 2, 2, 17, 0, 50, 64),
    ("bf16", 128, 32, 8, 1, 5, 0, 1, 1),
    ("bf16", 64, 8, 2, 3, 33, 20, 17, 40),
    ("f32", 32, 4, 4, 2, 5, 9, 11, 20),
    ("f32", 64, 8, 2, 1, 0, 0, 1, 1),
    ("f32", 32, 8, 1, 2, 3, 64, 40, 110),
]


@pytest.mark.parametrize("dtype,hd,hq,hkv,rows,P,t0,lr,cap", PREFILL_CASES)
def test_prefill_attention(dtype, hd, hq, hkv, rows, P, t0, lr, cap):
    """The new tokens' outputs equal the last lr rows of the causal attention
    of the whole sequence (prefix, cached tokens, new tokens)."""
    torch, sr = need_gpu()
    say(f"prefill attention {dtype} hd={hd} hq={hq} hkv={hkv} rows={rows} P={P} t0={t0} lr={lr} cap={cap}")
    bf16 = dtype == "bf16"
    rng = np.random.default_rng(hd + hq + rows + P + t0 + lr)
    q = rng.normal(size=(rows, lr, hq, hd)).astype(np.float32)
    kp, vp = rng.normal(size=(2, hkv, P, hd)).astype(np.float32)
    ko, vo = rng.normal(size=(2, rows, hkv, cap, hd)).astype(np.float32)   # beyond t0 + lr: never read
    if bf16:
        kp, vp, ko, vo = (bf16_round(a) for a in (kp, vp, ko, vo))
    out = torch.zeros((rows, lr, hq * hd), dtype=torch.int16 if bf16 else torch.float32, device="cuda")
    kpd = to_dev(torch, kp, bf16) if P else None
    vpd = to_dev(torch, vp, bf16) if P else None
    sr.prefill_attention(torch.from_numpy(q).cuda(), kpd, vpd, to_dev(torch, ko, bf16), to_dev(torch, vo, bf16), t0,
                         out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    if bf16:
        got = (got.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    got = got.reshape(rows, lr, hq, hd)
    T = P + t0 + lr
    worst = 0.0
    for r in range(rows):
        k = np.concatenate([kp.transpose(1, 0, 2), ko[r, :, :t0 + lr].transpose(1, 0, 2)], axis=0).astype(np.float64)
        v = np.concatenate([vp.transpose(1, 0, 2), vo[r, :, :t0 + lr].transpose(1, 0, 2)], axis=0).astype(np.float64)
        qf = np.zeros((T, hq, hd))
        qf[T - lr:] = q[r]
        ref = causal_attention(qf, k, v, hkv)[T - lr:]
        worst = max(worst, float(np.abs(got[r] - ref).max() / np.abs(ref).max()))
    tol = 1e-2 if bf16 else 1e-5
    assert worst <= tol, worst
