"""Decode attention (sr_decode_attention) against the oracle's float64
decode attention on the same bf16 / fp32 inputs: shared prefix plus each
row's own tail, ragged tails, no prefix, prefix only, every query-group
size and head size the kernels take."""
import numpy as np
import pytest

from gpu_util import need_gpu, say
from oracle.transformer import decode_attention

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
    ("bf16", 128, 64, 8, 12, 100, 90, 96),
    ("bf16", 128, 32, 8, 17, 0, 77, 80),
    ("bf16", 128, 32, 8, 5, 256, 0, 16),
    ("bf16", 128, 8, 8, 3, 31, 5, 8),
    ("bf16", 128, 16, 2, 9, 64, 130, 130),
    ("bf16", 64, 32, 8, 33, 256, 129, 130),
    ("bf16", 64, 8, 2, 7, 128, 33, 40),
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
        worst = max(worst, float(np.abs(got[r] - ref).max() / max(1.0, np.abs(ref).max())))
    tol = 1e-2 if bf16 else 1e-5
    assert worst <= tol, worst
