"""sr_decode_attention_noalloc (the decode attention for callers that cannot
allocate) against sr_decode_attention on the same inputs: two calls in a row
on one device, the second smaller, each bit-identical to the entry point with
a caller scratch buffer (the same kernels) and within the bf16 bound of the
oracle's attention; a call whose partials exceed the static scratch is
rejected before any launch."""
import numpy as np
import pytest

from gpu_util import need_gpu, say
from oracle.transformer import decode_attention

pytestmark = pytest.mark.gpu


def _bf16(a):
    u = a.astype(np.float32).view(np.uint32)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _f32(u16):
    return (u16.astype(np.uint32) << 16).view(np.float32)


def _case(torch, sr, rows, P, lt, cap, hq=32, hkv=8, hd=128, seed=0):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(rows, hq, hd)).astype(np.float32)
    kp, vp = (_bf16(a) for a in rng.normal(size=(2, hkv, P, hd)))
    kt, vt = (_bf16(a) for a in rng.normal(size=(2, rows, hkv, cap, hd)))
    dev = lambda a: torch.from_numpy(a.view(np.int16)).cuda()
    args = (torch.from_numpy(q).cuda(), dev(kp), dev(vp), dev(kt), dev(vt))
    return q, kp, vp, kt, vt, args


# (rows, P, lt, cap): every case leaves split partials in the scratch
@pytest.mark.parametrize("first,second", [((512, 256, 127, 128), (21, 256, 700, 704)),
                                          ((1024, 256, 33, 40), (21, 31, 600, 640))])
def test_noalloc_matches_scratch_entry(first, second):
    torch, sr = need_gpu()
    for rows, P, lt, cap in (first, second):
        say(f"noalloc decode attention rows={rows} P={P} lt={lt} cap={cap}")
        q, kp, vp, kt, vt, args = _case(torch, sr, rows, P, lt, cap, seed=rows + lt)
        hq, hd = q.shape[1], q.shape[2]
        ref_out = torch.zeros((rows, hq * hd), dtype=torch.int16, device="cuda")
        sr.decode_attention(*args, lt, ref_out)
        out = torch.full((rows, hq * hd), -1, dtype=torch.int16, device="cuda")
        sr.decode_attention_noalloc(*args, lt, out)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out)
        got = _f32(out.cpu().numpy().view(np.uint16)).reshape(rows, hq, hd)
        for r in sorted({0, rows // 2, rows - 1}):
            k = np.concatenate([_f32(kp).transpose(1, 0, 2), _f32(kt[r, :, :lt]).transpose(1, 0, 2)]).astype(np.float64)
            v = np.concatenate([_f32(vp).transpose(1, 0, 2), _f32(vt[r, :, :lt]).transpose(1, 0, 2)]).astype(np.float64)
            ref = decode_attention(q[r].astype(np.float64), k, v, 8)
            assert np.abs(got[r] - ref).max() <= 1e-2 * np.abs(ref).max(), r


def test_noalloc_rejects_partials_beyond_the_static_scratch():
    torch, sr = need_gpu()
    limit = sr.decode_attention_noalloc_limit()
    assert limit == 32 << 20
    # 2100 rows of 32 query heads, one per KV head (the row groups that share
    # the prefix take 2, 4 or 8 query heads per KV head): one partial slot of
    # 130 floats per row and head for the prefix pass to fold in, 8.7 M
    # floats > 8 M
    rows, P, lt, cap = 2100, 256, 9, 16
    q = torch.zeros((rows, 32, 128), dtype=torch.float32, device="cuda")
    kp = torch.zeros((32, P, 128), dtype=torch.int16, device="cuda")
    kt = torch.zeros((rows, 32, cap, 128), dtype=torch.int16, device="cuda")
    out = torch.zeros((rows, 32 * 128), dtype=torch.int16, device="cuda")
    with pytest.raises(sr.SpecRejError) as e:
        sr.decode_attention_noalloc(q, kp, kp, kt, kt, lt, out)
    assert e.value.status == sr.SR_ERR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
    assert int(out.abs().sum()) == 0
