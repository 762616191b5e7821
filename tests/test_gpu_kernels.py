"""Kernel-level parity: Philox, the sampler, the cut and the KV compaction
against the oracle, bit-exact (they are integer decisions)."""
import numpy as np
import pytest

from gpu_util import need_gpu, say
from oracle import sampler as osamp
from oracle import specrej
from oracle.philox import philox4x32_10_np

pytestmark = pytest.mark.gpu


def test_philox_bit_exact():
    torch, sr = need_gpu()
    rng = np.random.default_rng(0)
    n = 100_003
    ctr = rng.integers(0, 2**32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
    for seed in (0, 42, (7 << 32) | 99, 2**64 - 1):
        out = torch.empty((n, 4), dtype=torch.int32, device="cuda")
        sr.philox_fill(seed, torch.from_numpy(ctr.view(np.int32)).cuda(), out)
        got = out.cpu().numpy().view(np.uint32)
        ref = philox4x32_10_np(ctr[:, 0], ctr[:, 1], ctr[:, 2], ctr[:, 3], seed & 0xFFFFFFFF, seed >> 32)
        assert np.array_equal(got, np.stack(ref, axis=1))


def oracle_tokens(logits, cand, step, temperature, seed):
    return np.array([osamp.sample(logits[r], temperature, seed, int(cand[r]), step) for r in range(len(cand))])


@pytest.mark.parametrize("vocab", [1, 2, 63, 64, 65, 511, 512, 8192, 32000, 128256])
@pytest.mark.parametrize("temperature", [1.0, 0.7, 0.0])
def test_sampler_bit_exact(vocab, temperature):
    torch, sr = need_gpu()
    say(f"sampler vocab={vocab} T={temperature}")
    rng = np.random.default_rng(vocab)
    rows = 37
    logits = (rng.standard_normal((rows, vocab)) * rng.uniform(0.5, 6.0, size=(rows, 1))).astype(np.float32)
    logits[0, : min(vocab, 5)] = -np.inf           # excluded tokens
    logits[1] = 3.0                                # all equal
    logits[2, vocab // 2] = 80.0                   # near-deterministic
    cand = rng.permutation(4096)[:rows].astype(np.int32)
    for step in (0, 1, 1023):
        tok = torch.empty(rows, dtype=torch.int32, device="cuda")
        sr.sample(torch.from_numpy(logits).cuda(), torch.from_numpy(cand).cuda(), step, temperature, 42, tok)
        got = tok.cpu().numpy()
        ref = oracle_tokens(logits, cand, step, temperature, 42)
        assert np.array_equal(got, ref), (step, np.flatnonzero(got != ref)[:5])


def test_sampler_weights_near_boundaries():
    """Logits spread over the whole exp range, many rows: every weight must
    round exactly as the oracle's float32 steps."""
    torch, sr = need_gpu()
    rng = np.random.default_rng(11)
    rows, vocab = 512, 4096
    logits = rng.uniform(-30, 0, size=(rows, vocab)).astype(np.float32)
    cand = np.arange(rows, dtype=np.int32)
    tok = torch.empty(rows, dtype=torch.int32, device="cuda")
    sr.sample(torch.from_numpy(logits).cuda(), torch.from_numpy(cand).cuda(), 5, 1.0, 7, tok)
    assert np.array_equal(tok.cpu().numpy(), oracle_tokens(logits, cand, 5, 1.0, 7))


@pytest.mark.parametrize("b,keep", [(1, 1), (2, 1), (7, 3), (64, 16), (103, 21), (512, 103), (1000, 999),
                                    (4096, 410)])
def test_select_bit_exact(b, keep):
    torch, sr = need_gpu()
    rng = np.random.default_rng(b)
    scores = rng.normal(size=b).astype(np.float32)
    scores[rng.integers(0, b, size=b // 5)] = np.float32(0.25)   # ties
    if b > 4:
        scores[1] = np.nan
        scores[2] = -np.inf
        scores[3] = -0.0
    cand = rng.permutation(8192)[:b].astype(np.int32)
    acc = torch.empty(b, dtype=torch.int32, device="cuda")
    sr.select(torch.from_numpy(scores).cuda(), torch.from_numpy(cand).cuda(), keep, acc)
    got = acc.cpu().numpy()
    sd = {int(c): float(s) for c, s in zip(cand, scores)}
    kept = set(specrej.top_k([int(c) for c in cand], sd, keep))
    ref = np.array([1 if int(c) in kept else 0 for c in cand])
    assert got.sum() == keep and np.array_equal(got, ref)


@pytest.mark.parametrize("elem_bytes,hd", [(2, 128), (2, 64), (4, 32)])
def test_compact_bit_exact(elem_bytes, hd):
    torch, sr = need_gpu()
    rng = np.random.default_rng(hd)
    nl, hkv, b, cap_src, cap_dst, length = 3, 2, 37, 20, 33, 19
    dt = np.uint16 if elem_bytes == 2 else np.uint32
    sb = b * hkv * cap_src * hd + 17
    db = b * hkv * cap_dst * hd + 5
    src = rng.integers(0, 2**15, size=2 * nl * sb).astype(dt)
    flags = (rng.random(b) < 0.4).astype(np.int32)
    flags[0] = 1
    tdt = torch.int16 if elem_bytes == 2 else torch.int32
    s_t = torch.from_numpy(src.view(np.int16 if elem_bytes == 2 else np.int32)).cuda()
    d_t = torch.zeros(2 * nl * db, dtype=tdt, device="cuda")
    src_row = torch.full((b,), -1, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    sr.compact(s_t, sb, d_t, db, torch.from_numpy(flags).cuda(), nl, hkv, hd, elem_bytes, cap_src, cap_dst, length,
               src_row, cnt)
    torch.cuda.synchronize()
    kept = np.flatnonzero(flags)
    assert int(cnt.item()) == len(kept)
    assert np.array_equal(src_row.cpu().numpy()[: len(kept)], kept)
    dst = d_t.cpu().numpy().view(dt)
    for blk in range(2 * nl):
        S = src[blk * sb: blk * sb + b * hkv * cap_src * hd].reshape(b, hkv, cap_src, hd)
        Dd = dst[blk * db: blk * db + b * hkv * cap_dst * hd].reshape(b, hkv, cap_dst, hd)
        assert np.array_equal(Dd[: len(kept), :, :length], S[kept, :, :length])
        assert not Dd[len(kept):].any() and not Dd[:, :, length:].any()
