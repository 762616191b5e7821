"""Projection GEMM parity (sr_projection) against a float64 product of the
same bf16/fp32 inputs, over ragged shapes, every epilogue and the split-K
path.  The max-abs error is bounded relative to the oracle product's
max-abs: 1e-2 where the output is rounded to bf16, else 1e-4."""
import numpy as np
import pytest

from gpu_util import need_gpu, say

pytestmark = pytest.mark.gpu


def bf16_round(a):
    u = a.astype(np.float32).view(np.uint32)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.view(np.float32)


SHAPES = [(1, 64, 64), (17, 100, 128), (33, 1000, 512), (100, 384, 4096), (129, 130, 64), (300, 257, 1024),
          (512, 512, 14336), (1000, 96, 192), (1100, 300, 256), (2048, 520, 1024), (4000, 129, 64),
          (128, 200, 1024), (64, 64, 14336), (21, 4100, 1792), (112, 130, 384),
          # a few hundred rows with enough 256 x 256 tiles for the three-deep weight ring
          (300, 49152, 256), (257, 24576, 128),
          # the 103-row QKV projection of the 8B shape
          (103, 6144, 4096),
          # 65-112 rows, long K, ragged N
          (70, 2000, 8192), (103, 4096, 14336),
          # 65-112 rows with 2 to 6 K steps of 256 per work-group
          (97, 4150, 512), (65, 4200, 768), (100, 4096, 4096), (112, 4100, 1280), (77, 4200, 1536),
          # 65-112 rows, more than 65536 columns (the LM head's tiles), ragged N
          (103, 66000, 384), (70, 65601, 128),
          # paired few-row tiles with 512-byte rows per copy (K steps of 256), ragged N
          (21, 4100, 2048),
          # thousands of rows, ragged in M and N, ten K steps (the 256 x 256 tile)
          (2600, 1100, 640)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("mode", [0, 1, 2, 3])
@pytest.mark.parametrize("M,N,K", SHAPES)
def test_projection(dtype, mode, M, N, K):
    torch, sr = need_gpu()
    if dtype == "f32" and K > 4096:
        pytest.skip("fp32 model shapes stay small")
    say(f"projection {dtype} mode={mode} M={M} N={N} K={K}")
    rng = np.random.default_rng(M * 7 + N + K + mode)
    x = rng.normal(0, 1, size=(M, K)).astype(np.float32)
    w = rng.normal(0, 0.05, size=((2, N, K) if mode == 2 else (N, K))).astype(np.float32)
    if dtype == "bf16":
        x, w = bf16_round(x), bf16_round(w)
        xt = torch.from_numpy(x.view(np.uint32) >> 16).to(torch.int32).to(torch.int16).cuda()
        wt = torch.from_numpy((w.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).cuda()
        xt = torch.from_numpy((x.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).cuda()
    else:
        xt, wt = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    if mode == 2:
        g, u = x64 @ w64[0].T, x64 @ w64[1].T
        ref = g / (1 + np.exp(-g)) * u
    else:
        ref = x64 @ w64.T
    init = rng.normal(size=(M, N)).astype(np.float32)
    if mode in (0, 1):
        out = torch.from_numpy(init.copy()).cuda()
    else:
        out = torch.zeros((M, N), dtype=torch.int16 if dtype == "bf16" else torch.float32, device="cuda")
    sr.projection(xt, wt, mode, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    if mode in (2, 3) and dtype == "bf16":
        got = (got.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    if mode == 1:
        ref = ref + init
    scale = np.abs(ref).max()
    rtol = 1e-2 if (mode in (2, 3) and dtype == "bf16") else 1e-4
    assert np.abs(got - ref).max() <= rtol * scale, np.abs(got - ref).max()


@pytest.mark.parametrize("M", [8, 41, 103, 120])
def test_projection_paired_8b(M):
    """The 8B gate/up projection (N 14336, K 4096) at the row counts of the
    decode rounds: every few-row tile kind with its rotated K order."""
    torch, sr = need_gpu()
    N, K = 14336, 4096
    say(f"paired projection bf16 M={M} N={N} K={K}")
    rng = np.random.default_rng(M)
    x = bf16_round(rng.normal(0, 1, size=(M, K)).astype(np.float32))
    w = bf16_round(rng.normal(0, 0.02, size=(2, N, K)).astype(np.float32))
    xt = torch.from_numpy((x.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).cuda()
    wt = torch.from_numpy((w.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)).cuda()
    out = torch.zeros((M, N), dtype=torch.int16, device="cuda")
    sr.projection(xt, wt, 2, out)
    torch.cuda.synchronize()
    got = (out.cpu().numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    g, u = x64 @ w64[0].T, x64 @ w64[1].T
    ref = g / (1 + np.exp(-g)) * u
    assert np.abs(got - ref).max() <= 1e-2 * np.abs(ref).max(), np.abs(got - ref).max()
