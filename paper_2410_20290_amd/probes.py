"""Measurement launches for profiling (run under rocprofv3 from any cwd).

    python3 <repo>/paper_2410_20290_amd/probes.py traffic
        A 1 GiB device copy (to scale the FETCH_SIZE / WRITE_SIZE counters),
        then the decode projections of the 8B-shaped generator at 103 and at
        21 rows, three launches each; prints the algorithmic bytes of each.
    python3 <repo>/paper_2410_20290_amd/probes.py gemm [rows,rows,...]
        Graph-replay timing of the projections at the given row counts, each
        launch on a different copy of the weights (>= 1 GiB in all).
    python3 <repo>/paper_2410_20290_amd/probes.py sample
        Timing of the sampler over 512, 103 and 21 rows of 8B-shaped logits.
    python3 <repo>/paper_2410_20290_amd/probes.py attn
        Timing of decode attention at the row counts and tail lengths of the
        three rounds of the 8B-shaped run.
    python3 <repo>/paper_2410_20290_amd/probes.py vendor [rows]
        For comparison only: the four projections of the 8B-shaped model at
        one row count (default 32768, a reward-model prefill chunk) through
        sr_projection and through torch.matmul (the vendor GEMM library) on
        the same operands; the library's product is plain (no SwiGLU, bf16
        out), so it writes more bytes than the fused paired projection.
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

SHAPES = [("qkv", 6144, 4096, 0), ("o", 4096, 4096, 1), ("w13", 14336, 4096, 2), ("w2", 4096, 14336, 1),
          ("head", 128256, 4096, 0)]


def _operands(torch, M, N, K, mode):
    import paper_2410_20290_amd as sr
    nw = 2 * N if mode == 2 else N
    x = torch.randn(M, K, device="cuda").to(torch.bfloat16).view(torch.int16)
    w = (torch.randn(nw, K, device="cuda") * 0.02).to(torch.bfloat16).view(torch.int16)
    out = torch.zeros(M, N, device="cuda", dtype=torch.float32 if mode in (0, 1) else torch.int16)
    need = int(sr.lib().sr_projection_scratch(1, M, N, K, mode))
    part = torch.empty(max(need, 1), dtype=torch.float32, device="cuda")
    return x, w, out, part, need, nw


def _launch(torch, x, w, out, part, need, M, N, K, mode):
    import paper_2410_20290_amd as sr
    st = sr.lib().sr_projection(1, x.data_ptr(), w.data_ptr(), M, N, K, mode, out.data_ptr(), part.data_ptr(),
                                need, torch.cuda.current_stream().cuda_stream)
    if st != 0:
        raise RuntimeError(sr.last_error())


def traffic():
    import torch
    n = 256 << 20
    a = torch.ones(n, device="cuda")
    b = torch.empty(n, device="cuda")
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print("copy_bytes", 4 * n, flush=True)
    for M in (103, 21):
        for name, N, K, mode in SHAPES:
            x, w, out, part, need, nw = _operands(torch, M, N, K, mode)
            torch.cuda.synchronize()
            for _ in range(3):
                _launch(torch, x, w, out, part, need, M, N, K, mode)
            torch.cuda.synchronize()
            alg = 2 * (nw * K + M * K) + M * N * (8 if mode == 1 else (2 if mode == 2 else 4))
            print("shape", M, name, N, K, mode, alg, flush=True)


def gemm(rows):
    import torch

    def gtime(f, reps=10):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            f()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                f()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (2 * reps) * 1e-3

    for M in rows:
        for name, N, K, mode in SHAPES:
            if name == "head" and M > 512:
                continue
            x, w, out, part, need, nw = _operands(torch, M, N, K, mode)
            # weight copies totalling >= 1 GiB, one per launch in turn, so that
            # no launch finds its weights in the last-level cache (as in a
            # decode step, which streams every layer's weights once)
            copies = [w] + [w.clone() for _ in range(max(0, -(-(1 << 30) // (2 * nw * K)) - 1))]
            turn = [0]

            def one():
                wc = copies[turn[0] % len(copies)]
                turn[0] += 1
                _launch(torch, x, wc, out, part, need, M, N, K, mode)

            t = gtime(lambda: [one() for _ in range(len(copies))]) / len(copies)
            del copies
            fl = 2.0 * M * nw * K
            by = 2.0 * (nw * K + M * K) + M * N * 4
            print(json.dumps({"M": M, "op": name, "us": round(t * 1e6, 1), "TFLOPs": round(fl / t / 1e12, 1),
                              "GBs": round(by / t / 1e9)}), flush=True)


def attn(cases):
    """Graph-replay timing of decode attention at (rows, tail length) cases
    of the 8B shape (prefix 256)."""
    import torch
    import paper_2410_20290_amd as sr

    def gtime(f, reps=10):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            f()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                f()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    hq, hkv, hd, P = 32, 8, 128, 256
    for rows, lt in cases:
        cap = lt
        q = torch.randn(rows, hq, hd, device="cuda")
        kp = (torch.randn(hkv, P, hd, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
        vp = torch.randn(hkv, P, hd, device="cuda").to(torch.bfloat16).view(torch.int16)
        kt = (torch.randn(rows, hkv, cap, hd, device="cuda") * 0.5).to(torch.bfloat16).view(torch.int16)
        vt = torch.randn(rows, hkv, cap, hd, device="cuda").to(torch.bfloat16).view(torch.int16)
        out = torch.empty(rows, hq * hd, device="cuda", dtype=torch.int16)
        t = gtime(lambda: sr.decode_attention(q, kp, vp, kt, vt, lt, out))
        by = 2 * hkv * hd * 2 * (P + rows * lt) + rows * hq * hd * (4 + 2)
        print(json.dumps({"rows": rows, "lt": lt, "us": round(t * 1e6, 1), "GBs": round(by / t / 1e9)}), flush=True)


def vendor(M):
    import torch

    def etime(f, reps=10):
        f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            f()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    for name, N, K, mode in SHAPES[:4]:
        x, w, out, part, need, nw = _operands(torch, M, N, K, mode)
        t_sr = etime(lambda: _launch(torch, x, w, out, part, need, M, N, K, mode))
        xb, wb = x.view(torch.bfloat16), w.view(torch.bfloat16)
        t_lib = etime(lambda: torch.matmul(xb, wb.t()))
        fl = 2.0 * M * nw * K
        print(json.dumps({"M": M, "op": name, "sr_us": round(t_sr * 1e6, 1), "sr_TFLOPs": round(fl / t_sr / 1e12),
                          "library_us": round(t_lib * 1e6, 1), "library_TFLOPs": round(fl / t_lib / 1e12)}),
              flush=True)
        del x, w, out, part, xb, wb
        torch.cuda.empty_cache()


def sample_timing(rows_list):
    """Graph-replay timing of the sampler over 8B-shaped logits rows."""
    import torch
    import paper_2410_20290_amd as sr
    V = 128256
    for rows in rows_list:
        logits = torch.randn(rows, V, device="cuda") * 2.0
        cand = torch.arange(rows, dtype=torch.int32, device="cuda")
        tok = torch.empty(rows, dtype=torch.int32, device="cuda")
        f = lambda: sr.sample(logits, cand, 7, 1.0, 42, tok)
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            f()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(10):
                f()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 10 * 1e-3
        print(json.dumps({"rows": rows, "vocab": V, "us": round(t * 1e6, 1),
                          "GBs": round(rows * V * 4 / t / 1e9)}), flush=True)


if __name__ == "__main__":
    if sys.argv[1] == "traffic":
        traffic()
    elif sys.argv[1] == "sample":
        sample_timing([512, 103, 21])
    elif sys.argv[1] == "vendor":
        vendor(int(sys.argv[2]) if len(sys.argv) > 2 else 32768)
    elif sys.argv[1] == "attn":
        attn([(512, 64), (512, 128), (103, 200), (103, 400), (103, 630), (21, 650), (21, 850), (21, 1020)])
    else:
        gemm([int(v) for v in (sys.argv[2] if len(sys.argv) > 2 else "21,103,512,4096,32768").split(",")])
