"""The QAT layer step captured in a HIP graph (torch.cuda.CUDAGraph).

The library allocates nothing, records no memset and never synchronises, so
a caller may capture its calls.  A captured step (fused quantize + fake-quant
of X and W with computed global scales, the product, the one-call linear and,
for decode-sized X, the packed weight image and the linear call on it)
is replayed several times, with other eager library work and host
synchronisation between replays and its outputs overwritten before each
replay; every replay must reproduce the eager outputs bit for bit.  Eager
parity with the oracle is covered by the other GPU tests.
"""
import pytest
import torch

from paper_2606_15682_amd import reqat

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def log(msg):
    print(msg, flush=True)


def _inputs(M, N, K, seed):
    gen = torch.Generator().manual_seed(seed)
    x = (torch.randn(M, K, generator=gen) * 2.0).to(torch.bfloat16).to(DEV)
    w = (torch.randn(N, K, generator=gen) * 0.02).to(torch.bfloat16).to(DEV)
    return x, w


def _buffers(fmt, M, N, K):
    B = reqat.BLOCK[fmt]
    def q(R):
        return (torch.empty((R, K // 2), dtype=torch.uint8, device=DEV),
                torch.empty((R, K // B), dtype=torch.uint8, device=DEV),
                torch.empty((R, K), dtype=torch.bfloat16, device=DEV),
                torch.empty(1, dtype=torch.float32, device=DEV))
    return {"x": q(M), "w": q(N),
            "y": torch.empty((M, N), dtype=torch.bfloat16, device=DEV),
            "yl": torch.empty((M, N), dtype=torch.bfloat16, device=DEV),
            "gl": torch.empty(1, dtype=torch.float32, device=DEV),
            "lws": torch.empty(max(reqat.reqat_linear_workspace_bytes(fmt, M, K), 16), dtype=torch.uint8,
                               device=DEV),
            "pk": torch.empty(max(reqat.reqat_w4a4_packed_bytes(fmt, N, K), 16), dtype=torch.uint8, device=DEV),
            "yp": torch.empty((M, N), dtype=torch.bfloat16, device=DEV),
            "gp": torch.empty(1, dtype=torch.float32, device=DEV)}


def _step(fmt, x, w, b):
    """One pass of the layer's hot path into the preallocated buffers."""
    xc, xs, xy, xg = b["x"]
    wc, ws, wy, wg = b["w"]
    reqat.quantize_fakequant(x, fmt, out=(xc, xs, xy), g_out=xg if fmt == reqat.NVFP4 else None)
    reqat.quantize_fakequant(w, fmt, out=(wc, ws, wy), g_out=wg if fmt == reqat.NVFP4 else None)
    nv = fmt == reqat.NVFP4
    reqat.gemm(fmt, xc, xs, xg if nv else None, wc, ws, wg if nv else None, out_dtype=torch.bfloat16, out=b["y"])
    reqat.linear(x, fmt, wc, ws, wg if nv else None, out_dtype=torch.bfloat16, out=b["yl"],
                 g_out=b["gl"] if nv else None, ws=b["lws"])
    if x.shape[0] <= 64:
        reqat.pack_w4a4(wc, ws, fmt, out=b["pk"])
        reqat.linear_packed(x, fmt, b["pk"], w.shape[0], wg if nv else None, out_dtype=torch.bfloat16,
                            out=b["yp"], g_out=b["gp"] if nv else None, ws=b["lws"])


def _flat(fmt, b):
    """Every output of the step (the global scales only for NVFP4, which has them)."""
    nv = fmt == reqat.NVFP4
    out = []
    for k in ("x", "w"):
        out += list(b[k][:3]) + ([b[k][3]] if nv else [])
    out += [b["y"], b["yl"]] + ([b["gl"]] if nv else [])
    if b["y"].shape[0] <= 64:
        out += [b["pk"], b["yp"]] + ([b["gp"]] if nv else [])
    return out


def _scramble(fmt, b):
    for t in _flat(fmt, b):
        if t.dtype == torch.uint8:
            t.fill_(0xA5)
        else:
            t.fill_(float("nan"))


@pytest.mark.parametrize("fmt", [reqat.NVFP4, reqat.MXFP4], ids=["nvfp4", "mxfp4"])
@pytest.mark.parametrize("M,N,K", [(300, 520, 1024), (16, 768, 512)])
def test_step_graph_replays_match_eager(fmt, M, N, K):
    log(f"graph step fmt={fmt} M={M} N={N} K={K}")
    nv = int(fmt == reqat.NVFP4)
    x, w = _inputs(M, N, K, seed=1000 + 7 * M + fmt)
    b = _buffers(fmt, M, N, K)
    reqat.workspace(torch.device(DEV))                  # library workspace exists before capture
    _step(fmt, x, w, b)
    torch.cuda.synchronize()
    ref = [t.clone() for t in _flat(fmt, b)]

    # unrelated eager work between replays: the same step on other inputs into other buffers
    x2, w2 = _inputs(M, N, K, seed=2000 + M)
    b2 = _buffers(fmt, M, N, K)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):                          # warm-up on the capture stream
        _step(fmt, x, w, b)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _step(fmt, x, w, b)
    torch.cuda.synchronize()

    if M <= 64:
        assert torch.equal(ref[-1 - nv].view(torch.uint8), ref[-3 - 2 * nv].view(torch.uint8)), \
            "linear on the packed image differs from the row-major linear"
    for rep in range(3):
        _scramble(fmt, b)
        _step(fmt, x2, w2, b2)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(_flat(fmt, b), ref)):
            assert torch.equal(got.view(torch.uint8), want.view(torch.uint8)), \
                f"replay {rep}: output {i} differs from the eager step"
    log("graph replays match")


def test_kv4_graph_replays_match_eager():
    """KV4 quantize (computed g: one pass + fix-up, and a given g) and
    fake-quant of shifted keys, captured and replayed."""
    T, C = 300, 1024
    log(f"graph kv4 T={T} C={C}")
    gen = torch.Generator().manual_seed(77)
    mu = (torch.randn(C, generator=gen) * 2.0).to(DEV)
    def keys(seed):
        g2 = torch.Generator().manual_seed(seed)
        return (torch.randn(T, C, generator=g2) + mu.cpu()).to(torch.bfloat16).to(DEV)
    def bufs():
        return [torch.empty((T, C // 2), dtype=torch.uint8, device=DEV),
                torch.empty((T, C // 16), dtype=torch.uint8, device=DEV),
                torch.empty(1, dtype=torch.float32, device=DEV),
                torch.empty((T, C), dtype=torch.bfloat16, device=DEV),
                torch.empty(1, dtype=torch.float32, device=DEV),
                torch.empty((T, C // 2), dtype=torch.uint8, device=DEV),
                torch.empty((T, C // 16), dtype=torch.uint8, device=DEV)]
    gq = torch.tensor([2.0 ** -7], dtype=torch.float32, device=DEV)
    def step(k, b):
        reqat.quantize_kv4(k, mu, out=(b[0], b[1]), g_out=b[2])
        reqat.fakequant_kv4(k, mu, out=b[3], g_out=b[4])
        reqat.quantize_kv4(k, mu, tensor_scale=gq, out=(b[5], b[6]))
    k1, k2 = keys(1), keys(2)
    b1, b2 = bufs(), bufs()
    reqat.workspace(torch.device(DEV))
    step(k1, b1)
    torch.cuda.synchronize()
    ref = [t.clone() for t in b1]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(k1, b1)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(k1, b1)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in b1:
            t.fill_(0xA5) if t.dtype == torch.uint8 else t.fill_(float("nan"))
        step(k2, b2)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(b1, ref)):
            assert torch.equal(got.view(torch.uint8), want.view(torch.uint8)), \
                f"replay {rep}: kv4 output {i} differs from the eager step"
    log("kv4 graph replays match")


@pytest.mark.parametrize("M,N,K", [(16, 640, 4096), (5, 1536, 1024)])
def test_w4a16_graph_replays_match_eager(M, N, K):
    """W4A16 product (row-major and packed weights) captured and replayed.
    640 rows give 10 workgroups, so K is split and the FP32 partial sums meet
    in the workspace through the reduction kernel; 1536 rows are not split."""
    log(f"graph w4a16 M={M} N={N} K={K}")
    gen = torch.Generator().manual_seed(5 + M)
    w = (torch.randn(N, K, generator=gen) * 0.02).to(torch.bfloat16).to(DEV)
    wc, ws, _ = reqat.quantize(w, reqat.MXFP4)
    packed = reqat.pack_w4a16(wc, ws)
    x1 = (torch.randn(M, K, generator=gen) * 2.0).to(torch.bfloat16).to(DEV)
    x2 = (torch.randn(M, K, generator=gen) * 2.0).to(torch.bfloat16).to(DEV)
    nws = max(reqat.reqat_w4a16_workspace_bytes(M, N, K), 16)
    if N == 640:
        assert reqat.reqat_w4a16_workspace_bytes(M, N, K) > 0, "expected a split product"

    def bufs():
        return {"y": torch.empty((M, N), dtype=torch.bfloat16, device=DEV),
                "yp": torch.empty((M, N), dtype=torch.float32, device=DEV),
                "ws": torch.empty(nws, dtype=torch.uint8, device=DEV)}

    def step(x, b):
        reqat.gemm_w4a16(x, wc, ws, out_dtype=torch.bfloat16, out=b["y"], ws=b["ws"])
        reqat.gemm_w4a16_packed(x, packed, N, out_dtype=torch.float32, out=b["yp"], ws=b["ws"])

    b1, b2 = bufs(), bufs()
    step(x1, b1)
    torch.cuda.synchronize()
    ref = [b1["y"].clone(), b1["yp"].clone()]
    assert torch.equal(ref[0], ref[1].to(torch.bfloat16)), "packed and row-major products differ"
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(x1, b1)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(x1, b1)
    torch.cuda.synchronize()
    for rep in range(3):
        b1["y"].fill_(float("nan"))
        b1["yp"].fill_(float("nan"))
        b1["ws"].fill_(0xA5)
        step(x2, b2)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(b1["y"].view(torch.int16), ref[0].view(torch.int16)), f"replay {rep}: bf16 output differs"
        assert torch.equal(b1["yp"].view(torch.int32), ref[1].view(torch.int32)), f"replay {rep}: fp32 output differs"
    log("graph replays match")
