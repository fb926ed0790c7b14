"""GPU parity at the full workload sizes, in the launch configuration the
benchmark uses.  Quantize outputs of the full X and W are compared with the
oracle bit for bit; the GEMM is checked on sampled (m, n) outputs that the
oracle evaluates one by one (plus the corners), against
|Y - Yref| <= 1e-3 * sum_k |A^ B^|.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_15682_amd import reqat
from paper_2606_15682_amd import workloads as wl
from tests import indep

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def log(msg):
    print(msg, flush=True)


def _quant_both(w):
    fmt = reqat.NVFP4 if w.fmt == "nvfp4" else reqat.MXFP4
    ofmt = oracle.FMT_NVFP4 if fmt == reqat.NVFP4 else oracle.FMT_MXFP4
    x, wt = wl.make_x(w), wl.make_w(w)
    out = {}
    for name, t in (("x", x), ("w", wt)):
        c, s, g = reqat.quantize(t.to(DEV), fmt)
        torch.cuda.synchronize()
        bits = wl.bf16_bits(t)
        oc, os_, og = oracle.quantize(ofmt, bits)
        assert np.array_equal(s.cpu().numpy(), os_), "%s scales differ" % name
        assert np.array_equal(c.cpu().numpy(), oc), "%s codes differ" % name
        if fmt == reqat.NVFP4:
            assert float(g.cpu()[0]) == og
        out[name] = (c, s, g, oc, os_, og, bits)
        log("  %s quantize bit-exact (%d x %d)" % (name, t.shape[0], t.shape[1]))
    return fmt, ofmt, out


def _check_gemm(w, fmt, ofmt, q, out_dtype, npts=2000, seed=0):
    xc, xs, xg, oxc, oxs, oxg, _ = q["x"]
    wc, ws, wg, owc, ows, owg, _ = q["w"]
    y = torch.full((w.M, w.N), float("nan"), dtype=out_dtype, device=DEV)
    reqat.gemm(fmt, xc, xs, xg, wc, ws, wg, out_dtype=out_dtype, out=y)
    torch.cuda.synchronize()
    assert not torch.isnan(y).any().item(), "unwritten or NaN outputs"
    if w.M <= 64:
        # the packed decode image (the layout the bench streams): same product bit for bit
        yp = torch.full((w.M, w.N), float("nan"), dtype=out_dtype, device=DEV)
        reqat.gemm_packed(fmt, xc, xs, xg, reqat.pack_w4a4(wc, ws, fmt), w.N, wg, out_dtype=out_dtype, out=yp)
        torch.cuda.synchronize()
        iv = torch.int32 if out_dtype == torch.float32 else torch.int16
        assert torch.equal(y.view(iv), yp.view(iv)), "packed decode product differs"
        log("  packed decode image: same product bit for bit")
    rng = np.random.default_rng(seed)
    ms = np.concatenate([rng.integers(0, w.M, npts), [0, 0, w.M - 1, w.M - 1]])
    ns = np.concatenate([rng.integers(0, w.N, npts), [0, w.N - 1, 0, w.N - 1]])
    ref, aref = oracle.gemm_points(ofmt, oxc, oxs, oxg, owc, ows, owg, ms, ns)
    got = y[torch.from_numpy(ms).to(DEV), torch.from_numpy(ns).to(DEV)].float().cpu().numpy()
    got = got.astype(np.float64)
    if out_dtype == torch.float32:
        m = indep.gemm_error_metrics(got, ref, aref)
        log("  gemm fp32 M=%d N=%d K=%d %s" % (w.M, w.N, w.K, indep.format_metrics(m)))
        assert m["max_rel_sum"] <= 1e-3, m
        assert m["max_rel_sum"] <= indep.fp32_accumulation_bound(w.K), m
    else:
        rb = indep.bf16_values(oracle.bf16_from_double_array(ref))
        ulp = np.maximum(np.abs(rb), 2.0 ** -133) * 2.0 ** -7
        assert np.all(np.abs(got - rb) <= ulp + 1e-3 * aref)
    log("  gemm %s sampled parity ok (%d points)" % (out_dtype, len(ms)))


@pytest.mark.parametrize("idx", [1, 2, 3])
def test_fullsize_small_workloads(idx):
    w = wl.WORKLOADS[idx]
    log("full-size workload %d: %s" % (idx, w.name))
    fmt, ofmt, q = _quant_both(w)
    _check_gemm(w, fmt, ofmt, q, torch.float32, seed=idx)
    _check_gemm(w, fmt, ofmt, q, torch.bfloat16, seed=idx + 10)


def test_fullsize_14b_gate_up_nvfp4():
    w = wl.WORKLOADS[4]
    log("full-size workload 4: %s" % w.name)
    fmt, ofmt, q = _quant_both(w)
    _check_gemm(w, fmt, ofmt, q, torch.bfloat16, seed=4)
    _check_gemm(w, fmt, ofmt, q, torch.float32, seed=5, npts=1000)


def test_fullsize_14b_fakequant():
    """Fake-quant (QAT forward) of the full X and the full W (27648 x 5120), and
    the one-pass quantize + fake-quant the benchmark step runs on both, bit-exact
    over every element (W's computed g goes through the segment fix-up: 138,240
    segments of 64 blocks)."""
    w = wl.WORKLOADS[4]
    log("full-size fake-quant, workload 4")
    for name, t in (("x", wl.make_x(w)), ("w", wl.make_w(w))):
        y, g = reqat.fakequant(t.to(DEV), reqat.NVFP4)
        torch.cuda.synchronize()
        oy, og = oracle.fakequant(oracle.FMT_NVFP4, wl.bf16_bits(t))
        assert float(g.cpu()[0]) == og
        assert np.array_equal(wl.bf16_bits(y.cpu()), oy), "%s fake-quant differs" % name
        log("  %s fake-quant bit-exact" % name)
        # the one-pass quantize + fake-quant the benchmark step runs
        c, sc, y2, g2 = reqat.quantize_fakequant(t.to(DEV), reqat.NVFP4)
        torch.cuda.synchronize()
        oc, os_, og2 = oracle.quantize(oracle.FMT_NVFP4, wl.bf16_bits(t))
        assert float(g2.cpu()[0]) == og2 == og
        assert np.array_equal(sc.cpu().numpy(), os_) and np.array_equal(c.cpu().numpy(), oc)
        assert np.array_equal(wl.bf16_bits(y2.cpu()), oy), "%s fused fake-quant differs" % name
        log("  %s fused quantize + fake-quant bit-exact" % name)


def test_fullsize_7b_qkv_linear():
    """The fused linear call of the 7B-like QKV projection (2048 x 4608 x 3584,
    NVFP4, computed activation scale): the activation codes and scales it leaves
    in its workspace are the oracle's bit for bit, and the product meets the
    GEMM bar on sampled outputs (FP32 and bfloat16 out)."""
    w = wl.WORKLOADS[3]
    log("full-size linear, workload 3: %s" % w.name)
    x, wt = wl.make_x(w), wl.make_w(w)
    xb, wb = wl.bf16_bits(x), wl.bf16_bits(wt)
    oxc, oxs, oxg = oracle.quantize(oracle.FMT_NVFP4, xb)
    owc, ows, owg = oracle.quantize(oracle.FMT_NVFP4, wb)
    wc, ws_, wg = reqat.quantize(wt.to(DEV), reqat.NVFP4)
    torch.cuda.synchronize()
    assert np.array_equal(wc.cpu().numpy(), owc) and np.array_equal(ws_.cpu().numpy(), ows)
    rng = np.random.default_rng(33)
    ms = np.concatenate([rng.integers(0, w.M, 2000), [0, 0, w.M - 1, w.M - 1]])
    ns = np.concatenate([rng.integers(0, w.N, 2000), [0, w.N - 1, 0, w.N - 1]])
    ref, aref = oracle.gemm_points(oracle.FMT_NVFP4, oxc, oxs, oxg, owc, ows, owg, ms, ns)
    xd = x.to(DEV)
    for dt in (torch.float32, torch.bfloat16):
        ws = torch.full((reqat.reqat_linear_workspace_bytes(reqat.NVFP4, w.M, w.K),), 0xAB,
                        dtype=torch.uint8, device=DEV)
        y = torch.full((w.M, w.N), float("nan"), dtype=dt, device=DEV)
        _, g = reqat.linear(xd, reqat.NVFP4, wc, ws_, wg, out_dtype=dt, out=y, ws=ws)
        torch.cuda.synchronize()
        assert float(g.cpu()[0]) == oxg
        assert not torch.isnan(y).any().item(), "unwritten or NaN outputs"
        codes, scales = reqat.linear_workspace_views(ws, reqat.NVFP4, w.M, w.K)
        assert np.array_equal(codes.cpu().numpy(), oxc) and np.array_equal(scales.cpu().numpy(), oxs)
        got = y[torch.from_numpy(ms).to(DEV), torch.from_numpy(ns).to(DEV)].float().cpu().numpy()
        got = got.astype(np.float64)
        if dt == torch.float32:
            m = indep.gemm_error_metrics(got, ref, aref)
            log("  linear fp32 " + indep.format_metrics(m))
            assert m["max_rel_sum"] <= 1e-3
            assert m["max_rel_sum"] <= indep.fp32_accumulation_bound(w.K), m
        else:
            rb = indep.bf16_values(oracle.bf16_from_double_array(ref))
            ulp = np.maximum(np.abs(rb), 2.0 ** -133) * 2.0 ** -7
            assert np.all(np.abs(got - rb) <= ulp + 1e-3 * aref)
        log("  linear %s: workspace codes bit-exact, sampled product ok" % dt)


def test_fullsize_14b_gate_up_mxfp4():
    """The 14B-like gate/up shape (4096 x 27648 x 5120) in MXFP4: full quantize
    of X and W bit-exact, the product on sampled outputs (both output types)."""
    w = wl.WORKLOADS[10]
    log("full-size workload 10: %s" % w.name)
    fmt, ofmt, q = _quant_both(w)
    _check_gemm(w, fmt, ofmt, q, torch.bfloat16, seed=40)
    _check_gemm(w, fmt, ofmt, q, torch.float32, seed=41, npts=1000)


def test_fullsize_32b_down_mxfp4():
    w = wl.WORKLOADS[5]
    log("full-size workload 5: %s" % w.name)
    fmt, ofmt, q = _quant_both(w)
    _check_gemm(w, fmt, ofmt, q, torch.float32, seed=7, npts=1000)


def test_nvfp4_computed_scale_beyond_segment_table():
    """A tensor of more than 2^19 segments of 64 NVFP4 blocks (33000 x 16384
    bfloat16, 1.08 GB) takes the two-pass quantizer (absmax, then quantize).
    Values are clipped normals with one planted maximum, so the tensor amax is
    known exactly; sampled rows are compared with the oracle under that g."""
    R, C = 33000, 16384
    log("nvfp4 computed scale, %d x %d (two-pass)" % (R, C))
    gen = torch.Generator(device=DEV)
    gen.manual_seed(11)
    x = torch.randn((R, C), generator=gen, device=DEV, dtype=torch.float32).clamp_(-4.0, 4.0)
    x = x.to(torch.bfloat16)
    x[R // 3, 777] = 100.0
    c, s, g = reqat.quantize(x, reqat.NVFP4)
    torch.cuda.synchronize()
    og = oracle.nv_global_scale(100.0)
    assert float(g.cpu()[0]) == og
    rows = np.array([0, 1, R // 3, R // 2, R - 2, R - 1])
    idx = torch.from_numpy(rows).to(DEV)
    bits = wl.bf16_bits(x[idx].cpu())
    oc, os_, _ = oracle.quantize(oracle.FMT_NVFP4, bits, og)
    assert np.array_equal(s[idx].cpu().numpy(), os_)
    assert np.array_equal(c[idx].cpu().numpy(), oc)
    del x, c, s
    torch.cuda.empty_cache()


def test_fullsize_rotated_mxfp4_activations():
    """Block-rotated MXFP4 quantization of the full 32B-like down-proj activations
    (8192 x 27648, Student-t with outlier channels); rows are independent, so 48
    sampled rows plus the first and last are compared with the oracle bit for bit."""
    w = wl.WORKLOADS[5]
    log("full-size rotated mxfp4, workload 5 X")
    x = wl.make_x(w)
    signs = 0x6C8E9CF5
    c, s = reqat.quantize_rht(x.to(DEV), signs)
    y = reqat.fakequant_rht(x.to(DEV), signs)
    torch.cuda.synchronize()
    rows = np.concatenate([[0, w.M - 1], np.random.default_rng(5).choice(w.M, 48, replace=False)])
    bits = wl.bf16_bits(x)[rows]
    oc, os_ = oracle.quantize_mx_rht(bits, signs)
    idx = torch.from_numpy(rows).to(DEV)
    bad = np.argwhere(s[idx].cpu().numpy() != os_)
    assert bad.size == 0, ("scales differ", len(bad), bad[:4].tolist())
    bad = np.argwhere(c[idx].cpu().numpy() != oc)
    assert bad.size == 0, ("codes differ", len(bad), bad[:4].tolist())
    assert np.array_equal(wl.bf16_bits(y[idx].cpu()), oracle.fakequant_mx_rht(bits, signs))


@pytest.mark.parametrize("idx", [6, 7])
def test_fullsize_w4a16_decode(idx):
    """W4A16 decode shapes at full size: weights quantized to MXFP4 by the oracle,
    the product checked on sampled outputs (plus corners) against the FP64 oracle,
    and the product from the packed weight image equal to it bit for bit."""
    w = wl.WORKLOADS[idx]
    log("full-size W4A16 workload %d: %s" % (idx, w.name))
    xb, wb = wl.bf16_bits(wl.make_x(w)), wl.bf16_bits(wl.make_w(w))
    wc, ws, _ = oracle.quantize(oracle.FMT_MXFP4, wb)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    xt, wct, wst = wl.from_bits(xb).to(DEV), t(wc), t(ws)
    y = reqat.gemm_w4a16(xt, wct, wst, out_dtype=torch.float32)
    # the packed weight image (the layout the bench streams): same result bit for bit
    yp = reqat.gemm_w4a16_packed(xt, reqat.pack_w4a16(wct, wst), w.N, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int32), yp.view(torch.int32)), "packed W4A16 product differs"
    rng = np.random.default_rng(idx)
    ms = np.concatenate([rng.integers(0, w.M, 2000), [0, 0, w.M - 1, w.M - 1]])
    ns = np.concatenate([rng.integers(0, w.N, 2000), [0, w.N - 1, 0, w.N - 1]])
    ref, aref = oracle.gemm_w4a16_points(xb, wc, ws, ms, ns)
    got = y.cpu().numpy().astype(np.float64)[ms, ns]
    m = indep.gemm_error_metrics(got, ref, aref)
    log("  w4a16 fp32 M=%d N=%d K=%d %s" % (w.M, w.N, w.K, indep.format_metrics(m)))
    assert m["max_rel_sum"] <= 1e-3, m
    assert m["max_rel_sum"] <= indep.fp32_accumulation_bound(w.K), m


def test_fullsize_kv4_keys_14b_prefill():
    """KV4 of the prefill keys of a 14B-like layer (4096 tokens x 8 KV heads x 128
    channels, Gaussian with outlier channels) with a calibrated channel shift,
    bit-exact against the oracle over the whole tensor."""
    w = wl.WORKLOADS[4]
    log("full-size kv4 keys 4096 x 1024")
    kb = wl.bf16_bits(wl.make_x(w))[:, :1024].copy()
    shift = np.random.default_rng(21).normal(0.0, 0.5, 1024).astype(np.float32)
    oc, os_, og = oracle.kv4_quantize(kb, shift)
    c, s, g = reqat.quantize_kv4(wl.from_bits(kb).to(DEV), torch.from_numpy(shift).to(DEV))
    torch.cuda.synchronize()
    assert float(g.cpu()[0]) == np.float32(og)
    assert np.array_equal(s.cpu().numpy(), os_) and np.array_equal(c.cpu().numpy(), oc)


def test_fullsize_kv4_keys():
    """KV4 quantization of the full 32768 x 1024 key workload (shift = the
    channel offsets), computed and given tensor scales, bit-exact; fake-quant
    on a 4096-row slice."""
    w = wl.WORKLOADS[9]
    log("full-size KV4 keys: %s" % w.name)
    k, mu = wl.make_keys(w)
    kb = wl.bf16_bits(k)
    kd, mud = k.to(DEV), mu.to(DEV)
    c, s, g = reqat.quantize_kv4(kd, mud)
    torch.cuda.synchronize()
    oc, os_, og = oracle.kv4_quantize(kb, mu.numpy())
    assert float(g.cpu()[0]) == og
    assert np.array_equal(s.cpu().numpy(), os_) and np.array_equal(c.cpu().numpy(), oc)
    log("  computed g bit-exact")
    gg = torch.tensor([og * 0.75], dtype=torch.float32, device=DEV)
    c2, s2, _ = reqat.quantize_kv4(kd, mud, tensor_scale=gg)
    torch.cuda.synchronize()
    oc2, os2, _ = oracle.kv4_quantize(kb, mu.numpy(), float(np.float32(og * 0.75)))
    assert np.array_equal(s2.cpu().numpy(), os2) and np.array_equal(c2.cpu().numpy(), oc2)
    log("  given g bit-exact")
    y, _ = reqat.fakequant_kv4(kd[:4096].contiguous(), mud)
    torch.cuda.synchronize()
    oy, _ = oracle.kv4_fakequant(kb[:4096], mu.numpy())
    assert np.array_equal(wl.bf16_bits(y.cpu()), oy)
    log("  fake-quant bit-exact")
