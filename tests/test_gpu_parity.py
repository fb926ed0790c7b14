"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Codes, scales, global scales and fake-quant outputs must match bit for bit;
GEMM outputs must satisfy |Y - Yref| <= 1e-3 * sum_k |A^ B^| (FP32 output;
Yref is the FP64 product of the exactly dequantized operands), and a bf16
output must additionally be within one bf16 ulp of round(Yref).  Outputs are
pre-filled with two different poison patterns, so an element the kernel does
not write, or a run-to-run difference, fails the comparison.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2606_15682_amd import reqat
from paper_2606_15682_amd import workloads as wl
from tests import indep

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
NV, MX = reqat.NVFP4, reqat.MXFP4
GEMM_TOL = 1e-3


def log(msg):
    print(msg, flush=True)


def gpu_quant(fmt, xb, g=None, poison=0, ldx_pad=0):
    R, C = xb.shape
    B = reqat.BLOCK[fmt]
    if ldx_pad:
        big = np.zeros((R, C + ldx_pad), np.uint16)
        big[:, :C] = xb
        xt = wl.from_bits(big).to(DEV)[:, :C]
    else:
        xt = wl.from_bits(xb).to(DEV)
    codes = torch.full((R, C // 2), poison, dtype=torch.uint8, device=DEV)
    scales = torch.full((R, C // B), poison, dtype=torch.uint8, device=DEV)
    gt = None if (g is None or fmt == MX) else torch.tensor([g], dtype=torch.float32, device=DEV)
    _, _, gg = reqat.quantize(xt, fmt, tensor_scale=gt, out=(codes, scales))
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy(), (1.0 if gg is None else float(gg.cpu()[0]))


def gpu_fakequant(fmt, xb, g=None, poison=0x7FFF):
    R, C = xb.shape
    xt = wl.from_bits(xb).to(DEV)
    y = wl.from_bits(np.full((R, C), poison, np.uint16)).to(DEV)
    gt = None if (g is None or fmt == MX) else torch.tensor([g], dtype=torch.float32, device=DEV)
    _, gg = reqat.fakequant(xt, fmt, tensor_scale=gt, out=y)
    torch.cuda.synchronize()
    return wl.bf16_bits(y.cpu()), (1.0 if gg is None else float(gg.cpu()[0]))


def assert_quant_parity(fmt, xb, g=None, ldx_pad=0):
    oc, os_, og = oracle.quantize(fmt, xb, g)
    for poison in (0x00, 0xFF):
        c, s, gg = gpu_quant(fmt, xb, g, poison, ldx_pad)
        if fmt == NV:
            assert gg == np.float32(og), (gg, og)
        bad = np.argwhere(s != os_)
        assert bad.size == 0, ("scales differ", bad[:4], s[tuple(bad[0])], os_[tuple(bad[0])])
        bad = np.argwhere(c != oc)
        assert bad.size == 0, ("codes differ", bad[:4], c[tuple(bad[0])], oc[tuple(bad[0])])


def assert_fq_parity(fmt, xb, g=None):
    oy, og = oracle.fakequant(fmt, xb, g)
    for poison in (0x7FFF, 0x0000):
        y, gg = gpu_fakequant(fmt, xb, g, poison)
        bad = np.argwhere(y != oy)
        assert bad.size == 0, ("fake-quant differs", bad[:4], hex(y[tuple(bad[0])]), hex(oy[tuple(bad[0])]))
    assert_both_parity(fmt, xb, g, oy=oy)


def assert_both_parity(fmt, xb, g=None, oy=None):
    """The one-pass quantize + fake-quant entry point: codes, scales, g and y all
    equal the oracle's quantize and fake-quant outputs."""
    R, C = xb.shape
    B = reqat.BLOCK[fmt]
    oc, os_, og = oracle.quantize(fmt, xb, g)
    if oy is None:
        oy, _ = oracle.fakequant(fmt, xb, g)
    xt = wl.from_bits(xb).to(DEV)
    gt = None if (g is None or fmt == MX) else torch.tensor([g], dtype=torch.float32, device=DEV)
    for pc, py in ((0x00, 0x7FFF), (0xFF, 0x0000)):
        codes = torch.full((R, C // 2), pc, dtype=torch.uint8, device=DEV)
        scales = torch.full((R, C // B), pc, dtype=torch.uint8, device=DEV)
        y = wl.from_bits(np.full((R, C), py, np.uint16)).to(DEV)
        _, _, _, gg = reqat.quantize_fakequant(xt, fmt, tensor_scale=gt, out=(codes, scales, y))
        torch.cuda.synchronize()
        if fmt == NV:
            assert float(gg.cpu()[0]) == np.float32(og)
        assert np.array_equal(scales.cpu().numpy(), os_), "fused: scales differ"
        assert np.array_equal(codes.cpu().numpy(), oc), "fused: codes differ"
        yb = wl.bf16_bits(y.cpu())
        bad = np.argwhere(yb != oy)
        assert bad.size == 0, ("fused fake-quant differs", bad[:4], hex(yb[tuple(bad[0])]), hex(oy[tuple(bad[0])]))


def _rand(R, C, seed, dist="normal", std=1.0, outliers=0):
    t = wl.random_bf16(R, C, seed, std, dist)
    xb = wl.bf16_bits(t).copy()
    if outliers:
        rng = np.random.default_rng(seed + 1)
        idx = rng.choice(C, outliers, replace=False)
        xb[:, idx] = indep.to_bf16_bits(indep.bf16_values(xb[:, idx]) * 20.0)
    return xb


SHAPES = [(16, 256), (37, 224), (1, 32), (129, 512), (300, 96)]


@pytest.mark.parametrize("fmt", [NV, MX])
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("dist", ["normal", "student_t"])
def test_quantize_parity_random(fmt, shape, dist):
    R, C = shape
    log("quantize parity fmt=%d shape=%s dist=%s" % (fmt, shape, dist))
    xb = _rand(R, C, 100 + R + C, dist, outliers=max(1, C // 100))
    assert_quant_parity(fmt, xb)
    assert_fq_parity(fmt, xb)


@pytest.mark.parametrize("g", [2.0 ** -7, 1.0, 0.0123456789, 3.0, 1e-30, 2.0 ** -140])
def test_nvfp4_given_global_scale(g):
    log("NVFP4 given g=%r" % g)
    xb = _rand(33, 256, 7, "student_t", outliers=3)
    g = float(np.float32(g))
    assert_quant_parity(NV, xb, g)
    assert_fq_parity(NV, xb, g)


def _ramp(R, C, seed, step):
    """Normal values with row r scaled by 2^(-step*r): segments of very different
    magnitude, so a computed g differs from most segments' own reference and the
    smallest rows fall into E4M3-subnormal block scales."""
    xb = wl.bf16_bits(wl.random_bf16(R, C, seed)).copy()
    return indep.to_bf16_bits(indep.bf16_values(xb) * (2.0 ** (-step * np.arange(R)))[:, None])


@pytest.mark.parametrize("shape,step", [((40, 1040), 1.5), ((48, 1024), 1.0), ((7, 4096), 9.0),
                                        ((300, 96), 0.25), ((80, 1040), 1.5), ((96, 1024), 1.0),
                                        ((20, 4096), 9.0), ((1000, 96), 0.1)])
def test_nvfp4_computed_scale_wide_range(shape, step):
    """NVFP4 with a computed g over tensors whose rows span many binades.  Up to
    2^16 elements (the first four shapes) the single-launch path computes g
    first; beyond (the last four), the one-pass quantizer must lower the scale
    exponents of rows quantized under a smaller reference and re-quantize
    blocks whose scale leaves the normal range."""
    R, C = shape
    log("nvfp4 computed scale, wide range shape=%s step=%g" % (shape, step))
    xb = _ramp(R, C, 31 + R, step)
    assert_quant_parity(NV, xb)
    assert_fq_parity(NV, xb)
    assert_quant_parity(NV, xb, ldx_pad=24)
    xs = xb.copy()
    xs[R // 2, 3] = 0x7FC0                       # NaN block
    xs[R - 1, :] = 0                             # zero row
    xs[1, C - 1] = 0xFF80                        # -Inf in the last block of a row
    assert_quant_parity(NV, xs)
    assert_fq_parity(NV, xs)


# ------------------------------------------------------- block-rotated MXFP4

def gpu_quant_rht(xb, signs, poison=0, ldx_pad=0):
    R, C = xb.shape
    if ldx_pad:
        big = np.zeros((R, C + ldx_pad), np.uint16)
        big[:, :C] = xb
        xt = wl.from_bits(big).to(DEV)[:, :C]
    else:
        xt = wl.from_bits(xb).to(DEV)
    codes = torch.full((R, C // 2), poison, dtype=torch.uint8, device=DEV)
    scales = torch.full((R, C // 32), poison, dtype=torch.uint8, device=DEV)
    reqat.quantize_rht(xt, signs, out=(codes, scales))
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy()


def assert_rht_parity(xb, signs, ldx_pad=0):
    oc, os_ = oracle.quantize_mx_rht(xb, signs)
    for poison in (0x00, 0xFF):
        c, s = gpu_quant_rht(xb, signs, poison, ldx_pad)
        bad = np.argwhere(s != os_)
        assert bad.size == 0, ("scales differ", bad[:4], s[tuple(bad[0])], os_[tuple(bad[0])])
        bad = np.argwhere(c != oc)
        assert bad.size == 0, ("codes differ", bad[:4], c[tuple(bad[0])], oc[tuple(bad[0])])
    oy = oracle.fakequant_mx_rht(xb, signs)
    for poison in (0x7FFF, 0x0000):
        y = wl.from_bits(np.full(xb.shape, poison, np.uint16)).to(DEV)
        reqat.fakequant_rht(wl.from_bits(xb).to(DEV), signs, out=y)
        torch.cuda.synchronize()
        yb = wl.bf16_bits(y.cpu())
        bad = np.argwhere(yb != oy)
        assert bad.size == 0, ("rotated fake-quant differs", bad[:4], hex(yb[tuple(bad[0])]), hex(oy[tuple(bad[0])]))


@pytest.mark.parametrize("shape", [(16, 256), (37, 224), (1, 32), (129, 512), (300, 96)])
@pytest.mark.parametrize("signs", [0x0, 0xFFFFFFFF, 0x9E3779B9])
def test_rotated_mxfp4_parity_random(shape, signs):
    R, C = shape
    log("rotated mxfp4 parity shape=%s signs=%08x" % (shape, signs))
    xb = _rand(R, C, 300 + R + C, "student_t", outliers=max(1, C // 100))
    assert_rht_parity(xb, signs)


@pytest.mark.parametrize("order", ["sorted", "shuffled"])
def test_rotated_mxfp4_exhaustive_bf16_patterns(order):
    """Every bfloat16 pattern (NaN, Inf, subnormals, overflowing sums) through the rotation."""
    log("rotated mxfp4 exhaustive %s" % order)
    pats = np.arange(65536, dtype=np.uint16)
    if order == "shuffled":
        pats = np.random.default_rng(11).permutation(pats)
    assert_rht_parity(pats.reshape(64, 1024), 0xA5A5F00F)


def test_rotated_mxfp4_tiny_and_strided():
    log("rotated mxfp4 tiny scales, strided rows")
    xb = _ramp(24, 320, 77, 6.0)                 # rows down to 2^-138: E8M0 byte 0 and FP32 subnormals
    assert_rht_parity(xb, 0x13579BDF)
    assert_rht_parity(_rand(45, 320, 9, "normal"), 0x2468ACE0, ldx_pad=40)


def _near_threshold_rows(signs):
    """Blocks whose scale or first code hinges on bits up to ~2^-128 below the leading
    one (each threshold from both sides): neither FP32 nor FP64 evaluation decides them,
    and with 12 or 16 slices the inputs span more than 40 binades (the wide-integer path)."""
    rows = []
    cases = [(Fraction(6), 0, None), (Fraction(6), 50, None), (Fraction(5), -3, None),
             (Fraction(7, 2), 10, None), (Fraction(1, 4), 2, 9), (Fraction(3, 4), -20, 9),
             (Fraction(5, 4), 0, 9), (Fraction(7, 4), 5, 9), (Fraction(5, 2), -7, 9)]
    for t, e, big in cases:
        for chunks in (3, 4, 6, 12, 16):
            for above in (False, True):
                bigv = None if big is None else Fraction(big) * Fraction(2) ** e
                rows.append(indep.rht_near_threshold_block(t, e, above, chunks, signs, bigv))
    return np.concatenate(rows).reshape(-1, 64) if len(rows) % 2 == 0 else np.concatenate(rows[:-1]).reshape(-1, 64)


@pytest.mark.parametrize("signs", [0, 0x13579BDF])
def test_rotated_mxfp4_decisions_below_fp32_and_fp64_precision(signs):
    """The exact rotation on blocks the FP32 fast path cannot decide: near-threshold
    blocks (FP64 and wide-integer paths), small-integer and constant blocks (exact zero
    outputs), and a mix of them with ordinary blocks in the same waves."""
    log("rotated mxfp4 near-threshold signs=%08x" % signs)
    near = _near_threshold_rows(signs)
    assert_rht_parity(near, signs)
    rng = np.random.default_rng(signs & 0xFFFF)
    ints = indep.to_bf16_bits(rng.integers(-40, 41, (96, 256)).astype(np.float64))
    const = np.repeat(indep.to_bf16_bits(rng.normal(0, 1, 96)), 256).reshape(96, 256)
    mixed = _rand(96, 256, 4, "student_t", outliers=2)
    mixed[::3] = ints[::3]
    mixed[1::7] = const[1::7]
    assert_rht_parity(np.concatenate([ints, const, mixed]), signs)
    spread = mixed.copy()
    spread[:, ::5] = indep.to_bf16_bits(indep.bf16_values(spread[:, ::5]) * 2.0 ** -90)   # wide spreads
    assert_rht_parity(spread, signs)


# ------------------------------------------------------------------ KV4

def assert_kv4_parity(xb, shift=None, g=None, ldx_pad=0):
    R, C = xb.shape
    oc, os_, og = oracle.kv4_quantize(xb, shift, g)
    oy, _ = oracle.kv4_fakequant(xb, shift, g)
    if ldx_pad:
        big = np.zeros((R, C + ldx_pad), np.uint16)
        big[:, :C] = xb
        xt = wl.from_bits(big).to(DEV)[:, :C]
    else:
        xt = wl.from_bits(xb).to(DEV)
    sh = None if shift is None else torch.from_numpy(np.ascontiguousarray(shift, np.float32)).to(DEV)
    gt = None if g is None else torch.tensor([g], dtype=torch.float32, device=DEV)
    for poison in (0x00, 0xFF):
        codes = torch.full((R, C // 2), poison, dtype=torch.uint8, device=DEV)
        scales = torch.full((R, C // 16), poison, dtype=torch.uint8, device=DEV)
        _, _, gg = reqat.quantize_kv4(xt, sh, tensor_scale=gt, out=(codes, scales))
        torch.cuda.synchronize()
        assert float(gg.cpu()[0]) == np.float32(og)
        s_, c_ = scales.cpu().numpy(), codes.cpu().numpy()
        bad = np.argwhere(s_ != os_)
        assert bad.size == 0, ("kv4 scales differ", bad[:4], s_[tuple(bad[0])], os_[tuple(bad[0])])
        bad = np.argwhere(c_ != oc)
        assert bad.size == 0, ("kv4 codes differ", bad[:4], c_[tuple(bad[0])], oc[tuple(bad[0])])
    y = wl.from_bits(np.full((R, C), 0x7FFF, np.uint16)).to(DEV)
    reqat.fakequant_kv4(xt, sh, tensor_scale=gt, out=y)
    torch.cuda.synchronize()
    yb = wl.bf16_bits(y.cpu())
    bad = np.argwhere(yb != oy)
    assert bad.size == 0, ("kv4 fake-quant differs", bad[:4], hex(yb[tuple(bad[0])]), hex(oy[tuple(bad[0])]))


@pytest.mark.parametrize("shape", [(16, 1024), (37, 96), (1, 16), (300, 512)])
@pytest.mark.parametrize("shifted", [False, True])
def test_kv4_parity_random(shape, shifted):
    R, C = shape
    log("kv4 parity shape=%s shifted=%s" % (shape, shifted))
    xb = _rand(R, C, 500 + R + C, "normal", outliers=max(1, C // 64))
    shift = np.random.default_rng(R + C).normal(0.0, 1.5, C).astype(np.float32) if shifted else None
    assert_kv4_parity(xb, shift)
    assert_kv4_parity(xb, shift, g=0.0123456789)
    assert_kv4_parity(xb, shift, g=2.0 ** -6)


def test_kv4_exhaustive_patterns_and_specials():
    log("kv4 exhaustive bf16 patterns with a shift, specials, strided rows")
    pats = np.random.default_rng(13).permutation(np.arange(65536, dtype=np.uint16)).reshape(64, 1024)
    shift = np.random.default_rng(14).normal(0.0, 3.0, 1024).astype(np.float32)
    shift[::7] = 0.0
    assert_kv4_parity(pats, None)
    assert_kv4_parity(pats, shift)
    x = np.zeros((5, 32), np.uint16)
    x[0, 3] = 0x7FC0
    x[1, :] = 0x8000
    x[2, :16] = 0x7F7F
    x[3, 16:] = 0x0001
    x[4, :] = 0x3F80
    sh = np.zeros(32, np.float32)
    sh[:16] = -3.0e38                     # 0x7F7F - (-3e38) overflows FP32: a NaN block
    assert_kv4_parity(x, sh)
    assert_kv4_parity(x, None, g=2.0 ** -12)          # caller's g too small: 448 and saturation
    # FP32 element thresholds (power-of-two g up to 2^100): the smallest g (E4M3
    # subnormal scales times 2^-126 are FP32 subnormals) and the largest; above
    # 2^100 and for other g the FP64 comparisons run
    for g in (2.0 ** -126, 2.0 ** 100, 2.0 ** 101, 3.0 * 2.0 ** 90):
        assert_kv4_parity(pats[:8], shift, g=g)
    tiny = np.arange(1, 1025, dtype=np.uint16).reshape(32, 32)       # BF16 subnormals and the smallest normals
    tiny[1] = 1 + np.arange(32) % 3                                  # E4M3 subnormal scale bytes
    tiny[3] = 1
    tiny[5] = 1 + np.arange(32) % 6
    tiny[::2] |= 0x8000
    assert_kv4_parity(tiny, None)                                   # computed g = 2^-126: subnormal S
    assert_kv4_parity(tiny, None, g=2.0 ** -126)
    assert_kv4_parity(_rand(45, 320, 19, "student_t"), np.linspace(-2, 2, 320).astype(np.float32), ldx_pad=24)


@pytest.mark.parametrize("shifted", [False, True])
def test_kv4_one_pass_segments(shifted):
    """A computed g runs one pass under per-segment reference scales (64 blocks
    = 4 rows of 256 channels here) and a fix-up.  Segment k is scaled by
    2^-(3k mod 41), so the fix-up lowers some segments' scale exponents and
    re-quantizes the blocks of others whose scales would leave the normal E4M3
    range; plus an all-zero segment, a segment of NaN blocks whose finite
    elements still count for g, and a final partial segment (2080 blocks)."""
    log("kv4 one-pass segments shifted=%s" % shifted)
    R, C = 130, 256
    v = indep.bf16_values(_rand(R, C, 77, "student_t"))
    for k in range(R // 4 + 1):
        v[4 * k:4 * k + 4] *= 2.0 ** -(3 * k % 41)
    v[8:12] = 0.0                                          # an all-zero segment
    v[20:24, ::16] = np.nan                                # every block of this segment has a NaN
    v[21, 5] = 300.0                                       # a finite element of a NaN block sets g
    xb = indep.to_bf16_bits(v)
    shift = np.random.default_rng(5).normal(0.0, 0.5, C).astype(np.float32) if shifted else None
    assert_kv4_parity(xb, shift)


def _kv4_midpoint_targets():
    """FP32 values at and next to the E1M2 rounding midpoints.  Block b sets
    its amax to 7 H (H = s g / 2 for the scale s it gets, any of the eight
    E4M3 mantissas), the other 15 elements are +-((k + 1/2) H + j ulp),
    k = 0..6, j = -2..2: exact ties and values one or two FP32 ulps away."""
    vals = []
    combos = [(k, j) for k in range(7) for j in range(-2, 3)]
    for m in range(8, 16):
        for e in (-9, -3, 0, 5):
            H = np.float32(m / 8.0 * 2.0 ** e)
            for b0 in range(0, len(combos), 15):
                blk = [np.float32(7.0) * H]
                for i, (k, j) in enumerate(combos[b0:b0 + 15]):
                    t = np.float32((k + 0.5) * H)
                    for _ in range(abs(j)):
                        t = np.nextafter(t, np.float32(np.inf if j > 0 else -np.inf), dtype=np.float32)
                    blk.append(-t if i % 2 else t)
                blk += [np.float32(0.0)] * (16 - len(blk))
                vals += blk
    return np.array(vals, np.float32)


@pytest.mark.parametrize("g", [None, 1.0, 2.0 ** -3])
def test_kv4_rounding_near_midpoints(g):
    """d = x - shift with x = +-0 makes d any FP32 value, so the elements sit
    exactly on, or one or two ulps beside, the midpoints between codes."""
    log("kv4 near-midpoint rounding g=%s" % g)
    t = _kv4_midpoint_targets()
    C = t.size
    x = np.zeros((3, C), np.uint16)
    x[1] = 0x8000
    x[2] = indep.to_bf16_bits(np.random.default_rng(3).normal(0.0, 2.0 ** -12, C))
    assert_kv4_parity(x, -t, g=g)
    wide = np.zeros((2, 4224), np.uint16)                      # shift read from global memory (> 4096 channels)
    assert_kv4_parity(wide, -np.resize(t, 4224), g=g)


@pytest.mark.parametrize("g", [2.0 ** -6, 0.0123456789])
def test_kv4_fakequant_in_place(g):
    """KV4 fake-quant in place (y is x) with a given g, as the header allows:
    each block is read once before its values are written (FP32 element path
    for the power-of-two g, FP64 for the other)."""
    log("kv4 fake-quant in place g=%r" % g)
    xb = _rand(37, 512, 78, "normal", outliers=4)
    shift = np.random.default_rng(9).normal(0.0, 1.0, 512).astype(np.float32)
    g = float(np.float32(g))
    oy, _ = oracle.kv4_fakequant(xb, shift, g)
    xt = wl.from_bits(xb).to(DEV)
    reqat.fakequant_kv4(xt, torch.from_numpy(shift).to(DEV), tensor_scale=torch.tensor([g], dtype=torch.float32,
                                                                                      device=DEV), out=xt)
    torch.cuda.synchronize()
    assert np.array_equal(wl.bf16_bits(xt.cpu()), oy)


def test_kv4_empty_writes_unit_scale():
    log("kv4 empty")
    x = torch.empty((0, 128), dtype=torch.bfloat16, device=DEV)
    _, _, g = reqat.quantize_kv4(x, out=(torch.empty((0, 64), dtype=torch.uint8, device=DEV),
                                         torch.empty((0, 8), dtype=torch.uint8, device=DEV)))
    torch.cuda.synchronize()
    assert float(g.cpu()[0]) == 1.0


# ------------------------------------------------------------------ SEM loss

def run_sem_case(T, V, seed, lam=0.5, eps=1e-6, std=3.0):
    rng = np.random.default_rng(seed)
    zb = indep.to_bf16_bits(rng.normal(0.0, std, (T, V)))
    tg = rng.integers(0, V, T).astype(np.int32)
    H, nll, lse = oracle.sem_row_stats(zb, tg)
    L, l_sft, l_ent, w = oracle.sem_loss(H, nll, lam, eps)
    zt = wl.from_bits(zb).to(DEV)
    tt = torch.from_numpy(tg).to(DEV)
    loss, stats, weights = reqat.sem_loss(zt, tt, lam, eps)
    torch.cuda.synchronize()
    st = stats.cpu().numpy().astype(np.float64)
    # FP32 sums of about V / 256 terms per thread and exp2 of arguments rounded
    # once: errors of order 1e-6; the bounds below leave two orders of margin
    for got, ref in ((st[:, 0], H), (st[:, 1], nll), (st[:, 2], lse)):
        assert np.all(np.abs(got - ref) <= 1e-4 * (1 + np.abs(ref))), float(np.max(np.abs(got - ref)))
    wg = weights.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(wg - w) <= 1e-3), float(np.max(np.abs(wg - w)))
    lg = loss.cpu().numpy().astype(np.float64)
    for got, ref in ((lg[0], L), (lg[1], l_sft), (lg[2], l_ent)):
        assert abs(got - ref) <= 1e-4 * (1 + abs(ref)), (got, ref)
    # backward, with the GPU's own weights (the weights are an input of the gradient)
    gref = oracle.sem_grad(zb, tg, H, lse, wg, lam, scale=1.0)
    z = indep.bf16_values(zb)
    p = np.exp(z - lse[:, None])
    logp = z - lse[:, None]
    size = (p + lam * wg[:, None] * p * (np.abs(logp) + H[:, None])) / T
    size[np.arange(T), tg] += 1.0 / T
    for dt, ulp in ((torch.float32, 0.0), (torch.bfloat16, 2.0 ** -8)):
        g = reqat.sem_loss_backward(zt, tt, stats, weights, lam, 1.0, out_dtype=dt)
        torch.cuda.synchronize()
        gg = g.float().cpu().numpy().astype(np.float64)
        err = np.abs(gg - gref)
        assert np.all(err <= 2e-3 * size + ulp * np.abs(gref) + 1e-30), float(np.max(err / (size + 1e-30)))


@pytest.mark.parametrize("T,V", [(1, 64), (7, 1000), (64, 4096), (300, 2048), (4, 152064)])
def test_sem_loss_parity(T, V):
    log("sem loss T=%d V=%d" % (T, V))
    run_sem_case(T, V, T + V)


def _tau_from_entropies(H, T):
    """The 75th percentile the batch kernel defines, from its own FP32 entropies:
    linear interpolation at q = 0.75 (T - 1) between the order statistics at
    floor(q) and floor(q) + 1, in FP64, rounded to FP32."""
    hs = np.sort(H.astype(np.float32)).astype(np.float64)
    q = 0.75 * (T - 1)
    lo = int(q)
    hi = min(lo + 1, T - 1)
    return np.float32(hs[lo] + (q - lo) * (hs[hi] - hs[lo]))


@pytest.mark.parametrize("T,dup", [(4096, 1), (4097, 37), (1000, 1000), (8192, 5), (8193, 3), (9001, 1)])
def test_sem_batch_order_statistics_exact(T, dup):
    """tau (loss[3]) equals, bit for bit, the interpolated 75th percentile of the
    kernel's own entropies: batches held in registers (T <= 8192) and larger
    ones, distinct entropies and runs of equal ones (rows repeated dup times,
    so both order statistics can fall in one run or straddle two)."""
    log("sem batch order statistics T=%d dup=%d" % (T, dup))
    rng = np.random.default_rng(T + dup)
    V = 64
    base = indep.to_bf16_bits(rng.normal(0.0, 2.0, (-(-T // dup), V)))
    zb = np.repeat(base, dup, axis=0)[:T]
    tg = rng.integers(0, V, T).astype(np.int32)
    loss, stats, _ = reqat.sem_loss(wl.from_bits(zb).to(DEV), torch.from_numpy(tg).to(DEV), 0.5, 1e-6)
    torch.cuda.synchronize()
    H = stats.cpu().numpy()[:, 0]
    assert np.float32(loss.cpu().numpy()[3]) == _tau_from_entropies(H, T)


def test_sem_loss_low_entropy_rows():
    log("sem loss with near-deterministic rows")
    run_sem_case(33, 1024, 7, std=12.0)           # peaked softmax rows: entropies near zero


def test_qat_autograd_functions():
    """The QAT forward (fake-quant) with the straight-through backward, and the
    SEM loss as an autograd function: gradients reach the inputs unchanged /
    as the backward kernel computes them."""
    log("QAT autograd: fake-quant STE and SEM loss")
    x = wl.from_bits(_rand(8, 64, 71, "normal")).to(DEV).requires_grad_(True)
    y = reqat.FakeQuantSTE.apply(x, NV)
    oy, _ = oracle.fakequant(NV, wl.bf16_bits(x.detach().cpu()))
    assert np.array_equal(wl.bf16_bits(y.detach().cpu()), oy)
    gy = torch.randn_like(y)
    y.backward(gy)
    assert torch.equal(x.grad, gy)
    rng = np.random.default_rng(72)
    z = wl.from_bits(indep.to_bf16_bits(rng.normal(0, 2, (16, 512)))).to(DEV).requires_grad_(True)
    t = torch.from_numpy(rng.integers(0, 512, 16).astype(np.int32)).to(DEV)
    loss = reqat.SemLoss.apply(z, t, 0.5)
    loss.backward()
    _, stats, weights = reqat.sem_loss(z.detach(), t, 0.5)
    g = reqat.sem_loss_backward(z.detach(), t, stats, weights, 0.5, 1.0, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(z.grad, g)


@pytest.mark.parametrize("fmt", [NV, MX])
def test_strided_rows(fmt):
    log("strided rows fmt=%d" % fmt)
    xb = _rand(45, 320, 9, "normal")
    assert_quant_parity(fmt, xb, ldx_pad=40)


@pytest.mark.parametrize("fmt", [NV, MX])
@pytest.mark.parametrize("order", ["sorted", "shuffled"])
def test_exhaustive_bf16_patterns(fmt, order):
    """Every bfloat16 bit pattern (NaN/Inf make NaN blocks when shuffled in)."""
    log("exhaustive bf16 fmt=%d order=%s" % (fmt, order))
    allp = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    if order == "sorted":
        v = indep.bf16_values(allp)
        allp = allp[np.isfinite(v)]
        allp = allp[np.argsort(np.abs(indep.bf16_values(allp)), kind="stable")]
        allp = allp[: (allp.size // 512) * 512]
    else:
        allp = np.random.default_rng(3).permutation(allp)
    xb = allp.reshape(-1, 512)
    assert_quant_parity(fmt, xb)
    assert_fq_parity(fmt, xb)
    if fmt == NV:
        for g in (2.0 ** -20, 0.3):
            assert_quant_parity(NV, xb, float(np.float32(g)))
            assert_fq_parity(NV, xb, float(np.float32(g)))


@pytest.mark.parametrize("fmt", [NV, MX])
def test_exact_ties_and_neighbours(fmt):
    """Blocks whose elements sit exactly on rounding midpoints (and one bf16
    step either side), for many scales across the exponent range."""
    log("ties fmt=%d" % fmt)
    B = reqat.BLOCK[fmt]
    rows = []
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    e4 = indep.e4m3_table()
    for e in range(-130, 126, 3):
        if fmt == MX:
            S = 2.0 ** e
        else:
            S = e4[(e * 7) % 0x7E + 1] * 2.0 ** (e // 2)
        vals = np.concatenate([[6.0 * S], mids * S, -mids * S])
        vals = np.resize(vals, B)
        b = indep.to_bf16_bits(vals)
        rows.append(b)
        rows.append(np.where(b & 0x7FFF, b + 1, b).astype(np.uint16))
        rows.append(np.where(b & 0x7FFF, b - 1, b).astype(np.uint16))
    xb = np.concatenate(rows).reshape(-1, 2 * B)
    assert_quant_parity(fmt, xb)
    assert_fq_parity(fmt, xb)
    if fmt == NV:
        assert_quant_parity(NV, xb, 2.0 ** -3)
        assert_fq_parity(NV, xb, 2.0 ** -3)


@pytest.mark.parametrize("fmt", [NV, MX])
def test_special_values(fmt):
    log("special values fmt=%d" % fmt)
    B = reqat.BLOCK[fmt]
    x = np.zeros((6, 2 * B), np.uint16)
    x[0, :] = 0x8000
    x[1, 0] = 0x7FC0
    x[1, B] = 0x3F80
    x[2, 3] = 0xFF80
    x[2, B:] = np.arange(1, B + 1)
    x[3, :B] = 0x7F7F
    x[3, B] = 0x0001
    x[4, :] = 0x0001
    x[5, :B] = 0x7F80
    assert_quant_parity(fmt, x)
    assert_fq_parity(fmt, x)
    assert_quant_parity(fmt, x[[0, 4]])           # tensor of only zeros / subnormals


@pytest.mark.parametrize("fmt,g", [(MX, None), (NV, 2.0 ** -5), (NV, 0.0123456789)])
def test_fakequant_in_place(fmt, g):
    """In place (y is x) is allowed when x is not read again after y is written:
    MXFP4, and NVFP4 with a given tensor scale."""
    log("fake-quant in place fmt=%d g=%r" % (fmt, g))
    xb = _rand(37, 512, 77, "student_t", outliers=5)
    g = None if g is None else float(np.float32(g))
    oy, _ = oracle.fakequant(fmt, xb, g)
    xt = wl.from_bits(xb).to(DEV)
    gt = None if g is None else torch.tensor([g], dtype=torch.float32, device=DEV)
    reqat.fakequant(xt, fmt, tensor_scale=gt, out=xt)
    torch.cuda.synchronize()
    assert np.array_equal(wl.bf16_bits(xt.cpu()), oy)


def test_fused_rejects_overlap():
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(RuntimeError):
        reqat.quantize_fakequant(x, NV, out=(torch.empty((4, 32), dtype=torch.uint8, device=DEV),
                                             torch.empty((4, 4), dtype=torch.uint8, device=DEV), x))
    with pytest.raises(RuntimeError):
        reqat.fakequant(x, NV, out=x)             # computed g re-reads x in its second pass


def test_empty_tensor_writes_unit_global_scale():
    log("empty tensor")
    x = torch.empty((0, 64), dtype=torch.bfloat16, device=DEV)
    c, s, gg = reqat.quantize(x, NV, out=(torch.empty((0, 32), dtype=torch.uint8, device=DEV),
                                          torch.empty((0, 4), dtype=torch.uint8, device=DEV)))
    torch.cuda.synchronize()
    assert float(gg.cpu()[0]) == 1.0


# ------------------------------------------------------------------ GEMM

def gpu_gemm(fmt, ac, as_, ga, bc, bs, gb, out_dtype, poison):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    gat = None if fmt == MX else torch.tensor([ga], dtype=torch.float32, device=DEV)
    gbt = None if fmt == MX else torch.tensor([gb], dtype=torch.float32, device=DEV)
    M, N = ac.shape[0], bc.shape[0]
    y = torch.full((M, N), poison, dtype=out_dtype, device=DEV)
    reqat.gemm(fmt, t(ac), t(as_), gat, t(bc), t(bs), gbt, out_dtype=out_dtype, out=y)
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64)


def check_gemm_points(fmt, ac, as_, ga, bc, bs, gb, y32, ybf, ms, ns):
    ref, aref = oracle.gemm_points(fmt, ac, as_, ga, bc, bs, gb, ms, ns)
    got = y32[ms, ns]
    nanref = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nanref)
    ok = ~nanref
    err = np.abs(got[ok] - ref[ok])
    m = indep.gemm_error_metrics(got, ref, aref)
    K = ac.shape[1] * 2
    log("  gemm fp32 K=%d %s" % (K, indep.format_metrics(m)))
    assert np.all(err <= GEMM_TOL * aref[ok]), float(np.max(err / np.maximum(aref[ok], 1e-300)))
    assert m["max_rel_sum"] <= indep.fp32_accumulation_bound(K), m
    if ybf is not None:
        gb_ = ybf[ms, ns][ok]
        rb = indep.bf16_values(oracle.bf16_from_double_array(ref[ok]))
        ulp = np.maximum(np.abs(rb), 2.0 ** -133) * 2.0 ** -7
        assert np.all(np.abs(gb_ - rb) <= ulp + GEMM_TOL * aref[ok])


def _w4a4_pack_ref(bc, bs, fmt):
    """The packed decode image as the header defines it, by numpy indexing:
    16-row groups and 256-element chunks (zero-padded); per unit (g, c) 2048
    code bytes (half h of piece q of row r at 1024 h + 16 (r + 16 q)) and,
    after all code units, 16 S scale bytes (piece q of row r at (S/4)(r + 16 q))."""
    N, Kh = bc.shape
    S = 16 if fmt == NV else 8
    G, C = -(-N // 16), -(-Kh // 128)
    cp = np.zeros((G * 16, C * 128), np.uint8)
    cp[:N, :Kh] = bc
    sp = np.zeros((G * 16, C * S), np.uint8)
    sp[:N, :bs.shape[1]] = bs
    codes = cp.reshape(G, 16, C, 4, 2, 16).transpose(0, 2, 4, 3, 1, 5).reshape(-1)   # [g][c][h][q][r][i]
    scales = sp.reshape(G, 16, C, 4, S // 4).transpose(0, 2, 3, 1, 4).reshape(-1)    # [g][c][q][r][j]
    return np.concatenate([codes, scales])


def check_gemm_packed(fmt, ac, as_, ga, bc, bs, gb):
    """M <= 64: the packed decode image equals the header's layout, and the
    product on it equals the row-major product bit for bit (FP32 and BF16)."""
    M, N, K = ac.shape[0], bc.shape[0], ac.shape[1] * 2
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    nb = reqat.reqat_w4a4_packed_bytes(fmt, N, K)
    packed = torch.full((max(nb, 16),), 0xA5, dtype=torch.uint8, device=DEV)
    reqat.pack_w4a4(t(bc), t(bs), fmt, out=packed)
    torch.cuda.synchronize()
    pref = _w4a4_pack_ref(bc, bs, fmt)
    assert pref.size == nb
    assert np.array_equal(packed.cpu().numpy()[:nb], pref), "packed image differs from the documented layout"
    gat = None if fmt == MX else torch.tensor([ga], dtype=torch.float32, device=DEV)
    gbt = None if fmt == MX else torch.tensor([gb], dtype=torch.float32, device=DEV)
    for dt, iv in ((torch.float32, torch.int32), (torch.bfloat16, torch.int16)):
        y = torch.full((M, N), float("nan"), dtype=dt, device=DEV)
        reqat.gemm(fmt, t(ac), t(as_), gat, t(bc), t(bs), gbt, out_dtype=dt, out=y)
        yp = torch.full((M, N), float("nan"), dtype=dt, device=DEV)
        reqat.gemm_packed(fmt, t(ac), t(as_), gat, packed, N, gbt, out_dtype=dt, out=yp)
        torch.cuda.synchronize()
        assert torch.equal(y.view(iv), yp.view(iv)), "packed product differs from the row-major one"


def run_gemm_case(fmt, M, N, K, seed, dist="normal", wstd=0.02, g=(None, None), all_points=True):
    xa = _rand(M, K, seed, dist, outliers=max(1, K // 100))
    xb = _rand(N, K, seed + 7, "normal", std=wstd)
    ac, as_, ga = oracle.quantize(fmt, xa, g[0])
    bc, bs, gb = oracle.quantize(fmt, xb, g[1])
    y1 = gpu_gemm(fmt, ac, as_, ga, bc, bs, gb, torch.float32, float("nan"))
    y2 = gpu_gemm(fmt, ac, as_, ga, bc, bs, gb, torch.float32, 0.0)
    assert np.array_equal(y1, y2, equal_nan=True), "poison visible or nondeterministic"
    yb = gpu_gemm(fmt, ac, as_, ga, bc, bs, gb, torch.bfloat16, float("nan"))
    if all_points:
        ms, ns = np.arange(M).repeat(N), np.tile(np.arange(N), M)
    else:
        rng = np.random.default_rng(seed)
        ms = np.concatenate([rng.integers(0, M, 3000), [0, M - 1, M - 1, 0]])
        ns = np.concatenate([rng.integers(0, N, 3000), [0, N - 1, 0, N - 1]])
    check_gemm_points(fmt, ac, as_, ga, bc, bs, gb, y1, yb, ms, ns)
    if M <= 64:
        check_gemm_packed(fmt, ac, as_, ga, bc, bs, gb)


@pytest.mark.parametrize("fmt", [NV, MX])
@pytest.mark.parametrize("M,N,K", [(16, 256, 256), (37, 200, 384), (1, 1, 128), (130, 129, 512),
                                   (256, 384, 1024), (5, 300, 128), (300, 520, 768),
                                   (257, 256, 2048), (512, 1000, 1280), (48, 100, 1152),
                                   (64, 40, 640), (33, 17, 128), (2, 8960, 1536),
                                   (100, 96, 384), (200, 130, 1152), (65, 300, 128),
                                   (20, 150, 640), (32, 96, 384)])
def test_gemm_parity(fmt, M, N, K):
    """(100, 96, 384), (200, 130, 1152) and (65, 300, 128): K % 256 == 128 with
    M > 64, which NVFP4 runs on the 128 x 128 register-staged kernel.
    (20, 150, 640) and (32, 96, 384): two 16-row activation tiles in the
    decode-shaped product, row-major and packed, with a ragged N and half a
    256-element chunk at the end of K."""
    log("gemm parity fmt=%d M=%d N=%d K=%d" % (fmt, M, N, K))
    run_gemm_case(fmt, M, N, K, seed=M * 31 + N * 7 + K, dist="student_t")


@pytest.mark.parametrize("fmt,K", [(MX, 1024), (MX, 1152), (NV, 1024)])
def test_gemm_many_tiles_per_workgroup(fmt, K):
    """More 256 x 256 tiles than workgroups (17 x 17 = 289), ragged edge tiles
    (4200 = 16*256 + 104 rows, 4100 = 16*256 + 4 columns); for MXFP4, K = 1024
    takes the grouped scale loads (K % 512 == 0) and K = 1152 the per-stage ones."""
    log("gemm many tiles fmt=%d K=%d" % (fmt, K))
    run_gemm_case(fmt, 4200, 4100, K, seed=K + fmt, dist="student_t", all_points=False)


def test_gemm_given_scales_nv():
    log("gemm NV given scales")
    run_gemm_case(NV, 64, 96, 256, seed=5, g=(0.0123, 3.5))


@pytest.mark.parametrize("fmt", [NV, MX])
def test_gemm_nan_block_propagates(fmt):
    log("gemm NaN fmt=%d" % fmt)
    B = reqat.BLOCK[fmt]
    xa = _rand(8, 256, 1)
    xa[3, B + 2] = 0x7FC0
    xb = _rand(16, 256, 2)
    ac, as_, ga = oracle.quantize(fmt, xa)
    bc, bs, gb = oracle.quantize(fmt, xb)
    y = gpu_gemm(fmt, ac, as_, ga, bc, bs, gb, torch.float32, 0.0)
    assert np.all(np.isnan(y[3])) and not np.any(np.isnan(np.delete(y, 3, axis=0)))


# ------------------------------------------------------------------ W4A16

def _w4a16_pack_ref(wc, ws):
    """The packed W4A16 weight image as the header defines it, by numpy
    indexing: 16-row groups (zero-padded), 128-element chunks; per unit (g, c)
    1024 code bytes (piece q of row r at 16 (r + 16 q)) and, after all code
    units, 64 scale bytes (row r's four bytes at 4 r)."""
    N, Kh = wc.shape
    G, C = -(-N // 16), Kh // 64
    cp = np.zeros((G * 16, Kh), np.uint8)
    cp[:N] = wc
    sp = np.zeros((G * 16, ws.shape[1]), np.uint8)
    sp[:N] = ws
    codes = cp.reshape(G, 16, C, 4, 16).transpose(0, 2, 3, 1, 4).reshape(-1)    # [g][c][q][r][i]
    scales = sp.reshape(G, 16, C, 4).transpose(0, 2, 1, 3).reshape(-1)          # [g][c][r][j]
    return np.concatenate([codes, scales])


def run_w4a16(xb, wc, ws):
    """Parity of reqat_gemm_w4a16 with the oracle (FP32 and BF16 outputs), and
    the packed path: the image equals the header's layout, the packed product
    equals the unpacked one bit for bit."""
    M, K = xb.shape
    N = wc.shape[0]
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    xt = wl.from_bits(xb).to(DEV)
    packed = torch.full((max(reqat.reqat_w4a16_packed_bytes(N, K), 16),), 0xA5, dtype=torch.uint8, device=DEV)
    reqat.pack_w4a16(t(wc), t(ws), out=packed)
    torch.cuda.synchronize()
    pref = _w4a16_pack_ref(wc, ws)
    assert np.array_equal(packed.cpu().numpy()[:pref.size], pref), "packed image differs from the documented layout"
    outs = []
    for dt, poison in ((torch.float32, float("nan")), (torch.float32, 0.0), (torch.bfloat16, float("nan"))):
        y = torch.full((M, N), poison, dtype=dt, device=DEV)
        reqat.gemm_w4a16(xt, t(wc), t(ws), out_dtype=dt, out=y)
        yp = torch.full((M, N), poison, dtype=dt, device=DEV)
        reqat.gemm_w4a16_packed(xt, packed, N, out_dtype=dt, out=yp)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.uint8) if dt == torch.bfloat16 else y.view(torch.int32),
                           yp.view(torch.uint8) if dt == torch.bfloat16 else yp.view(torch.int32)), \
            "packed product differs from the unpacked one"
        outs.append(y.float().cpu().numpy().astype(np.float64))
    assert np.array_equal(outs[0], outs[1], equal_nan=True), "poison visible or nondeterministic"
    ms, ns = np.arange(M).repeat(N), np.tile(np.arange(N), M)
    ref, aref = oracle.gemm_w4a16_points(xb, wc, ws, ms, ns)
    got = outs[0].reshape(-1)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    inf = np.isinf(ref)
    assert np.array_equal(got[inf], ref[inf])
    ok = ~(np.isnan(ref) | inf)
    err = np.abs(got[ok] - ref[ok])
    assert np.all(err <= GEMM_TOL * aref[ok]), float(np.max(err / np.maximum(aref[ok], 1e-300)))
    gb_ = outs[2].reshape(-1)[ok]
    rb = indep.bf16_values(oracle.bf16_from_double_array(ref[ok]))
    ulp = np.maximum(np.abs(rb), 2.0 ** -133) * 2.0 ** -7
    assert np.all(np.abs(gb_ - rb) <= ulp + GEMM_TOL * aref[ok])


def _w4a16_weights(N, K, seed, lo=110, hi=140):
    rng = np.random.default_rng(seed)
    return (rng.integers(0, 256, (N, K // 2), dtype=np.uint8),
            rng.integers(lo, hi, (N, K // 32), dtype=np.uint8))


@pytest.mark.parametrize("M,N,K", [(1, 16, 128), (5, 40, 256), (16, 256, 1536), (17, 33, 512),
                                   (33, 100, 384), (64, 48, 640), (100, 70, 1024)])
def test_w4a16_parity(M, N, K):
    log("w4a16 parity M=%d N=%d K=%d" % (M, N, K))
    xb = _rand(M, K, 40 + M + N, "student_t", outliers=max(1, K // 100))
    run_w4a16(xb, *_w4a16_weights(N, K, M + N))


def test_w4a16_special_scales():
    log("w4a16 special scale bytes")
    xb = _rand(8, 512, 91, "student_t", outliers=5)
    wc, ws = _w4a16_weights(24, 512, 91)
    ws[0, :] = 0                               # bfloat16-subnormal weights
    ws[1, 0] = 0xFF                            # a NaN block
    wc[3, :16] = 0
    ws[3, 0] = 0xFF                            # a NaN block of zero codes: NaN too
    ws[2, :] = 200                             # large but far from overflow for these x
    run_w4a16(xb, wc, ws)
    # every scale byte 0..250, small activations so that no FP32 sum overflows
    xs = indep.to_bf16_bits(np.random.default_rng(3).normal(0.0, 1e-3, (3, 128)))
    wc, _ = _w4a16_weights(251, 128, 4)
    ws = np.repeat(np.arange(251, dtype=np.uint8)[:, None], 4, axis=1)
    run_w4a16(xs, wc, ws)
    # scale bytes 253/254 with code 6.0: the bfloat16 weight overflows to +Inf
    ones = np.full((2, 128), 0x3F80, np.uint16)
    wc = np.full((3, 64), 0x77, np.uint8)
    ws = np.array([[253] * 4, [254] * 4, [127] * 4], np.uint8)
    run_w4a16(ones, wc, ws)


def test_w4a16_k_zero_writes_zeros():
    log("w4a16 K = 0")
    x = torch.empty((3, 0), dtype=torch.bfloat16, device=DEV)
    y = torch.full((3, 5), float("nan"), dtype=torch.float32, device=DEV)
    reqat.gemm_w4a16(x, torch.empty((5, 0), dtype=torch.uint8, device=DEV),
                     torch.empty((5, 0), dtype=torch.uint8, device=DEV), out=y)
    torch.cuda.synchronize()
    assert torch.equal(y.cpu(), torch.zeros(3, 5))


def test_gemm_k_zero_writes_zeros():
    log("gemm K=0")
    y = torch.full((4, 8), float("nan"), dtype=torch.float32, device=DEV)
    z = torch.zeros(16, dtype=torch.uint8, device=DEV)
    st = reqat.reqat_gemm_w4a4(MX, 4, 8, 0, z.data_ptr(), z.data_ptr(), None, z.data_ptr(),
                               z.data_ptr(), None, y.data_ptr(), reqat.DT_F32, 8,
                               torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert torch.all(y == 0).item()

def test_packed_decode_edge_cases():
    """The packed decode calls at the edges: K = 0 writes zeros (no operand is
    read), M = 0 with a computed activation scale writes g = 1, N = 0 leaves
    the output alone."""
    log("packed decode edge cases")
    stream = torch.cuda.current_stream().cuda_stream
    z = torch.zeros(16, dtype=torch.uint8, device=DEV)
    y = torch.full((4, 8), float("nan"), dtype=torch.float32, device=DEV)
    assert reqat.reqat_gemm_w4a4_packed(MX, 4, 8, 0, z.data_ptr(), z.data_ptr(), None, z.data_ptr(), None,
                                        y.data_ptr(), reqat.DT_F32, 8, stream) == 0
    torch.cuda.synchronize()
    assert torch.all(y == 0).item()
    one = torch.ones(1, dtype=torch.float32, device=DEV)
    g = torch.full((1,), float("nan"), dtype=torch.float32, device=DEV)
    x = torch.zeros(16, dtype=torch.bfloat16, device=DEV)
    ws = torch.zeros(256, dtype=torch.uint8, device=DEV)
    assert reqat.reqat_linear_w4a4_packed(NV, 0, 8, 128, x.data_ptr(), 128, g.data_ptr(), reqat.TS_COMPUTE,
                                          z.data_ptr(), one.data_ptr(), y.data_ptr(), reqat.DT_F32, 8,
                                          ws.data_ptr(), stream) == 0
    torch.cuda.synchronize()
    assert float(g.cpu()[0]) == 1.0
    y.fill_(float("nan"))
    assert reqat.reqat_linear_w4a4_packed(NV, 4, 0, 128, x.data_ptr(), 128, g.data_ptr(), reqat.TS_GIVEN,
                                          z.data_ptr(), one.data_ptr(), y.data_ptr(), reqat.DT_F32, 8,
                                          ws.data_ptr(), stream) == 0
    torch.cuda.synchronize()
    assert torch.isnan(y).all().item()

# ------------------------------------------------------------------ linear (quantize X + GEMM)

@pytest.mark.parametrize("fmt", [NV, MX])
@pytest.mark.parametrize("M,N,K,given", [(16, 256, 256, False), (5, 300, 128, False),
                                         (300, 520, 768, False), (257, 256, 2048, True),
                                         (16, 8960, 1536, False), (16, 1000, 1536, True),
                                         (64, 300, 1024, False), (33, 130, 1920, False),
                                         (1, 17, 128, False), (48, 64, 1280, True), (64, 96, 1152, False)])
def test_linear_parity(fmt, M, N, K, given):
    """reqat_linear_w4a4 = quantize X (same codes, scales and g as reqat_quantize_fp4,
    checked against the oracle) followed by the product, to the GEMM bar."""
    log("linear fmt=%d M=%d N=%d K=%d given=%s" % (fmt, M, N, K, given))
    seed = 11 * M + 5 * N + K
    xa = _rand(M, K, seed, "student_t", outliers=max(1, K // 100))
    xb = _rand(N, K, seed + 3, "normal", std=0.02)
    gx = 0.0625 if (given and fmt == NV) else None
    ac, as_, ga = oracle.quantize(fmt, xa, gx)
    bc, bs, gb = oracle.quantize(fmt, xb)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    x = wl.from_bits(xa).to(DEV)
    wg = None if fmt == MX else torch.tensor([gb], dtype=torch.float32, device=DEV)
    xg_in = None if gx is None else torch.tensor([gx], dtype=torch.float32, device=DEV)
    outs = []
    for dt, poison in ((torch.float32, float("nan")), (torch.float32, 0.0), (torch.bfloat16, float("nan"))):
        y = torch.full((M, N), poison, dtype=dt, device=DEV)
        ws = torch.full((reqat.reqat_linear_workspace_bytes(fmt, M, K),), 0xAB, dtype=torch.uint8, device=DEV)
        _, g = reqat.linear(x, fmt, t(bc), t(bs), wg, x_tensor_scale=xg_in, out_dtype=dt, out=y, ws=ws)
        torch.cuda.synchronize()
        if fmt == NV:
            assert float(g.cpu()[0]) == np.float32(ga)
        # the activation codes and scales the call left in its workspace are the oracle's
        off = 16384                                  # after the 4096 partial maxima
        wsn = ws.cpu().numpy()
        codes = wsn[off:off + M * K // 2].reshape(M, K // 2)
        off2 = off + ((M * K // 2 + 255) // 256) * 256
        scales = wsn[off2:off2 + M * (K // reqat.BLOCK[fmt])].reshape(M, K // reqat.BLOCK[fmt])
        assert np.array_equal(codes, ac) and np.array_equal(scales, as_)
        outs.append(y.float().cpu().numpy().astype(np.float64))
    assert np.array_equal(outs[0], outs[1], equal_nan=True), "poison visible or nondeterministic"
    ms, ns = np.arange(M).repeat(N), np.tile(np.arange(N), M)
    check_gemm_points(fmt, ac, as_, ga, bc, bs, gb, outs[0], outs[2], ms, ns)


@pytest.mark.parametrize("fmt", [NV, MX])
@pytest.mark.parametrize("M,K,given", [(16, 1536, False), (16, 1536, True), (64, 1024, False), (7, 2944, False),
                                       (24, 2048, False)])
def test_decode_linear_equals_two_launch_path(fmt, M, K, given):
    """The linear call on decode-sized activations: its outputs, the activation
    codes and scales it leaves in its workspace, and g are bitwise those of
    quantize() then gemm(), also with NaN blocks, an all-zero row, subnormal and
    huge values; the linear call on the packed weight image gives the same
    outputs and g bit for bit."""
    log("decode linear vs two launches fmt=%d M=%d K=%d given=%s" % (fmt, M, K, given))
    N = 700
    xa = _rand(M, K, 91 + M, "student_t", outliers=max(1, K // 100))
    xa[M // 2, 5] = 0x7FC0
    xa[M - 1, :] = 0x8000
    xa[0, 40:48] = 0x0003
    xa[0, 64] = 0x7F7F
    xb = _rand(N, K, 92, "normal", std=0.02)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    bc, bs, gb = oracle.quantize(fmt, xb)
    wg = None if fmt == MX else torch.tensor([gb], dtype=torch.float32, device=DEV)
    gx = None if not (given and fmt == NV) else torch.tensor([0.03125], dtype=torch.float32, device=DEV)
    x = wl.from_bits(xa).to(DEV)
    for dt in (torch.float32, torch.bfloat16):
        ws = torch.full((reqat.reqat_linear_workspace_bytes(fmt, M, K),), 0xCD, dtype=torch.uint8, device=DEV)
        y1 = torch.full((M, N), float("nan"), dtype=dt, device=DEV)
        _, g1 = reqat.linear(x, fmt, t(bc), t(bs), wg, x_tensor_scale=gx, out_dtype=dt, out=y1, ws=ws)
        xc, xs, g2 = reqat.quantize(x, fmt, tensor_scale=gx)
        y2 = torch.full((M, N), float("nan"), dtype=dt, device=DEV)
        reqat.gemm(fmt, xc, xs, g2, t(bc), t(bs), wg, out_dtype=dt, out=y2)
        torch.cuda.synchronize()
        c1, s1 = reqat.linear_workspace_views(ws, fmt, M, K)
        assert torch.equal(c1, xc) and torch.equal(s1, xs)
        if fmt == NV:
            assert float(g1.cpu()[0]) == float(g2.cpu()[0])
        iv = torch.int32 if dt == torch.float32 else torch.int16
        assert torch.equal(y1.view(iv), y2.view(iv)), "outputs differ"
        y3 = torch.full((M, N), float("nan"), dtype=dt, device=DEV)
        ws3 = torch.full((reqat.reqat_linear_workspace_bytes(fmt, M, K),), 0xCD, dtype=torch.uint8, device=DEV)
        _, g3 = reqat.linear_packed(x, fmt, reqat.pack_w4a4(t(bc), t(bs), fmt), N, wg, x_tensor_scale=gx,
                                    out_dtype=dt, out=y3, ws=ws3)
        torch.cuda.synchronize()
        assert torch.equal(y1.view(iv), y3.view(iv)), "packed linear differs"
        if fmt == NV:
            assert float(g3.cpu()[0]) == float(g1.cpu()[0])


# ------------------------------------------------------- strided operands

@pytest.mark.parametrize("fmt", [NV, MX])
@pytest.mark.parametrize("M,N,K", [(16, 200, 512), (300, 520, 1024), (130, 96, 384)])
def test_products_into_strided_output(fmt, M, N, K):
    """Products written into a wider row-major buffer (ldy > N, e.g. one slice
    of a fused QKV output) and, for the linear layer, read from a wider
    activation buffer (ldx > K): the slice matches the oracle and the padding
    columns keep their poison.  Covers the skinny (M <= 64), tiled and
    register-staged (NVFP4 with K % 256 == 128) kernels."""
    log("strided products fmt=%d M=%d N=%d K=%d" % (fmt, M, N, K))
    seed = 3 * M + N + K
    xa = _rand(M, K, seed, "student_t", outliers=max(1, K // 100))
    xb = _rand(N, K, seed + 1, "normal", std=0.02)
    ac, as_, ga = oracle.quantize(fmt, xa)
    bc, bs, gb = oracle.quantize(fmt, xb)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    gat = None if fmt == MX else torch.tensor([ga], dtype=torch.float32, device=DEV)
    gbt = None if fmt == MX else torch.tensor([gb], dtype=torch.float32, device=DEV)
    pad = 40
    ms, ns = np.arange(M).repeat(N), np.tile(np.arange(N), M)
    ref, aref = oracle.gemm_points(fmt, ac, as_, ga, bc, bs, gb, ms, ns)
    ref, aref = ref.reshape(M, N), aref.reshape(M, N)
    for dt in (torch.float32, torch.bfloat16):
        big = torch.full((M, N + pad), float("nan"), dtype=dt, device=DEV)
        reqat.gemm(fmt, t(ac), t(as_), gat, t(bc), t(bs), gbt, out_dtype=dt, out=big[:, :N])
        # the linear layer, activations read with ldx = K + 64
        xbig = np.zeros((M, K + 64), np.uint16)
        xbig[:, :K] = xa
        xv = wl.from_bits(xbig).to(DEV)[:, :K]
        big2 = torch.full((M, N + pad), float("nan"), dtype=dt, device=DEV)
        reqat.linear(xv, fmt, t(bc), t(bs), gbt, out_dtype=dt, out=big2[:, :N])
        torch.cuda.synchronize()
        for b in (big, big2):
            got = b.float().cpu().numpy().astype(np.float64)
            assert np.all(np.isnan(got[:, N:])), "padding columns written"
            y = got[:, :N]
            if dt == torch.float32:
                assert np.all(np.abs(y - ref) <= GEMM_TOL * aref)
            else:
                rb = indep.bf16_values(oracle.bf16_from_double_array(ref.reshape(-1))).reshape(M, N)
                ulp = np.maximum(np.abs(rb), 2.0 ** -133) * 2.0 ** -7
                assert np.all(np.abs(y - rb) <= ulp + GEMM_TOL * aref)


@pytest.mark.parametrize("M,N,K", [(16, 200, 512), (40, 130, 1024)])
def test_w4a16_strided(M, N, K):
    """W4A16 with activations read at ldx > K and the output written at ldy > N."""
    log("w4a16 strided M=%d N=%d K=%d" % (M, N, K))
    xb = _rand(M, K, 71 + M, "student_t", outliers=3)
    wc, ws = _w4a16_weights(N, K, 72 + N)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    xbig = np.zeros((M, K + 128), np.uint16)
    xbig[:, :K] = xb
    xv = wl.from_bits(xbig).to(DEV)[:, :K]
    big = torch.full((M, N + 24), float("nan"), dtype=torch.float32, device=DEV)
    reqat.gemm_w4a16(xv, t(wc), t(ws), out_dtype=torch.float32, out=big[:, :N])
    torch.cuda.synchronize()
    got = big.cpu().numpy().astype(np.float64)
    assert np.all(np.isnan(got[:, N:])), "padding columns written"
    ms, ns = np.arange(M).repeat(N), np.tile(np.arange(N), M)
    ref, aref = oracle.gemm_w4a16_points(xb, wc, ws, ms, ns)
    err = np.abs(got[:, :N].reshape(-1) - ref)
    assert np.all(err <= GEMM_TOL * aref)
