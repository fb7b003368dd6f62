"""Pins for the CPU oracle's primitives: Philox, element codecs, the fill's own
ln / sin / cos and its Box-Muller normal.  Each check ties the oracle to
something other than itself: published known-answer vectors, numpy / torch
casts, or extended-precision libm values."""
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append([int(t, 16) for t in line.split()])
    assert len(rows) == 3
    for r in rows:
        assert oracle.philox(r[0:4], r[4:6]) == r[6:10]
    # the bulk loop gives the same words
    ctr = np.array([r[0:4] for r in rows], dtype=np.uint32)
    key = np.array([r[4:6] for r in rows], dtype=np.uint32)
    out = oracle.philox_n(ctr, key)
    assert out.tolist() == [r[6:10] for r in rows]


# ---------------------------------------------------------------- decoders
def test_decode_f16_exhaustive_vs_numpy():
    raw = np.arange(1 << 16, dtype=np.uint64)
    cls, val = oracle.decode_n("f16", raw)
    ref = raw.astype(np.uint16).view(np.float16).astype(np.float64)
    assert np.array_equal(cls == 3, np.isnan(ref))
    assert np.array_equal(cls == 1, np.isposinf(ref))
    assert np.array_equal(cls == 2, np.isneginf(ref))
    fin = cls == 0
    assert np.array_equal(val[fin].view(np.uint64), ref[fin].view(np.uint64))   # incl. signed zeros


def test_decode_bf16_exhaustive_vs_torch():
    raw = np.arange(1 << 16, dtype=np.uint64)
    cls, val = oracle.decode_n("bf16", raw)
    t = torch.from_numpy(raw.astype(np.int64).astype(np.int16)).view(torch.bfloat16)
    ref = t.to(torch.float64).numpy()
    assert np.array_equal(cls == 3, np.isnan(ref))
    assert np.array_equal(cls == 1, np.isposinf(ref))
    assert np.array_equal(cls == 2, np.isneginf(ref))
    fin = cls == 0
    assert np.array_equal(val[fin].view(np.uint64), ref[fin].view(np.uint64))


def test_decode_fp8_exhaustive_vs_torch():
    raw = np.arange(256, dtype=np.uint64)
    cls, val = oracle.decode_n("fp8e4m3", raw)
    t = torch.from_numpy(raw.astype(np.uint8)).view(torch.float8_e4m3fn)
    ref = t.to(torch.float64).numpy()
    assert np.array_equal(cls == 3, np.isnan(ref))
    assert not np.any(cls == 1) and not np.any(cls == 2)     # no infinities in E4M3FN
    fin = cls == 0
    assert np.array_equal(val[fin].view(np.uint64), ref[fin].view(np.uint64))
    assert val[0x7E] == 448.0 and val[0xFE] == -448.0
    assert val[0x01] == 2.0 ** -9
    assert int((cls == 3).sum()) == 2                         # 0x7F and 0xFF


def test_decode_f32_sample_vs_numpy():
    rng = np.random.default_rng(1)
    raw = rng.integers(0, 1 << 32, size=1 << 18, dtype=np.uint64)
    raw[:8] = [0, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 1, 0x7F7FFFFF, 0x00800000]
    cls, val = oracle.decode_n("f32", raw)
    ref = raw.astype(np.uint32).view(np.float32).astype(np.float64)
    assert np.array_equal(cls == 3, np.isnan(ref))
    assert np.array_equal(cls == 1, np.isposinf(ref))
    fin = cls == 0
    assert np.array_equal(val[fin].view(np.uint64), ref[fin].view(np.uint64))


# ---------------------------------------------------------------- encoders
def _fp32_sample(n=1 << 20, seed=2):
    """Random fp32 bit patterns plus dense coverage of ties and boundaries."""
    rng = np.random.default_rng(seed)
    bits = rng.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    # values whose low mantissa bits sit exactly at / around rounding ties
    base = rng.integers(0, 1 << 32, size=n // 4, dtype=np.uint64).astype(np.uint32)
    ties = []
    for low in (0x8000, 0x7FFF, 0x8001, 0x10000, 0x18000, 0x100000, 0x080000, 0x07FFFF, 0x080001):
        ties.append((base & ~np.uint32(0x1FFFFF)) | np.uint32(low))
    t = np.concatenate(ties).view(np.float32)
    t = t[np.isfinite(t)]
    small = (rng.standard_normal(n // 4) * 4).astype(np.float32)
    return np.concatenate([x, t, small])


def test_encode_bf16_vs_torch():
    x = _fp32_sample()
    got = oracle.encode_f32_n("bf16", x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(got.astype(np.uint16), ref)


def test_encode_f16_vs_numpy():
    x = _fp32_sample(seed=3)
    # include the whole subnormal/normal boundary region of binary16 densely
    dense = np.arange(0x33000000, 0x39000000, 97, dtype=np.uint32).view(np.float32)
    edge = np.array([65504.0, 65519.99, 65520.0, 65536.0, 1e6, 2.0 ** -24, 2.0 ** -25,
                     2.0 ** -25 * 1.0000001, 3 * 2.0 ** -26], dtype=np.float32)
    x = np.concatenate([x, dense, -dense, edge, -edge])
    got = oracle.encode_f32_n("f16", x)
    ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got.astype(np.uint16), ref)


def test_encode_fp8_vs_torch_all_relevant_fp32():
    """Every fp32 value with exponent in the fp8 range (and beyond, up to 2^12),
    both signs, stepped densely; the non-saturating cast matches torch's E4M3FN
    cast, the saturating one matches torch after clamping to +-448."""
    lo = np.float32(2.0 ** -12).view(np.uint32)
    hi = np.float32(4096.0).view(np.uint32)
    bits = np.arange(lo, hi, 13, dtype=np.uint32)
    x = bits.view(np.float32)
    x = np.concatenate([x, -x, np.array([0.0, -0.0, 448.0, 464.0, 464.0001, 480.0, 1e30],
                                         dtype=np.float32)])
    got = oracle.encode_f32_n("fp8e4m3", x, saturate=False).astype(np.uint8)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got, ref)
    got_s = oracle.encode_f32_n("fp8e4m3", x, saturate=True).astype(np.uint8)
    ref_s = torch.from_numpy(np.clip(x, -448.0, 448.0)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got_s, ref_s)
    assert not np.any((got_s & 0x7F) == 0x7F)      # saturation never yields NaN


def test_encode_decode_roundtrip_exhaustive_16bit():
    for dt in ("bf16", "f16"):
        raw = np.arange(1 << 16, dtype=np.uint64)
        cls, val = oracle.decode_n(dt, raw)
        fin = cls == 0
        x = val[fin].astype(np.float32)         # exact: every bf16/f16 value is an fp32
        back = oracle.encode_f32_n(dt, x)
        assert np.array_equal(back, raw[fin])


# ------------------------------------------------------- fill transcendental
LD = np.longdouble
PI_LD = LD("3.141592653589793238462643383279502884")


def _ulp64(x):
    return np.spacing(np.abs(x).astype(np.float64))


def test_log_u_against_extended_precision():
    rng = np.random.default_rng(4)
    x = rng.integers(0, 1 << 32, size=1 << 18, dtype=np.uint64).astype(np.uint32)
    x = np.concatenate([x, np.array([0, 1, 2, 0x7FFFFFFF, 0x80000000, 0xB504F333, 0xB504F334,
                                     0xFFFFFFFE, 0xFFFFFFFF], dtype=np.uint32)])
    got = oracle.log_u_n(x)
    u = (x.astype(LD) + LD(0.5)) * LD(2.0) ** -32
    ref = np.log(u)
    err = np.abs(got.astype(LD) - ref)
    # within 2 ulp of the fp64 result everywhere
    assert np.all(err <= 2 * _ulp64(ref.astype(np.float64)))


def test_sincos_turns_against_extended_precision():
    rng = np.random.default_rng(5)
    x = rng.integers(0, 1 << 32, size=1 << 18, dtype=np.uint64).astype(np.uint32)
    edges = []
    for q in range(4):
        for d in (0, 1, 2, (1 << 29) - 1, 1 << 29, (1 << 29) + 1, (1 << 30) - 1):
            edges.append(q * (1 << 30) + d)
    x = np.concatenate([x, np.array(edges, dtype=np.uint64).astype(np.uint32)])
    c, s = oracle.sincos_turns_n(x)
    theta = LD(2) * PI_LD * x.astype(LD) * LD(2.0) ** -32
    rc, rs = np.cos(theta), np.sin(theta)
    # absolute error below 2^-52 (the values are bounded by 1)
    assert np.max(np.abs(c.astype(LD) - rc)) < LD(2.0) ** -52
    assert np.max(np.abs(s.astype(LD) - rs)) < LD(2.0) ** -52
    # exact quadrant points
    for q, (ec, es) in enumerate([(1, 0), (0, 1), (-1, 0), (0, -1)]):
        cc, ss = oracle.sincos_turns_n(np.array([q << 30], dtype=np.uint32))
        assert cc[0] == ec and ss[0] == es


def test_box_muller_against_extended_precision():
    rng = np.random.default_rng(6)
    xa = rng.integers(0, 1 << 32, size=1 << 16, dtype=np.uint64).astype(np.uint32)
    xb = rng.integers(0, 1 << 32, size=1 << 16, dtype=np.uint64).astype(np.uint32)
    u1 = (xa.astype(LD) + LD(0.5)) * LD(2.0) ** -32
    th = LD(2) * PI_LD * xb.astype(LD) * LD(2.0) ** -32
    rho = np.sqrt(LD(-2) * np.log(u1))
    for which, ref in ((0, rho * np.cos(th)), (1, rho * np.sin(th))):
        got = oracle.normal_n(xa, xb, which)
        assert np.max(np.abs(got.astype(LD) - ref)) < LD(1e-14)


def test_normal_extremes():
    # smallest u1 gives the largest radius sqrt(-2 ln 2^-33)
    z = oracle.normal_n(np.array([0], dtype=np.uint32), np.array([0], dtype=np.uint32), 0)
    assert abs(z[0] - np.sqrt(-2 * np.log(2.0 ** -33))) < 1e-13
