"""Exhaustive GPU pins of the library's per-element device arithmetic, each
output compared bit for bit with the CPU oracle (which shares no code with
it), through test-only kernels built from the library's own headers
(tests/hip/device_pins.hip):

 * the fill's encoder from binary32 to bf16, fp16 and fp8 e4m3 (saturating
   and not) over all 2^32 binary32 inputs (section 3.4, Tier 1: the seeded
   state synthesis);
 * the fill's uniform-to-normal pieces: log_u(x) = ln((x + 1/2) 2^-32) and
   cos / sin of 2 pi x 2^-32 over all 2^32 inputs x, and the Box-Muller pair
   over 2^26 seeded input pairs;
 * the comparison's rule for one pair of elements (section 3.2, Eq. 1: the
   outcome, the non-finite flag, |A - B| and the fp64 division |A - B| / |B|
   behind the segment maxima) over 2^27 seeded fp32 pairs per NaN policy,
   2^25 per 16-bit type and every fp8 pair: over 3.4e8 divisions, each
   compared on its own."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import device_pins
import oracle
from gpu_helpers import THREADS, log

pytestmark = pytest.mark.gpu

ALL = 1 << 32
CHUNK = 1 << 26


def _by_parts(fn, n):
    """fn(lo, hi) over THREADS * 2 sub-ranges of [0, n) in threads (the
    oracle's loops release the GIL); results in order."""
    step = -(-n // (THREADS * 2))
    with ThreadPoolExecutor(THREADS) as ex:
        return list(ex.map(lambda lo: fn(lo, min(n, lo + step)), range(0, n, step)))


def _assert_equal(what, got, want, inputs):
    if all(_by_parts(lambda lo, hi: np.array_equal(got[lo:hi], want[lo:hi]), got.size)):
        return
    bad = np.flatnonzero(got != want)
    show = [(hex(int(inputs[i])), hex(int(got[i])), hex(int(want[i]))) for i in bad[:8]]
    raise AssertionError(f"{what}: {bad.size} outputs differ; (input, gpu, oracle): {show}")


class _Chunk:
    """The inputs x0 .. x0 + CHUNK - 1 of one chunk, and host buffers reused
    from chunk to chunk (pinned for the device copies)."""

    def __init__(self):
        self.base = np.arange(CHUNK, dtype=np.uint32)
        self.x = np.empty(CHUNK, dtype=np.uint32)
        self.host = {}

    def inputs(self, x0):
        np.add(self.base, np.uint32(x0), out=self.x)
        return self.x

    def fetch(self, name, dev, view):
        """dev copied into this chunk's pinned host buffer `name`, as a numpy view."""
        if name not in self.host:
            self.host[name] = torch.empty(dev.shape, dtype=dev.dtype, pin_memory=True)
        h = self.host[name]
        h.copy_(dev)
        return h.numpy().view(view)


@pytest.mark.timeout(900)
def test_encoders_every_binary32_input():
    L = device_pins.lib()
    outs = {"bf16": (torch.int16, np.uint16, "bf16", False), "f16": (torch.int16, np.uint16, "f16", False),
            "fp8 saturating": (torch.uint8, np.uint8, "fp8e4m3", True),
            "fp8": (torch.uint8, np.uint8, "fp8e4m3", False)}
    dev = {k: torch.empty(CHUNK, dtype=t[0], device="cuda") for k, t in outs.items()}
    ch = _Chunk()
    want = np.empty(CHUNK, dtype=np.uint64)
    narrow = {np.uint16: np.empty(CHUNK, dtype=np.uint16), np.uint8: np.empty(CHUNK, dtype=np.uint8)}
    for c, x0 in enumerate(range(0, ALL, CHUNK)):
        device_pins.check(L.pins_encode(x0, CHUNK, *[d.data_ptr() for d in dev.values()], None), "pins_encode")
        torch.cuda.synchronize()
        x = ch.inputs(x0)
        f = x.view(np.float32)
        for name, (_, npt, dt, sat) in outs.items():
            got = ch.fetch(name, dev[name], npt)
            w = narrow[npt]

            def oracle_part(lo, hi):
                oracle.encode_f32_n(dt, f[lo:hi], sat, out=want[lo:hi])
                assert want[lo:hi].max(initial=0) <= np.iinfo(npt).max
                w[lo:hi] = want[lo:hi]

            _by_parts(oracle_part, CHUNK)
            _assert_equal(f"encode {name}", got, w, x)
        if c % 8 == 7:
            log(f"  encoders: {(c + 1) * CHUNK:#x} of 2^32 binary32 inputs equal")


@pytest.mark.timeout(900)
def test_log_u_every_input():
    L = device_pins.lib()
    dev = torch.empty(CHUNK, dtype=torch.float64, device="cuda")
    ch = _Chunk()
    want = np.empty(CHUNK, dtype=np.float64)
    for c, x0 in enumerate(range(0, ALL, CHUNK)):
        device_pins.check(L.pins_log_u(x0, CHUNK, dev.data_ptr(), None), "pins_log_u")
        torch.cuda.synchronize()
        x = ch.inputs(x0)
        got = ch.fetch("log", dev, np.uint64)
        _by_parts(lambda lo, hi: oracle.log_u_n(x[lo:hi], out=want[lo:hi]), CHUNK)
        _assert_equal("log_u", got, want.view(np.uint64), x)
        if c % 8 == 7:
            log(f"  log_u: {(c + 1) * CHUNK:#x} of 2^32 inputs equal")


@pytest.mark.timeout(900)
def test_sincos_turns_every_input():
    L = device_pins.lib()
    dc = torch.empty(CHUNK, dtype=torch.float64, device="cuda")
    ds = torch.empty(CHUNK, dtype=torch.float64, device="cuda")
    ch = _Chunk()
    wc = np.empty(CHUNK, dtype=np.float64)
    ws = np.empty(CHUNK, dtype=np.float64)
    for c, x0 in enumerate(range(0, ALL, CHUNK)):
        device_pins.check(L.pins_sincos(x0, CHUNK, dc.data_ptr(), ds.data_ptr(), None), "pins_sincos")
        torch.cuda.synchronize()
        x = ch.inputs(x0)
        _by_parts(lambda lo, hi: oracle.sincos_turns_n(x[lo:hi], c=wc[lo:hi], s=ws[lo:hi]), CHUNK)
        _assert_equal("cos", ch.fetch("cos", dc, np.uint64), wc.view(np.uint64), x)
        _assert_equal("sin", ch.fetch("sin", ds, np.uint64), ws.view(np.uint64), x)
        if c % 8 == 7:
            log(f"  sincos_turns: {(c + 1) * CHUNK:#x} of 2^32 inputs equal")


@pytest.mark.timeout(600)
def test_box_muller_seeded_pairs():
    L = device_pins.lib()
    rng = np.random.default_rng(0xB0C5)
    n = 1 << 26
    xa = rng.integers(0, ALL, size=n, dtype=np.uint32)
    xb = rng.integers(0, ALL, size=n, dtype=np.uint32)
    xa[:4], xb[:4] = [0, 0xFFFFFFFF, 0x80000000, 1], [0, 0xFFFFFFFF, 0x40000000, 0x20000000]   # ends and quadrants
    z0 = torch.empty(n, dtype=torch.float64, device="cuda")
    z1 = torch.empty(n, dtype=torch.float64, device="cuda")
    ta, tb = torch.from_numpy(xa).cuda(), torch.from_numpy(xb).cuda()
    device_pins.check(L.pins_normal(ta.data_ptr(), tb.data_ptr(), n, z0.data_ptr(), z1.data_ptr(), None),
                      "pins_normal")
    torch.cuda.synchronize()
    want = np.empty(n, dtype=np.float64)
    for which, z in ((0, z0), (1, z1)):
        _by_parts(lambda lo, hi: oracle.normal_n(xa[lo:hi], xb[lo:hi], which, out=want[lo:hi]), n)
        _assert_equal(f"box_muller z{which}", z.cpu().numpy().view(np.uint64), want.view(np.uint64), xa)
    log(f"  box_muller: {n} pairs equal")


def _pairs(seed, bits, exp_mask, n):
    """Seeded pairs of raw elements (each part of the range from a generator of
    its own, seeded by (seed, start)): a uniform over all patterns; b by kind
    -- a single-bit flip of a, a small integer offset of a's pattern (nearby
    values: the tolerance boundary, quotients far below 1), a uniform
    pattern, a with another exponent field, or a signed zero."""
    a = np.empty(n, dtype=np.uint32)
    b = np.empty(n, dtype=np.uint32)
    mask = np.uint64((1 << bits) - 1)
    em = np.uint64(exp_mask)

    def part(lo, hi):
        rng = np.random.default_rng([seed, lo])
        m = hi - lo
        x = rng.integers(0, 1 << bits, size=m, dtype=np.uint64)
        kind = rng.integers(0, 5, size=m)
        flip = np.uint64(1) << rng.integers(0, bits, size=m).astype(np.uint64)
        off = rng.integers(-(1 << (bits - 9)), 1 << (bits - 9), size=m, dtype=np.int64)
        off = (off >> rng.integers(0, bits - 9, size=m)).astype(np.uint64)    # wraps: x + off is modular
        other = rng.integers(0, 1 << bits, size=m, dtype=np.uint64)
        y = np.select([kind == 0, kind == 1, kind == 2, kind == 3, kind == 4],
                      [x ^ flip, (x + off) & mask, other, (x & ~em & mask) | (other & em),
                       other & np.uint64(1 << (bits - 1))])
        a[lo:hi] = x
        b[lo:hi] = y

    step = 1 << 18
    with ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(lambda lo: part(lo, min(n, lo + step)), range(0, n, step)))
    return a, b


def _check_pairs(dtype, policy, atol, rtol, a, b, what):
    L = device_pins.lib()
    n = a.size
    ta, tb = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    flags = torch.empty(n, dtype=torch.uint8, device="cuda")
    mabs = torch.empty(n, dtype=torch.int64, device="cuda")
    mrel = torch.empty(n, dtype=torch.int64, device="cuda")
    device_pins.check(L.pins_pairs(oracle.DTYPE[dtype], int(policy == "strict"), atol, rtol, ta.data_ptr(),
                                   tb.data_ptr(), n, flags.data_ptr(), mabs.data_ptr(), mrel.data_ptr(), None),
                      "pins_pairs")
    torch.cuda.synchronize()
    wf = np.empty(n, dtype=np.uint8)
    wa = np.empty(n, dtype=np.float64)
    wr = np.empty(n, dtype=np.float64)
    _by_parts(lambda lo, hi: oracle.compare_pair_n(dtype, "tolerance", policy, atol, rtol, a[lo:hi], b[lo:hi],
                                                   wf[lo:hi], wa[lo:hi], wr[lo:hi]), n)
    key = a.astype(np.uint64) << np.uint64(32) | b.astype(np.uint64)
    _assert_equal(f"{what} flags", flags.cpu().numpy(), wf, key)
    _assert_equal(f"{what} |A - B|", mabs.cpu().numpy().view(np.uint64), wa.view(np.uint64), key)
    _assert_equal(f"{what} |A - B| / |B|", mrel.cpu().numpy().view(np.uint64), wr.view(np.uint64), key)
    return int(np.count_nonzero(wf & 1))


TOLS = [(0.0, 0.0), (1e-5, 1e-5), (2.0 ** -10, 2.0 ** -8), (1e-3, 1.6e-2), (1e30, 0.5)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("policy", ["equal", "strict"])
def test_pair_rule_fp32_seeded(policy):
    n, pieces = 1 << 27, 8
    divisions = 0
    for k in range(pieces):
        a, b = _pairs(0x5EED0 + 16 * (policy == "strict") + k, 32, 0x7F800000, n // pieces)
        atol, rtol = TOLS[k % len(TOLS)]
        divisions += _check_pairs("f32", policy, atol, rtol, a, b, f"f32 {policy} piece {k}")
    log(f"  pair rule f32 {policy}: {n} pairs equal ({divisions} with differing bits)")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_pair_rule_16_bit_seeded(dtype):
    n, pieces = 1 << 25, 4
    for k in range(pieces):
        a, b = _pairs(0x1600 + 16 * (dtype == "f16") + k, 16, 0x7F80 if dtype == "bf16" else 0x7C00, n // pieces)
        policy = ("equal", "strict")[k % 2]
        atol, rtol = TOLS[k % len(TOLS)]
        _check_pairs(dtype, policy, atol, rtol, a, b, f"{dtype} {policy} piece {k}")
    log(f"  pair rule {dtype}: {n} pairs equal")


def test_pair_rule_every_fp8_pair():
    v = np.arange(256, dtype=np.uint32)
    a, b = np.repeat(v, 256), np.tile(v, 256)
    for policy in ("equal", "strict"):
        for atol, rtol in TOLS:
            _check_pairs("fp8e4m3", policy, atol, rtol, a, b, f"fp8 {policy} atol={atol} rtol={rtol}")
