"""The gated verification harness on the GPU (paper section 3.7, Algorithm 1;
Eq. 2): K0's reference post-states against a numpy evaluation of what K0
computes, every candidate's outcome, the commit decisions and lineage, and
the harness's per-buffer comparison records against the CPU oracle run on
host copies of the same two states."""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import U, gamma, log
from paper_2608_20711_amd.gated import candidates as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def harness():
    from paper_2608_20711_amd.gated.harness import GatedEval
    log("gated: building the oracle set (K0 once per input)")
    h = GatedEval(warmup=3, reps=15)
    yield h
    h.close()


def _host(x, arena, name):
    """Data region of allocation `name` of input x, from `arena`, as bytes."""
    k = [t[0] for t in x.table].index(name)
    _, dt, es, rows, cols, stride, *_ = x.table[k]
    off = x.offsets[k] + 4096
    n = ((rows - 1) * stride + cols) * es
    return arena[off:off + n].cpu().numpy(), rows, cols, stride, es


def _bf16(raw, rows, cols, stride):
    a = torch.from_numpy(raw.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
    full = np.zeros(rows * stride, np.float32)
    full[:a.size] = a
    return full.reshape(rows, stride)[:, :cols]


def test_reference_post_states_are_what_k0_computes(harness):
    for x in harness.inputs:
        s = x.spec
        xs = _bf16(*_host(x, x.pre, "x")[:4])
        rs = _bf16(*_host(x, x.pre, "residual")[:4])
        w = _bf16(*_host(x, x.pre, "weight")[:4])[0]
        h = torch.from_numpy(xs + rs).to(torch.bfloat16).float().numpy()       # RNE to bf16
        got_h = _bf16(*_host(x, x.ref, "res_out")[:4])
        nan = np.isnan(h)
        assert np.array_equal(np.isnan(got_h), nan), s.name                   # NaN payloads may differ
        assert np.array_equal(got_h[~nan].view(np.uint32), h[~nan].view(np.uint32)), s.name
        hd = h.astype(np.float64)
        with np.errstate(invalid="ignore", over="ignore"):
            rstd = 1.0 / np.sqrt((hd * hd).sum(axis=1) / s.hidden + 1e-5)
            want = hd * rstd[:, None] * w.astype(np.float64)[None, :]
            # K0 sums squares in fp32: a square above the fp32 maximum makes the
            # sum +Inf and rstd 0 (the boundary input holds bf16's largest values)
            overflow = np.nansum(hd * hd, axis=1) > float(np.finfo(np.float32).max)
        raw, rows, cols, stride, _ = _host(x, x.ref, "out")
        full = np.zeros(rows * stride, np.float32)
        full[:raw.size // 4] = raw.view(np.float32)
        out = full.reshape(rows, stride)[:, :cols].astype(np.float64)
        got_r = _host(x, x.ref, "rstd")[0].view(np.float32).astype(np.float64)
        assert np.all(got_r[overflow & ~np.isnan(rstd)] == 0.0), s.name
        keep = ~overflow
        want, out, rstd, got_r = want[keep], out[keep], rstd[keep], got_r[keep]
        fin = np.isfinite(want)
        assert np.array_equal(np.isnan(out), np.isnan(want)), s.name
        assert np.all(np.abs(out[fin] - want[fin]) <= 2e-5 * np.abs(want[fin]) + 1e-6), s.name
        finr = np.isfinite(rstd)
        assert np.all(np.abs(got_r[finr] - rstd[finr]) <= 2e-5 * rstd[finr]), s.name
        log(f"gated: {s.name}: {int(overflow.sum())} rows with an fp32 overflow of the sum of squares")
        a = np.abs(h.astype(np.float64))
        a[np.isnan(a)] = -1.0
        assert np.array_equal(_host(x, x.ref, "amax")[0].view(np.int32), np.argmax(a, axis=1)), s.name
        log(f"gated: K0 post-state of {s.name} checked")


def test_outcomes_commits_and_lineage(harness):
    from paper_2608_20711_amd.gated.harness import search
    lineage, records = search(harness, C.CANDIDATES)
    for name, out, committed, bar in records:
        log(f"gated: {name:16s} {out.status:13s} speedup={out.speedup} cv={out.cv} committed={committed} "
            f"bar={bar} {out.reason[:120]}")
    by = {name: (out, committed, bar) for name, out, committed, bar in records}
    for cand in C.CANDIDATES:
        assert by[cand.name][0].status == cand.expect, (cand.name, by[cand.name][0].reason)
    # equivalent candidates ran the check 3 times on each of the 3 inputs
    for name in ("k0_roundtrip", "k1_vectorized", "sleep_in_loop"):
        out = by[name][0]
        assert len(out.checks) == 9 and all(c["equal"] for c in out.checks)
        assert out.speedup > 0 and 0 <= out.cv < 0.5
    # the rewrite is faster and becomes the best; the slowed copy is never committed
    assert by["k1_vectorized"][0].speedup > 1.05 and by["k1_vectorized"][1]
    assert by["sleep_in_loop"][0].speedup < 1.0 and not by["sleep_in_loop"][1]
    assert 0.8 < by["k0_roundtrip"][0].speedup < 1.25
    assert lineage[-1].name == "k1_vectorized"
    # the gate's decision is Eq. 2 on the recorded numbers
    for name, out, committed, bar in records:
        if out.status == "ok":
            assert committed == (out.speedup >= bar)
    # the divergences name what broke
    assert "out" in by["eps_constant"][0].reason
    shift = by["out_store_shift"][0].checks[-1]["buffers"]["out"]
    assert shift["pad_bytes_corrupted"] > 0 and shift["mismatches"] > 0
    amax = by["amax_lds_slot"][0].checks[-1]["buffers"]
    assert not amax["amax"]["equal"] and amax["out"]["equal"]


@pytest.mark.parametrize("name", ["out_store_shift", "eps_constant", "amax_lds_slot"])
def test_comparison_records_match_the_oracle(harness, name):
    """The harness's records for a divergent candidate equal the CPU oracle's
    diff, cosine, guard and pad checks of host copies of the two states."""
    cand = next(c for c in C.CANDIDATES if c.name == name)
    out = harness.evaluate(cand.make(harness.s_k0, harness.s_k1))
    assert out.status == "divergent"
    x = next(x for x in harness.inputs if x.spec.name == out.checks[-1]["input"])
    rec = out.checks[-1]["buffers"]
    work = x.work.cpu().numpy()
    ref = x.ref.cpu().numpy()
    names = {1: "f32", 2: "bf16", 5: "i32"}
    for k, (bname, dt, es, rows, cols, stride, _, _, _, is_input) in enumerate(x.table):
        off = x.offsets[k] + 4096
        tol = not is_input and dt != 5
        r = oracle.diff_segment(names[dt], "tolerance" if tol else "bitwise", "equal", rows, cols, stride, stride,
                                1e-3 if tol else 0.0, 0.0, work, ref, off, off)
        got = rec[bname]
        assert got["mismatches"] == r["mismatches"] and got["first_mismatch"] == r["first_mismatch"], bname
        assert got["bitwise_mismatches"] == r["bitwise_mismatches"], bname
        assert got["max_abs"] == r["max_abs"], bname
        if tol:
            c = oracle.cosine_segment(names[dt], rows, cols, stride, stride, work, ref, off, off)
            if math.isnan(c["cosine"]):
                assert math.isnan(got["cosine"]), bname
            else:   # exact sums against the library's order: within its error bound
                assert abs(got["cosine"] - c["cosine"]) <= 2.5 * gamma(110) + 16 * U, bname
        lo = work[x.offsets[k]:off]
        n = ((rows - 1) * stride + cols) * es
        hi = work[off + n:off + n + 4096]
        g = oracle.guard_check(x.spec.seed, 100 + k, lo, hi)
        assert got["guard_bytes_corrupted"] == g["bad_lo"] + g["bad_hi"], bname
        p = oracle.pad_check_alloc(x.spec.seed, 100 + k, names[dt], rows, cols, stride, work[off:off + n])
        assert got["pad_bytes_corrupted"] == p["bad_pad"], bname
    log(f"gated: {name} records equal the oracle's")
