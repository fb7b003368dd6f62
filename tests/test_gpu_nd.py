"""GPU parity of N-dimensional segments (non-contiguous tensors and
block-table layouts, paper section 3.4) against the oracle's N-D compare:
transposed views (gathers), sliced views with long and short rows,
broadcast dimensions, scalars, empty shapes, result slots shared by the
blocks of a paged layout, every dtype, both NaN policies, and a larger
sliced 3-D tensor.  Every byte a segment names is checked to lie inside its
buffer before the launch."""
import numpy as np
import pytest
import torch

import cosine_order
import oracle
import paper_2608_20711_amd as lib
from gpu_helpers import assert_cosine, assert_results_equal, log
from paper_2608_20711_amd.state import SEG_RESULT_DTYPE

pytestmark = pytest.mark.gpu

NP_T = {"f32": np.float32, "f16": np.float16, "i32": np.int32, "i64": np.int64, "u8": np.uint8}


def _extent_bytes(shape, strides, es):
    if any(n == 0 for n in shape):
        return 0
    return (sum((n - 1) * s for n, s in zip(shape, strides)) + 1) * es


def _run(specs, a_host: np.ndarray, b_host: np.ndarray, n_results=None):
    """specs: dicts with dtype, mode, policy, shape, sa, sb, a_off, b_off, atol, rtol,
    result, index_base.  Returns (gpu results, oracle results)."""
    a_dev = torch.from_numpy(a_host.view(np.uint8).copy()).cuda()
    b_dev = torch.from_numpy(b_host.view(np.uint8).copy()).cuda()
    segs = []
    n_results = n_results if n_results is not None else len(specs)
    per_slot = [[] for _ in range(n_results)]
    for s in specs:
        es = oracle.ESIZE[oracle.DTYPE[s["dtype"]]]
        assert s["a_off"] + _extent_bytes(s["shape"], s["sa"], es) <= a_dev.numel(), s
        assert s["b_off"] + _extent_bytes(s["shape"], s["sb"], es) <= b_dev.numel(), s
        segs.append(lib.segment_nd(a_dev.data_ptr() + s["a_off"], b_dev.data_ptr() + s["b_off"],
                                   lib.DTYPE_CODE[s["dtype"]], lib.MODE_CODE[s["mode"]],
                                   lib.NAN_CODE[s["policy"]], s["shape"], s["sa"], s["sb"], s["atol"],
                                   s["rtol"], s["result"], s["index_base"]))
        per_slot[s["result"]].append(
            oracle.diff_segment_nd(s["dtype"], s["mode"], s["policy"], s["shape"], s["sa"], s["sb"], s["atol"],
                                   s["rtol"], a_host.view(np.uint8), b_host.view(np.uint8), s["a_off"],
                                   s["b_off"], s["index_base"]))
    res = torch.empty(max(1, n_results) * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    ws_size = lib.diff_nd_workspace_bytes(len(segs))
    ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
    lib.diff_segments_nd(segs, res.data_ptr(), n_results, ws.data_ptr(), ws_size)
    torch.cuda.synchronize()
    raw = res.cpu().numpy()[: n_results * SEG_RESULT_DTYPE.itemsize].view(SEG_RESULT_DTYPE)
    got = [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(n_results)]
    want = [oracle.merge_results(p) for p in per_slot]
    return got, want


def _spec(view, base_a, base_b, dtype, mode="tolerance", policy="equal", atol=1e-3, rtol=1e-3, result=0,
          index_base=0, view_b=None):
    view_b = view if view_b is None else view_b
    es = view.itemsize
    oa = view.__array_interface__["data"][0] - base_a.__array_interface__["data"][0]
    ob = view_b.__array_interface__["data"][0] - base_b.__array_interface__["data"][0]
    if dtype in ("i32", "i64", "u8"):
        mode = "bitwise"
    return dict(dtype=dtype, mode=mode, policy=policy, shape=list(view.shape),
                sa=[s // es for s in view.strides], sb=[s // es for s in view_b.strides],
                a_off=oa, b_off=ob, atol=atol, rtol=rtol, result=result, index_base=index_base)


def _perturbed(base: np.ndarray, rng, frac=0.002, specials=True):
    """A copy of `base` with a few elements changed (and NaN / Inf for floats)."""
    out = base.copy()
    flat = out.reshape(-1)
    k = max(1, int(frac * flat.size))
    idx = rng.choice(flat.size, size=k, replace=False)
    if np.issubdtype(base.dtype, np.floating):
        flat[idx] = (flat[idx].astype(np.float64) * (1 + rng.uniform(-0.01, 0.01, size=k))).astype(base.dtype)
        if specials:
            flat[idx[: k // 10]] = np.nan
            flat[idx[k // 10: k // 5]] = np.inf
    else:
        flat[idx] ^= 1
    return out


@pytest.mark.parametrize("dtype", ["f32", "f16", "i32", "i64", "u8"])
def test_views_of_one_tensor(dtype):
    rng = np.random.default_rng(11)
    shape = (6, 10, 34, 50)
    if dtype in ("f32", "f16"):
        b = rng.standard_normal(shape).astype(NP_T[dtype])
    else:
        b = rng.integers(0, 100, size=shape).astype(NP_T[dtype])
    a = _perturbed(b, rng)
    views = [
        lambda x: x,                                      # contiguous: one row
        lambda x: x.transpose(0, 1, 3, 2),                # innermost not unit-stride: gather
        lambda x: x.transpose(3, 2, 1, 0),
        lambda x: x[1:5, ::3, 2:30, 7:45],                # sliced, short rows
        lambda x: x[:, :, :, 7:45],                       # short rows whose outer dimensions merge into one
        lambda x: x[:, :, :, 8:40],                       # the same, rows 16-byte aligned for 8-byte elements
        lambda x: x[:, 2:9, :, :],                        # merges to long rows
        lambda x: x[::2, :, 5, :],                        # a dropped dimension
        lambda x: x[0, 0, 0, 0:1],                        # one element
        lambda x: x[:, :, 3:3, :],                        # empty
        lambda x: np.broadcast_to(x[:, :1, :, :], (6, 7, 34, 50)),   # broadcast
    ]
    specs = []
    for k, v in enumerate(views):
        for policy in ("equal", "strict"):
            va, vb = v(a), v(b)
            specs.append(_spec(va, a, b, dtype, policy=policy, result=len(specs), index_base=7 * k,
                               view_b=vb))
    got, want = _run(specs, a, b)
    assert_results_equal(got, want, f"{dtype} views")
    assert any(w["mismatches"] for w in want)


def test_scalar_and_differently_strided_operands():
    rng = np.random.default_rng(12)
    b = rng.standard_normal((40, 60)).astype(np.float32)
    a_full = _perturbed(np.ascontiguousarray(b.T), rng)          # candidate stored transposed
    specs = [
        _spec(a_full.T, a_full, b, "f32", view_b=b),               # a: column-major, b: row-major
        dict(dtype="f32", mode="tolerance", policy="equal", shape=[], sa=[], sb=[], a_off=4 * 17, b_off=4 * 17,
             atol=0.0, rtol=0.0, result=1, index_base=123),
    ]
    got, want = _run(specs, a_full, b)
    assert_results_equal(got, want, "scalar / mixed strides")


def test_block_table_segments_share_results():
    """A paged cache of 48 physical blocks of 16 x 64 bf16-sized (f16) values;
    two sequences, each a list of blocks; one segment per block, one result
    per sequence."""
    rng = np.random.default_rng(13)
    n_phys, blk, width = 48, 16, 64
    b = rng.standard_normal((n_phys, blk, width)).astype(np.float16)
    a = _perturbed(b, rng, frac=0.001, specials=False)
    order = rng.permutation(n_phys)
    seqs = [order[:20].tolist(), order[20:45].tolist()]
    specs = []
    for s, table in enumerate(seqs):
        for j, p in enumerate(table):
            specs.append(_spec(a[p], a, b, "f16", result=s, index_base=j * blk * width, view_b=b[p]))
    got, want = _run(specs, a, b, n_results=2)
    assert_results_equal(got, want, "block table")
    assert want[0]["mismatches"] > 0 and want[1]["mismatches"] > 0


def test_larger_sliced_tensor():
    rng = np.random.default_rng(14)
    shape = (48, 96, 2048)
    b = rng.standard_normal(shape).astype(np.float32)
    a = _perturbed(b, rng, frac=1e-4)
    log(f"nd large: {b.nbytes >> 20} MiB per side")
    specs = [_spec(a[3:45, 10:90, 16:2000], a, b, "f32", result=0, view_b=b[3:45, 10:90, 16:2000]),
             _spec(a[:, :, ::2], a, b, "f32", result=1, view_b=b[:, :, ::2]),
             _spec(a.transpose(1, 0, 2)[:, :, :1024], a, b, "f32", result=2,
                   view_b=b.transpose(1, 0, 2)[:, :, :1024])]
    got, want = _run(specs, a, b)
    assert_results_equal(got, want, "large sliced")


@pytest.mark.parametrize("dtype", ["f32", "f16", "i64", "u8"])
def test_every_other_element_views(dtype):
    """Views that take every other element of the innermost dimension: an
    operand whose rows start 16-byte aligned loads each chunk but the row's
    last as 32 contiguous bytes and keeps the even elements; misaligned
    operands, the last chunk of every row (partial or whole) and broadcast
    rows take the element-by-element path.  Row lengths from 1 to 2049
    elements, both operands or one of them aligned."""
    rng = np.random.default_rng(15)
    specs, tensors = [], []
    for L in (2, 3, 31, 32, 33, 64, 65, 129, 1000, 4098):
        rows = 2 + 3000 // L
        shape = (rows, L)
        if dtype in ("f32", "f16"):
            b = rng.standard_normal(shape).astype(NP_T[dtype])
        else:
            b = rng.integers(0, 200, size=shape).astype(NP_T[dtype])
        tensors.append((b, _perturbed(b, rng, frac=0.01)))
    for k, (b, a) in enumerate(tensors):
        views = [
            lambda x: x[:, ::2],                                     # aligned rows if L * es % 16 == 0
            lambda x: x[1:, ::2],                                    # from the second row
            lambda x: x[:, 1::2],                                    # odd start: misaligned
            lambda x: x.reshape(-1)[::2],                            # one long row
            lambda x: x.reshape(-1)[: x.size - 3][::2],              # a ragged last chunk
            lambda x: np.broadcast_to(x[:1, ::2], (4, (x.shape[1] + 1) // 2)),   # broadcast rows
        ]
        for j, v in enumerate(views):
            specs.append(_spec(v(a), a, b, dtype, result=len(specs), index_base=j, view_b=v(b)))
        # one operand aligned, the other not
        specs.append(_spec(a[:, ::2][:, : (a.shape[1] - 1) // 2], a, b, dtype, result=len(specs),
                           view_b=b[:, 1::2][:, : (b.shape[1] - 1) // 2]))
    # each tensor is its own pair of buffers
    got_all, want_all = [], []
    per = len(specs) // len(tensors)
    for k, (b, a) in enumerate(tensors):
        part = [dict(s, result=i) for i, s in enumerate(specs[k * per:(k + 1) * per])]
        got, want = _run(part, a, b)
        got_all += got
        want_all += want
    assert_results_equal(got_all, want_all, f"{dtype} every other element")
    assert any(w["mismatches"] for w in want_all)


_RAW_T = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16, "fp8e4m3": np.uint8, "i64": np.int64,
          "u8": np.uint8}


def _raw_pair(dtype, n, rng):
    """A reference buffer of n elements and a candidate that differs from it at
    about 2 % of the elements, with NaNs for the float types (raw patterns for
    bf16 and fp8)."""
    t = _RAW_T[dtype]
    if dtype in ("f32", "f16"):
        b = rng.standard_normal(n).astype(t)
    elif dtype == "bf16":
        b = (rng.standard_normal(n).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    elif dtype == "fp8e4m3":
        b = rng.integers(0, 256, size=n, dtype=np.uint8)
        b[(b & 0x7F) == 0x7F] ^= 1                         # finite reference values
    else:
        b = rng.integers(0, 1 << 20, size=n).astype(t)
    a = b.copy()
    idx = rng.choice(n, size=max(1, n // 50), replace=False)
    av = a.view(np.uint8).reshape(n, -1)
    av[idx, 0] ^= np.uint8(1) << rng.integers(0, 8, size=idx.size).astype(np.uint8)
    if dtype in ("f32", "f16", "bf16", "fp8e4m3"):
        nan = {"f32": np.uint32(0x7FC00000), "f16": np.uint16(0x7E00), "bf16": np.uint16(0x7FC0),
               "fp8e4m3": np.uint8(0x7F)}[dtype]
        j = rng.choice(n, size=max(1, n // 400), replace=False)
        a.view(nan.dtype)[j] = nan
        b.view(nan.dtype)[j[: j.size // 2]] = nan          # half of them on both sides
    return b, a


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16", "fp8e4m3", "i64", "u8"])
def test_strided_views_read_as_spans(dtype):
    """Gathers whose elements are s apart in both operands, s * esize up to 64
    bytes: with 16-byte aligned rows the plain N-D diff reads each row's
    covering bytes and compares only the elements at multiples of s.  The
    bytes between those elements differ between the operands (and hold NaN
    patterns) and must not count.  One long row, long rows spanning tiles,
    short rows (the narrow walk), a start off the 16-byte grid (the
    element-by-element path), ragged ends and a broadcast dimension; both NaN
    policies, index bases."""
    rng = np.random.default_rng(21)
    es = np.dtype(_RAW_T[dtype]).itemsize
    strides = sorted({2, 3, 4, 5, 8, 16, 64 // es} & set(range(2, 64 // es + 1)))
    specs_all, got_all, want_all = [], [], []
    for s_el in strides:
        n = 64 * 1024 // es * 3 + 37                        # not a whole number of rows or chunks
        b, a = _raw_pair(dtype, n, rng)
        row_long = 4096 // es * 4                           # elements per long row (16 KiB)
        row_short = 256 // es                               # 256 bytes: a few chunks per row
        g = 16 // es                                        # elements per 16 bytes
        views = [
            lambda x: x[::s_el],                                              # one long row
            lambda x: x[: x.size - 5][::s_el],                                # a ragged end
            lambda x: x[g:][::s_el],                                          # starts 16 bytes in
            lambda x: x[1:][::s_el] if es < 16 else x[::s_el],                # off the grid: elementwise
            lambda x: x[: (x.size // row_long) * row_long].reshape(-1, row_long)[:, ::s_el],
            lambda x: x[: (x.size // row_short) * row_short].reshape(-1, row_short)[:, ::s_el],
            lambda x: x[: (x.size // row_short) * row_short].reshape(-1, row_short)[3:40, g::s_el],
            lambda x: np.broadcast_to(x[: row_long * 2].reshape(2, row_long)[:1, ::s_el],
                                      (3, (row_long + s_el - 1) // s_el)),
        ]
        specs = []
        for k, v in enumerate(views):
            for policy in (("equal", "strict") if dtype in ("f32", "f16", "bf16", "fp8e4m3") else ("equal",)):
                sp = _spec(v(a), a, b, dtype, policy=policy, result=len(specs), index_base=1000 * k + 3,
                           view_b=v(b))
                if dtype in ("bf16", "fp8e4m3"):
                    sp["mode"] = "tolerance"
                specs.append(sp)
        got, want = _run(specs, a, b)
        specs_all += specs
        got_all += got
        want_all += want
        # the bytes between the elements differ: a plain contiguous compare of the covering region
        # would count them, the strided view must not
        assert any(w["bitwise_mismatches"] for w in want)
    assert_results_equal(got_all, want_all, f"{dtype} strided views")
    log(f"strided {dtype}: strides {strides}, {len(specs_all)} views equal")


# ------------------------------------------------------------ the cosine term over N-D segments
def _run_cos(specs, a_host: np.ndarray, b_host: np.ndarray, n_results: int):
    """asmevo_diff_cosine_nd over specs (the segments of a result consecutive):
    returns (gpu diff results, oracle diff results, gpu cosine results,
    (oracle cosine results from exact sums, documented-order model results,
    dtypes))."""
    from paper_2608_20711_amd.state import COS_RESULT_DTYPE as COS
    a_dev = torch.from_numpy(a_host.view(np.uint8).copy()).cuda()
    b_dev = torch.from_numpy(b_host.view(np.uint8).copy()).cuda()
    segs, per_slot, parts = [], [[] for _ in range(n_results)], [[] for _ in range(n_results)]
    dtypes = ["f32"] * n_results
    for s in specs:
        es = oracle.ESIZE[oracle.DTYPE[s["dtype"]]]
        assert s["a_off"] + _extent_bytes(s["shape"], s["sa"], es) <= a_dev.numel(), s
        assert s["b_off"] + _extent_bytes(s["shape"], s["sb"], es) <= b_dev.numel(), s
        segs.append(lib.segment_nd(a_dev.data_ptr() + s["a_off"], b_dev.data_ptr() + s["b_off"],
                                   lib.DTYPE_CODE[s["dtype"]], lib.MODE_CODE[s["mode"]],
                                   lib.NAN_CODE[s["policy"]], s["shape"], s["sa"], s["sb"], s["atol"],
                                   s["rtol"], s["result"], s["index_base"]))
        per_slot[s["result"]].append(
            oracle.diff_segment_nd(s["dtype"], s["mode"], s["policy"], s["shape"], s["sa"], s["sb"], s["atol"],
                                   s["rtol"], a_host.view(np.uint8), b_host.view(np.uint8), s["a_off"],
                                   s["b_off"], s["index_base"]))
        parts[s["result"]].append((s["shape"], s["sa"], s["sb"], s["a_off"], s["b_off"]))
        dtypes[s["result"]] = s["dtype"]
    res = torch.empty(max(1, n_results) * SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
    cres = torch.empty(max(1, n_results) * COS.itemsize, dtype=torch.uint8, device="cuda")
    ws_size = lib.diff_cosine_nd_workspace_bytes(segs, n_results)
    assert ws_size > 0
    ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
    lib.diff_cosine_nd(segs, res.data_ptr(), n_results, cres.data_ptr(), ws.data_ptr(), ws_size)
    torch.cuda.synchronize()
    raw = res.cpu().numpy()[: n_results * SEG_RESULT_DTYPE.itemsize].view(SEG_RESULT_DTYPE)
    got = [{f: raw[f][k].item() for f in SEG_RESULT_DTYPE.names} for k in range(n_results)]
    craw = cres.cpu().numpy()[: n_results * COS.itemsize].view(COS)
    cgot = [{f: craw[f][k].item() for f in COS.names} for k in range(n_results)]
    want = [oracle.merge_results(p) for p in per_slot]
    exact = [oracle.cosine_nd(dtypes[r], parts[r], a_host.view(np.uint8), b_host.view(np.uint8))
             for r in range(n_results)]
    model = [cosine_order.cosine_nd(dtypes[r], parts[r], a_host.view(np.uint8), b_host.view(np.uint8))
             for r in range(n_results)]
    return got, want, cgot, (exact, model, dtypes)


@pytest.mark.parametrize("dtype", ["f32", "f16", "i32"])
def test_cosine_views_of_one_tensor(dtype):
    """The cosine term of every view of test_views_of_one_tensor (contiguous,
    transposed gathers, sliced short rows, merged rows, a dropped dimension,
    one element, empty, broadcast), against the oracle's exact sums within
    the bound of the documented walk order and bit for bit against a model
    of that order; the diff results of the same pass equal the oracle's too."""
    rng = np.random.default_rng(21)
    shape = (6, 10, 34, 50)
    if dtype in ("f32", "f16"):
        b = rng.standard_normal(shape).astype(NP_T[dtype])
    else:
        b = rng.integers(0, 100, size=shape).astype(NP_T[dtype])
    a = _perturbed(b, rng)
    views = [
        lambda x: x,
        lambda x: x.transpose(0, 1, 3, 2),
        lambda x: x.transpose(3, 2, 1, 0),
        lambda x: x[1:5, ::3, 2:30, 7:45],
        lambda x: x[:, 2:9, :, :],
        lambda x: x[::2, :, 5, :],
        lambda x: x[0, 0, 0, 0:1],
        lambda x: x[:, :, 3:3, :],
        lambda x: np.broadcast_to(x[:, :1, :, :], (6, 7, 34, 50)),
    ]
    specs = []
    for k, v in enumerate(views):
        specs.append(_spec(v(a), a, b, dtype, result=len(specs), index_base=5 * k, view_b=v(b)))
    got, want, cgot, cwant = _run_cos(specs, a, b, len(specs))
    assert_results_equal(got, want, f"{dtype} views diff")
    assert_cosine(cgot, *cwant, f"{dtype} views cosine")
    if dtype != "i32":
        assert all(c["blocks"] > 0 for c in cgot[:7])


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_cosine_every_short_row_width_nd(dtype):
    """N-D views whose rows span 1 to 32 chunks, each with a partial last
    chunk, read with unit stride (sliced, rows aligned to 16 bytes or not)
    and element by element (a stride-3 gather): a lane holds chunks t and
    t + P of its row, so every width puts the row's last chunk in one of its
    two slots.  Each view is a result of its own; the cosine against the
    oracle's exact sums within the order's bound and bit for bit against the
    order model, the diff results equal."""
    rng = np.random.default_rng(23)
    epc = 16 // np.dtype(NP_T[dtype]).itemsize
    width = 3 * (32 * epc + epc)
    b = rng.standard_normal((3, 12, width)).astype(NP_T[dtype])
    a = _perturbed(b, rng, frac=0.003)
    specs = []
    for chunks in range(1, 33):
        cols = (chunks - 1) * epc + max(1, epc // 2 + chunks % (epc // 2))   # the last chunk partial
        for v in (lambda x, c=cols: x[:, 1:11, epc:epc + c],        # rows 16-byte aligned: vector loads
                  lambda x, c=cols: x[:, 1:11, 5:5 + c],            # rows off 16 bytes
                  lambda x, c=cols: x[:, :, 2:2 + 3 * c:3]):
            specs.append(_spec(v(a), a, b, dtype, result=len(specs), index_base=7 * len(specs), view_b=v(b)))
    got, want, cgot, cwant = _run_cos(specs, a, b, len(specs))
    assert_results_equal(got, want, f"{dtype} short-row widths diff")
    assert_cosine(cgot, *cwant, f"{dtype} short-row widths cosine")
    assert all(c["blocks"] > 0 for c in cgot)


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_cosine_row_tails_nd(dtype):
    """Rows of more than 32 chunks whose last tile is partial, tiled row by
    row: rows 16-byte aligned (every chunk of the last tile loaded, the
    lanes past the row's whole chunks cleared, a partial last chunk read
    element by element) with single rows shorter than one chunk, in a call
    of their own (the kernel for long aligned rows), rows off 16 bytes
    (chunk by chunk) in another, long gathers (strides 2, 3 and 5, rows
    16-byte aligned or not, a partial last chunk) in a third, and gathers of
    elements 2 apart in 16-byte-aligned rows in a fourth (the gathers'
    kernel); lengths that end on a chunk boundary or inside a chunk; against
    the oracle's exact sums within the order's bound and bit for bit against
    the order model."""
    rng = np.random.default_rng(24)
    es = np.dtype(NP_T[dtype]).itemsize
    epc = 16 // es
    width = 260 * epc + 2 * epc
    b = rng.standard_normal((3, 5, width)).astype(NP_T[dtype])
    a = _perturbed(b, rng, frac=0.002)
    lengths = [256 * epc + 3, 257 * epc + epc // 2, 175 * epc, 33 * epc + 1, 40 * epc - 1]
    aligned = [lambda x, n=n: x[:, :, epc:epc + n] for n in lengths]
    aligned += [lambda x: x[1, 2, epc:epc + 3], lambda x: x[2, 0, 0:1], lambda x: x[0, 4, epc:2 * epc - 1]]
    unaligned = [lambda x, n=n: x[:, 1:4, 1:1 + n] for n in lengths]
    gathers = [lambda x: x[:, :, ::2], lambda x: x[:, :, 1::3], lambda x: x[:, 1:4, 3::2], lambda x: x[0, 0, ::5]]
    pairs = [lambda x: x[:, :, ::2], lambda x: x[:, 2:5, 2 * epc::2], lambda x: x[1, 1, ::2],
             lambda x: x[:, 2:5, 2 * epc:2 * epc + 2 * 521:2]]      # the last chunk partial
    # one call of aligned rows only (the long-row kernel), one of rows off 16
    # bytes, one of gathers, one of gathers of elements 2 apart whose rows are
    # 16-byte aligned (the gathers' kernel)
    for name, views in (("aligned", aligned), ("unaligned", unaligned), ("gathers", gathers), ("pairs", pairs)):
        specs = [_spec(v(a), a, b, dtype, result=k, index_base=11 * k, view_b=v(b)) for k, v in enumerate(views)]
        got, want, cgot, cwant = _run_cos(specs, a, b, len(specs))
        assert_results_equal(got, want, f"{dtype} {name} row tails diff")
        assert_cosine(cgot, *cwant, f"{dtype} {name} row tails cosine")
        assert all(c["blocks"] > 0 for c in cgot)


def test_cosine_block_table_at_scale_equals_gathered_copy():
    """A shuffled block table of 8192 segments (1 GiB per side, 262144
    tiles): enough tiles that a workgroup of the cosine pass takes a second
    dealt block of tiles, thousands of segments past its first.  Its diff and
    cosine results equal, bit for bit, those of the same bytes gathered into
    one contiguous segment: the block sums and the tree over a result's
    blocks do not depend on where its segments lie in memory."""
    from paper_2608_20711_amd.state import COS_RESULT_DTYPE as COS
    n_blocks, blk = 8192, 32 * 1024                      # fp32 blocks of 128 KiB: 32 tiles each
    total = n_blocks * blk
    g = torch.Generator(device="cuda")
    g.manual_seed(25)
    b = torch.randn(total, device="cuda", generator=g)
    a = b.clone()
    hit = torch.randint(0, total, (total // 5000,), device="cuda", generator=g)
    a[hit] = a[hit] * 1.001
    perm = np.random.default_rng(25).permutation(n_blocks)
    pt = torch.from_numpy(perm).cuda()
    a2 = a.view(n_blocks, blk).index_select(0, pt).contiguous().view(-1)
    b2 = b.view(n_blocks, blk).index_select(0, pt).contiguous().view(-1)
    code = (lib.DTYPE_CODE["f32"], lib.MODE_CODE["tolerance"], lib.NAN_CODE["equal"])
    table = [lib.segment_nd(a.data_ptr() + int(p) * blk * 4, b.data_ptr() + int(p) * blk * 4, *code, [blk], [1], [1],
                            1e-4, 1e-4, 0, j * blk) for j, p in enumerate(perm)]
    whole = [lib.segment_nd(a2.data_ptr(), b2.data_ptr(), *code, [total], [1], [1], 1e-4, 1e-4, 0, 0)]
    out = []
    for segs in (table, whole):
        res = torch.empty(SEG_RESULT_DTYPE.itemsize, dtype=torch.uint8, device="cuda")
        cres = torch.empty(COS.itemsize, dtype=torch.uint8, device="cuda")
        ws_size = lib.diff_cosine_nd_workspace_bytes(segs, 1)
        ws = torch.empty(ws_size, dtype=torch.uint8, device="cuda")
        lib.diff_cosine_nd(segs, res.data_ptr(), 1, cres.data_ptr(), ws.data_ptr(), ws_size)
        torch.cuda.synchronize()
        out.append((bytes(res.cpu().numpy()), bytes(cres.cpu().numpy())))
    assert out[0] == out[1]
    r = out[0][0]
    got = np.frombuffer(r, dtype=SEG_RESULT_DTYPE)[0]
    cg = np.frombuffer(out[0][1], dtype=COS)[0]
    log(f"block table at scale: {int(got['mismatches'])} mismatches, "
        f"{int(cg['blocks'])} blocks, cosine {float(cg['cosine']):.12f}")
    assert int(cg["blocks"]) == total * 4 // 4096
    assert int(got["mismatches"]) > 0


def test_cosine_block_table_and_large_sliced_views():
    """Results made of several consecutive segments (a paged cache: one
    segment per block, one result per sequence), and large sliced and
    transposed views whose block trees use the level kernel (thousands of
    blocks per result)."""
    rng = np.random.default_rng(22)
    n_phys, blk, width = 48, 16, 64
    b = rng.standard_normal((n_phys, blk, width)).astype(np.float16)
    a = _perturbed(b, rng, frac=0.001, specials=False)
    order = rng.permutation(n_phys)
    seqs = [order[:20].tolist(), order[20:45].tolist(), []]
    specs = []
    for s, table in enumerate(seqs):
        for j, p in enumerate(table):
            specs.append(_spec(a[p], a, b, "f16", result=s, index_base=j * blk * width, view_b=b[p]))
    got, want, cgot, cwant = _run_cos(specs, a, b, 3)
    assert_results_equal(got, want, "block table diff")
    assert_cosine(cgot, *cwant, "block table cosine")
    assert cgot[2]["blocks"] == 0 and cgot[2]["cosine"] == 1.0
    shape = (48, 96, 2048)
    b = rng.standard_normal(shape).astype(np.float32)
    a = _perturbed(b, rng, frac=1e-4)
    specs = [_spec(a[3:45, 10:90, 16:2000], a, b, "f32", result=0, view_b=b[3:45, 10:90, 16:2000]),
             _spec(a[:, :, ::2], a, b, "f32", result=1, view_b=b[:, :, ::2]),
             _spec(a.transpose(1, 0, 2)[:, :, :1024], a, b, "f32", result=2,
                   view_b=b.transpose(1, 0, 2)[:, :, :1024])]
    log(f"nd cosine large: {b.nbytes >> 20} MiB per side")
    got, want, cgot, cwant = _run_cos(specs, a, b, 3)
    assert_results_equal(got, want, "large diff")
    assert_cosine(cgot, *cwant, "large cosine")
    assert cgot[0]["blocks"] > 256
