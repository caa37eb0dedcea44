"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Bar (per element, per row): max |y - y_ref| / y_ref <= 4e-6 and
|sum_j y_ij - 1| <= 1e-5, with y_ref from ``oracle.softmax_clipped`` on the
same seeded fp32 input.  Special rows (uniform, NaN, inf) are checked
exactly against the oracle's reading.
"""
import ctypes
import sys

import numpy as np
import pytest

import oracle
import paper_1904_12380_amd as sm
import workloads

pytestmark = pytest.mark.gpu

REL_TOL = 4e-6
SUM_TOL = 1e-5


def _torch():
    import torch
    return torch


def _dev():
    return _torch().device("cuda:0")


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(x: np.ndarray) -> np.ndarray:
    torch = _torch()
    xt = torch.from_numpy(np.ascontiguousarray(x)).to(_dev())
    yt = sm.softmax_fwd(xt)
    torch.cuda.synchronize()
    return yt.cpu().numpy()


def check_parity(x: np.ndarray, y: np.ndarray, what: str):
    want = oracle.softmax_clipped(x)
    y64 = y.astype(np.float64)
    finite = np.isfinite(want)
    assert np.array_equal(np.isnan(y64), np.isnan(want)), what
    rel = np.abs(y64[finite] - want[finite]) / want[finite]
    worst = float(rel.max()) if rel.size else 0.0
    if worst > REL_TOL:
        rel_all = np.where(finite, np.abs(y64 - want) / np.where(finite, want, 1), 0)
        idx = np.unravel_index(np.argmax(rel_all), y.shape)
        pytest.fail(f"{what}: max rel err {worst:.3e} at {idx}: got {y64[idx]!r}, "
                    f"want {want[idx]!r}, x={x[idx]!r}, rowmax={x[idx[0]].max()!r}")
    rows_ok = np.all(finite, axis=1)
    if rows_ok.any():
        sums = np.abs(y64[rows_ok].sum(axis=1) - 1.0)
        assert float(sums.max()) <= SUM_TOL, (what, float(sums.max()))
    return worst


@pytest.mark.parametrize("key", list(workloads.WORKLOADS))
def test_workload_parity(key):
    log(f"[parity] workload {key}")
    x = workloads.generate(key)
    y = run_gpu(x)
    worst = check_parity(x, y, key)
    log(f"[parity] {key}: max rel err {worst:.3e}")


EDGE_COLS = [1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 31, 32, 33, 49, 50, 51, 63, 64, 65, 100, 127,
             128, 129, 255, 256, 257, 1000, 1001, 1023, 1024, 1025, 2048, 4095, 4096, 4097,
             8191, 8192, 16384, 32767, 32768, 32769, 65536, 65537, 100003]
EDGE_ROWS = [1, 2, 3, 5, 63, 64, 65, 1000]


@pytest.mark.parametrize("cols", EDGE_COLS)
def test_edge_shapes(cols):
    log(f"[parity] edge cols={cols}")
    for rows in EDGE_ROWS:
        if rows * cols > 4_000_000:
            continue
        for kind in ("normal", "clip_heavy"):
            x = workloads.random_logits(rows, cols, seed=rows * 7919 + cols, kind=kind)
            check_parity(x, run_gpu(x), f"{rows}x{cols} {kind}")


@pytest.mark.parametrize("rows,cols", [(400001, 7), (200003, 21), (99999, 33), (98305, 62),
                                       (300001, 65), (100003, 250), (77777, 129)])
def test_packed_persistent_tiles(rows, cols):
    """More tiles than the persistent grid: every workgroup loops over
    several tiles with the next tile's loads in flight; ragged last tile."""
    log(f"[parity] packed persistent {rows}x{cols}")
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == "packed"
    tile_rows = 256 // p["lanes_per_row"]
    assert -(-rows // tile_rows) > p["grid"]
    x = workloads.random_logits(rows, cols, seed=rows, kind="clip_heavy")
    check_parity(x, run_gpu(x), f"packed {rows}x{cols}")


@pytest.mark.parametrize("rows,cols", [(1000003, 16), (300001, 100), (77777, 256), (5, 4),
                                       (1, 128), (129, 8), (1000, 32)])
def test_group_rows(rows, cols):
    """Aligned rows of up to 256 columns: G lanes per row, several rows per
    wavefront, ragged last row group, more row groups than the grid."""
    log(f"[parity] group rows {rows}x{cols}")
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == "group_rows" and p["elems_per_lane"] == 4
    assert p["lanes_per_row"] == max(1, 1 << (cols // 4 - 1).bit_length())
    for kind in ("normal", "clip_heavy", "offset"):
        x = workloads.random_logits(rows, cols, seed=rows + 3 * cols, kind=kind)
        check_parity(x, run_gpu(x), f"group rows {rows}x{cols} {kind}")


@pytest.mark.parametrize("cols,steps,rounds", [(4, 2, 1.5), (16, 2, 1.5), (32, 2, 1.5), (64, 2, 1.5),
                                               (128, 1, 1.125), (256, 1, 1.125), (16, 1, 1.125)])
def test_group_rows_looping_grid(cols, steps, rounds):
    """Launches that one workgroup per row block would spread over one to two
    rounds of the resident workgroups: the grid is capped at the resident
    ones, each loops over row blocks with the next block's loads in flight,
    and the last block is ragged.  steps = 2 row groups per wavefront step
    (1.5 rounds of blocks), steps = 1 (1.125 rounds at one row group per
    step, which the library runs with one).  The row count is chosen from
    the plan, so the test does not assume the device's occupancy."""
    g = max(1, 1 << (cols // 4 - 1).bit_length())
    per_wg = 4 * steps * (64 // g)      # 4 wavefronts x steps row groups x 64/G rows
    chosen = None
    for resident in (1024, 2048, 4096):
        rows = per_wg * int(rounds * resident) + 7
        p = sm.softmax_plan(rows, cols)
        needed = -(-rows // per_wg)
        if p["kernel_name"] == "group_rows" and p["grid"] == resident and resident < needed:
            chosen = (rows, p, needed)
            break
    assert chosen is not None, "no row count took the capped grid"
    rows, p, needed = chosen
    assert needed <= 2 * p["grid"]
    log(f"[parity] group rows looping {rows}x{cols}, grid {p['grid']} of {needed} blocks")
    x = workloads.random_logits(rows, cols, seed=rows + cols, kind="clip_heavy")
    check_parity(x, run_gpu(x), f"group rows looping {rows}x{cols}")


@pytest.mark.parametrize("cols,mid,large", [(36, "packed", "packed"), (100, "packed", "group_rows"),
                                             (128, "packed", "group_rows"),
                                             (244, "packed", "group_rows"),
                                             (64, "group_rows", "group_rows")])
def test_short_row_dispatch(cols, mid, large):
    """Whole-strip rows of at most 256 columns: grouped rows for a small
    launch whatever the fill; past it, the packed kernel for rows that fill
    less than 3/4 of their lanes, and for rows of more than 64 columns or
    filling their lanes in part while the grouped-rows grid takes one to
    2.5 rounds of the resident workgroups.  The resident count is found
    from the plans, not assumed; the mid-size launch is checked for parity."""
    g = 1 << (cols // 4 - 1).bit_length()
    per_wg = 4 * 2 * (64 // g)          # rows per workgroup at two row groups per step
    found = None
    for resident in (1024, 2048, 4096):
        kinds = [sm.softmax_plan(per_wg * int(f * resident), cols)["kernel_name"]
                 for f in (0.3, 2, 6)]
        if kinds == ["group_rows", mid, large]:
            found = resident
            break
    assert found is not None, "no resident count explains the plans"
    rows = per_wg * 2 * found + 5
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == mid
    log(f"[parity] short-row dispatch {rows}x{cols} on {mid}")
    x = workloads.random_logits(rows, cols, seed=rows, kind="clip_heavy")
    check_parity(x, run_gpu(x), f"short-row dispatch {rows}x{cols}")


@pytest.mark.parametrize("rows,cols", [(257, 50), (64, 1000), (33, 1001), (5, 8192), (3, 100003),
                                       (131, 7), (257, 130), (99, 3001)])
def test_misaligned_views(rows, cols):
    """x and y start 4 bytes past a 16-byte boundary: the 32-bit paths."""
    torch = _torch()
    log(f"[parity] misaligned {rows}x{cols}")
    x = workloads.random_logits(rows, cols, seed=cols, kind="offset")
    n = rows * cols
    xb = torch.empty(n + 4, dtype=torch.float32, device=_dev())
    yb = torch.empty(n + 4, dtype=torch.float32, device=_dev())
    xb[1:n + 1] = torch.from_numpy(x.reshape(-1)).to(_dev())
    xv = xb[1:n + 1].view(rows, cols)
    yv = yb[1:n + 1].view(rows, cols)
    assert xv.data_ptr() % 16 == 4
    p = sm.softmax_plan(rows, cols, xv.data_ptr(), yv.data_ptr())
    assert p["vec_width"] == 1
    sm.softmax_fwd(xv, out=yv)
    torch.cuda.synchronize()
    check_parity(x, yv.cpu().numpy(), f"misaligned {rows}x{cols}")


@pytest.mark.parametrize("rows,cols", [(17, 2049), (33, 3001), (9, 4093), (11, 4095), (5, 6143),
                                       (7, 8189), (9, 16381), (5, 32765), (6, 65533), (3, 100003),
                                       (2, 262147)])
def test_row_phase_access(rows, cols):
    """Rows that are not whole 16-byte strips in aligned x and y: 128-bit
    access in the aligned strips around each row (every phase 0..3 occurs
    over four consecutive rows), straddling strips element by element."""
    log(f"[parity] row phase {rows}x{cols}")
    p = sm.softmax_plan(rows, cols)
    assert p["vec_width"] == 4 and p["kernel_name"] in ("wave_row", "block_row", "split_row")
    for kind in ("normal", "clip_heavy", "offset"):
        x = workloads.random_logits(rows, cols, seed=rows * 5 + cols, kind=kind)
        check_parity(x, run_gpu(x), f"row phase {rows}x{cols} {kind}")


@pytest.mark.parametrize("rows,cols", [(115200, 50), (64, 1000), (512, 32768), (64, 262144),
                                       (7, 3), (67, 1001), (9, 4093), (13, 250), (5, 8189),
                                       (7, 32767), (3, 100003)])
def test_in_place(rows, cols):
    torch = _torch()
    log(f"[parity] in-place {rows}x{cols}")
    x = workloads.random_logits(rows, cols, seed=3, kind="normal")
    xt = torch.from_numpy(x).to(_dev())
    out = sm.softmax_fwd(xt, out=xt)
    assert out.data_ptr() == xt.data_ptr()
    torch.cuda.synchronize()
    check_parity(x, xt.cpu().numpy(), f"in-place {rows}x{cols}")


def test_non_default_stream_and_determinism():
    torch = _torch()
    log("[parity] side stream + determinism")
    for key in ("dam_attention_115200x50", "vocab_512x32768", "longrow_64x262144"):
        x = workloads.generate(key)
        xt = torch.from_numpy(x).to(_dev())
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            y1 = sm.softmax_fwd(xt)
            y2 = sm.softmax_fwd(xt)
        s.synchronize()
        y3 = sm.softmax_fwd(xt)
        torch.cuda.synchronize()
        a, b, c = y1.cpu().numpy(), y2.cpu().numpy(), y3.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), key
        assert np.array_equal(a.view(np.uint32), c.view(np.uint32)), key
        check_parity(x, a, key)


@pytest.mark.parametrize("cols", [1, 3, 50, 64, 1000, 4096, 32768, 262144])
def test_uniform_rows_are_exactly_one_over_n(cols):
    """Equal logits: exp gives exactly 1, the sum exactly N, and the output
    must be the fp32 division 1/N (bitwise)."""
    log(f"[parity] uniform cols={cols}")
    rows = max(1, min(64, 2_000_000 // cols))
    x = np.full((rows, cols), -3.75, dtype=np.float32)
    x[::2] = 12.5
    y = run_gpu(x)
    want = np.float32(1.0) / np.float32(cols)
    assert np.all(y == want), (cols, np.unique(y)[:5], want)


def test_clip_rows():
    """Rows where the clip is active, including values straddling -64."""
    log("[parity] clip rows")
    base = [
        [0.0, -100.0, -64.0, -63.5, -1.0e4],
        [10.0, -54.0, -53.999996185302734, -54.000003814697266, 9.0],
        [-3.0, -70.0, -2.0, -66.5, -67.0, -65.99999237060547],
    ]
    for row in base:
        for cols in (len(row), 50, 1000, 40000):
            x = np.full((4, cols), -500.0, dtype=np.float32)
            x[:, :len(row)] = np.asarray(row, dtype=np.float32)
            check_parity(x, run_gpu(x), f"clip row {row[:2]} cols={cols}")
            e64 = np.exp(-64.0)
            assert np.all(run_gpu(x) >= np.float32(e64 / cols * (1 - 1e-5)))


@pytest.mark.parametrize("cols", [5, 50, 1000, 8192, 70000])
def test_nonfinite_rows(cols):
    log(f"[parity] non-finite cols={cols}")
    x = workloads.random_logits(6, cols, seed=cols, kind="normal")
    x[0, cols // 2] = np.nan
    x[1, cols - 1] = np.inf
    x[2, :] = -np.inf
    x[3, 0] = -np.inf
    x[4, :] = -np.inf
    x[4, cols // 3] = 1.0
    y = run_gpu(x)
    want = oracle.softmax_clipped(x)
    assert np.all(np.isnan(y[0])) and np.all(np.isnan(y[1])) and np.all(np.isnan(y[2]))
    check_parity(x[3:], y[3:], f"non-finite finite rows cols={cols}")
    assert np.allclose(y[4].astype(np.float64), want[4], rtol=REL_TOL, atol=0)


@pytest.mark.parametrize("rows,cols", [(257, 50), (65, 1000), (3, 8192), (2, 262144), (9, 1001),
                                       (6, 4093), (5, 257), (3, 100003), (4, 16385)])
def test_guard_bands_untouched(rows, cols):
    """Sentinels before and after y survive the call."""
    torch = _torch()
    log(f"[parity] guard bands {rows}x{cols}")
    pad = 1024
    n = rows * cols
    x = workloads.random_logits(rows, cols, seed=11, kind="normal")
    xt = torch.from_numpy(x).to(_dev())
    yb = torch.full((n + 2 * pad,), 12345.0, dtype=torch.float32, device=_dev())
    yv = yb[pad:pad + n].view(rows, cols)
    sm.softmax_fwd(xt, out=yv)
    torch.cuda.synchronize()
    yb_h = yb.cpu().numpy()
    assert np.all(yb_h[:pad] == 12345.0) and np.all(yb_h[pad + n:] == 12345.0)
    check_parity(x, yv.cpu().numpy(), f"guard {rows}x{cols}")


def test_empty_inputs_launch_nothing():
    torch = _torch()
    for shape in ((0, 50), (5, 0)):
        xt = torch.empty(shape, dtype=torch.float32, device=_dev())
        assert sm.softmax_fwd(xt).shape == shape


def test_exp_probe_error_bound():
    """The kernels' clipped exp against float64 exp over the whole clipped
    domain, with x and m drawn so that x - m is not exact in fp32 (the dense
    scans are in test_gpu_exp_scan.py)."""
    torch = _torch()
    log("[parity] exp probe")
    rng = np.random.default_rng(99)
    n = 1 << 22
    m = rng.uniform(-60.0, 60.0, n).astype(np.float32)
    d = np.concatenate([rng.uniform(-70.0, 0.0, n - 4096),
                        rng.uniform(-64.001, -63.999, 4096)])
    x = (m.astype(np.float64) + d).astype(np.float32)
    e = sm.softmax_exp_probe(torch.from_numpy(x).to(_dev()),
                             torch.from_numpy(m).to(_dev())).cpu().numpy()
    want = oracle.exp_clipped(x.astype(np.float64) - m.astype(np.float64))
    rel = np.abs(e.astype(np.float64) - want) / want
    worst = float(rel.max())
    log(f"[parity] exp probe max rel err {worst:.3e} ({worst / 2**-24:.2f} half-ulps)")
    # 1.5 ulp, as a relative error: ulp(w) / w <= 2^-23
    assert worst <= 1.5 * 2.0**-23


def test_copy_probe():
    torch = _torch()
    x = torch.randn(1 << 20, device=_dev())
    assert torch.equal(sm.softmax_copy_probe(x), x)
    xo = x[1:]
    assert torch.equal(sm.softmax_copy_probe(xo), xo)
    # in place, 128-bit and 32-bit paths
    for t in (x.clone(), x.clone()[1:]):
        ref = t.clone()
        assert torch.equal(sm.softmax_copy_probe(t, out=t), ref)


def _hip():
    lib = ctypes.CDLL("libamdhip64.so")
    lib.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    lib.hipFree.argtypes = [ctypes.c_void_p]
    lib.hipMemGetAddressRange.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                          ctypes.POINTER(ctypes.c_size_t), ctypes.c_void_p]
    return lib


def test_range_past_allocation_is_rejected():
    """A byte range that ends 16 bytes past a hipMalloc allocation is refused
    before launch.  The overrun is inside the allocation's page, so the check
    is exercised without any access outside mapped memory."""
    torch = _torch()
    torch.cuda.init()
    hip = _hip()
    nbytes = 1 << 20
    p = ctypes.c_void_p()
    assert hip.hipMalloc(ctypes.byref(p), nbytes) == 0
    try:
        base, size = ctypes.c_void_p(), ctypes.c_size_t()
        assert hip.hipMemGetAddressRange(ctypes.byref(base), ctypes.byref(size), p) == 0
        if size.value != nbytes:
            pytest.skip(f"allocation reported as {size.value} bytes")
        xp = p.value + 16
        # rows*cols*4 == nbytes: ends 16 bytes past the allocation
        rc = sm.softmax_fwd_ptr(xp, xp, 1, nbytes // 4, 0)
        assert rc == sm.ERR_NOT_DEVICE
        assert sm.softmax_fwd_ptr(p.value, p.value, 1, nbytes // 4, 0) == sm.OK
        torch.cuda.synchronize()
    finally:
        hip.hipFree(p)


def test_host_pointer_is_rejected():
    """Unregistered host memory is refused before launch.  The test first
    confirms through HIP itself that the pointer is unregistered."""
    torch = _torch()
    torch.cuda.init()
    hip = ctypes.CDLL("libamdhip64.so")
    buf = np.zeros(4096, dtype=np.float32)

    class Attr(ctypes.Structure):
        _fields_ = [("type", ctypes.c_int), ("device", ctypes.c_int),
                    ("devicePointer", ctypes.c_void_p), ("hostPointer", ctypes.c_void_p),
                    ("isManaged", ctypes.c_int), ("allocationFlags", ctypes.c_uint)]
    a = Attr()
    hip.hipPointerGetAttributes.argtypes = [ctypes.POINTER(Attr), ctypes.c_void_p]
    rc = hip.hipPointerGetAttributes(ctypes.byref(a), buf.ctypes.data)
    hip.hipGetLastError()
    if rc == 0 and a.type != 0:
        pytest.skip(f"HIP reports host memory type {a.type}")
    assert sm.softmax_fwd_ptr(buf.ctypes.data, buf.ctypes.data, 64, 64, 0) == sm.ERR_NOT_DEVICE


def test_split_rows_several_one_pass_launches():
    """More rows than one launch holds: several one-pass launches back to
    back, each claiming and releasing its own exchange region."""
    log("[parity] split rows, several one-pass launches")
    p = sm.softmax_plan(65, 262144)
    assert p["kernel_name"] == "split_row" and p["launches"] == 2
    assert p["grid"] % p["chunks_per_row"] == 0
    x = workloads.random_logits(65, 262144, seed=5, kind="offset")
    y1 = run_gpu(x)
    check_parity(x, y1, "65x262144")
    y2 = run_gpu(x)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("rows,cols", [(55, 300000), (20, 200000), (419, 40000), (6, 300001)])
def test_split_rows_chunk_by_row_count(rows, cols):
    """Long rows whose chunk size the library picks by row count (8192-column
    chunks where 16384-column ones would take more launches or leave the
    chip thin), and a call whose last one-pass launch is short (its store
    delay follows its own reads).  The plan is read back, not assumed: the
    geometry must be consistent and the output must match the oracle."""
    log(f"[parity] split rows, chunk by row count {rows}x{cols}")
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == "split_row" and p["block_threads"] in (256, 512)
    chunk = p["block_threads"] * p["elems_per_lane"]
    assert p["chunks_per_row"] == -(-(cols + (3 if cols % 4 else 0)) // chunk) or \
        p["chunks_per_row"] == -(-cols // chunk)
    assert p["grid"] % p["chunks_per_row"] == 0
    per_launch = p["grid"] // p["chunks_per_row"]
    assert p["launches"] == -(-rows // per_launch)
    x = workloads.random_logits(rows, cols, seed=rows + cols, kind="offset")
    y1 = run_gpu(x)
    check_parity(x, y1, f"{rows}x{cols}")
    y2 = run_gpu(x)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("rows_of_cus,cols,kernel", [
    (lambda c: c * 204 // 256, 20480, "block_row"),
    (lambda c: c // 3 + 1, 17408, "block_row"),
    (lambda c: c * 15 // 16, 22528, "block_row"),
    (lambda c: c // 3 - 1, 20480, "split_row"),
    (lambda c: c * 15 // 16 + 1, 18432, "split_row"),
    (lambda c: c * 170 // 256, 24576, "split_row"),
], ids=["0.8cus-20480", "cus/3+1-17408", "15/16cus-22528", "cus/3-1-20480",
        "15/16cus+1-18432", "0.66cus-24576"])
def test_three_chunk_rows_by_row_count(rows_of_cus, cols, kernel):
    """Rows of 16384 to 24576 columns whose third 8192-column chunk would be
    partly empty take one workgroup per row when there are between 1/3 and
    15/16 as many rows as compute units; outside that band, or with whole
    chunks, the split kernel.  The row counts follow the device's CU count.
    The output must match the oracle and repeat bit for bit."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rows = rows_of_cus(cus)
    log(f"[parity] three-chunk rows by row count {rows}x{cols} ({cus} CUs)")
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == kernel and p["vec_width"] == 4, p
    if kernel == "block_row":
        assert p["block_threads"] == 1024 and p["grid"] == rows
    x = workloads.random_logits(rows, cols, seed=rows * 3 + cols, kind="offset")
    y1 = run_gpu(x)
    check_parity(x, y1, f"{rows}x{cols}")
    y2 = run_gpu(x)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("rows,cols", [(3, 1048580), (2, 2097152), (1, 1048576), (5, 524292)])
def test_split_rows_large_chunks(rows, cols):
    """Rows past 64 chunks of 16384 columns use 32768-column chunks (with
    128-bit access; a ragged 128-bit tail at 1048580); 524292 columns take
    33 chunks of 16384."""
    log(f"[parity] split rows, large chunks {rows}x{cols}")
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == "split_row" and p["launches"] == 1
    x = workloads.random_logits(rows, cols, seed=cols % 1000, kind="offset")
    check_parity(x, run_gpu(x), f"{rows}x{cols}")


def test_split_rows_two_pass_fallback():
    """A row longer than 64 one-pass chunks takes the two-pass path."""
    log("[parity] split rows, two-pass fallback")
    cols = 64 * 32768 + 1
    p = sm.softmax_plan(1, cols)
    assert p["kernel_name"] == "split_row" and p["launches"] == 2
    x = workloads.random_logits(1, cols, seed=6, kind="normal")
    check_parity(x, run_gpu(x), "1x2097153")
    x = workloads.random_logits(3, cols, seed=7, kind="clip_heavy")
    check_parity(x, run_gpu(x), "3x2097153 clip-heavy")
    # With 32-bit access (cols % 4 != 0) rows past 64 small chunks take the
    # two-pass path rather than the large chunks.
    cols = 1048577
    p = sm.softmax_plan(3, cols)
    assert p["kernel_name"] == "split_row" and p["launches"] == 2 and p["vec_width"] == 1
    x = workloads.random_logits(3, cols, seed=8, kind="offset")
    check_parity(x, run_gpu(x), "3x1048577 32-bit")


@pytest.mark.parametrize("rows,cols", [(115200, 50), (4096, 1000), (512, 32768), (64, 262144)])
def test_graph_capture_replays(rows, cols):
    """softmax_fwd captured in a HIP graph: every replay, with eager work and
    synchronisation in between, matches the eager output bit for bit."""
    torch = _torch()
    log(f"[parity] graph capture {rows}x{cols}")
    x = workloads.random_logits(rows, cols, seed=9, kind="clip_heavy" if cols < 1000 else "normal")
    xt = torch.from_numpy(x).to(_dev())
    y_eager = sm.softmax_fwd(xt)
    torch.cuda.synchronize()
    want = y_eager.cpu().numpy()
    check_parity(x, want, f"eager {rows}x{cols}")
    yg = torch.empty_like(xt)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        sm.softmax_fwd(xt, out=yg, stream=s)
    for rep in range(3):
        yg.fill_(-1.0)
        sm.softmax_fwd(xt, out=y_eager)   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = yg.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), rep


def test_exchange_at_rest_after_split_rows():
    """After the split-row tests above (one-pass, several launches, large
    chunks, two passes, graph replays): no exchange wait gave up, and every
    region of the table is back at rest."""
    torch = _torch()
    x = workloads.random_logits(9, 300000, seed=12, kind="offset")
    check_parity(x, run_gpu(x), "9x300000")
    torch.cuda.synchronize()
    st = sm.softmax_exchange_status()
    log(f"[parity] exchange status {st}")
    assert st == {"join_give_ups": 0, "wait_give_ups": 0, "entries_in_use": 0}, st
