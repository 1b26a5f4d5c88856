"""Batched FFT parity: the HIP kernels through the C ABI against the fp64 oracle.

Tolerances (relative L2 per transform, maximised over the batch): 1e-5 for
FP32 storage, 3e-3 for FP16 storage on the FP16-rounded input.  The paper's
own kernels reach 3.6e-7 .. 8.2e-7 (FP32) and 73.6 dB SQNR, about 2.1e-4 (FP16)
(Sections III, VI and VII), so both bounds carry over ten times margin.
"""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import log, rel_rows, to_dev, to_host, widen

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "fp16": 3e-3}
SIZES = [1024, 2048, 4096, 8192, 16384]


@pytest.fixture(scope="module")
def api():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2609_32237_amd import _lib, torch_api

    return torch_api


def storage_code(storage):
    return 0 if storage == "fp32" else 1


def run_plan(api, x_host, n, batch, stride, dist, storage, direction, inplace=False):
    import torch

    xd = to_dev(x_host)
    # out of place, the output starts as a copy of the input so that entries the
    # layout does not cover can be checked for being left alone
    out = xd if inplace else xd.clone()
    plan = api.Plan(n, batch, stride, dist, storage_code(storage), direction)
    plan.execute(xd, out)
    torch.cuda.synchronize()
    plan.close()
    return to_host(out)


def make_input(storage, shape, seed):
    if storage == "fp32":
        b, n = shape
        return workloads.uniform_complex(b, n, seed)
    return workloads.uniform_complex(shape[0], shape[1], seed, "fp16")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("storage", ["fp32", "fp16"])
@pytest.mark.parametrize("direction", [-1, 1])
@pytest.mark.parametrize("batch", [1, 3, 257])
def test_rows(api, n, storage, direction, batch):
    """Contiguous rows, ragged batches (257 is not a multiple of any workgroup's transform count)."""
    log(f"rows n={n} {storage} dir={direction} batch={batch}")
    x = make_input(storage, (batch, n), 100 + n + batch)
    y = widen(run_plan(api, x, n, batch, 1, n, storage, direction))
    ref = oracle.fft(x, direction)
    err = rel_rows(y, ref)
    assert err.max() < TOL[storage], err.max()


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("storage", ["fp32", "fp16"])
@pytest.mark.parametrize("direction", [-1, 1])
@pytest.mark.parametrize("cols, width", [(1, 1), (5, 5), (37, 40)])
def test_columns(api, n, storage, direction, cols, width):
    """Columns of a row-major (n, width) matrix: stride = width, dist = 1.
    Columns beyond ``cols`` must be left untouched."""
    log(f"cols n={n} {storage} dir={direction} cols={cols} width={width}")
    m = make_input(storage, (n, width), 200 + n + cols)
    y = run_plan(api, m, n, cols, width, 1, storage, direction)
    ref = oracle.fft_layout(m, n, cols, width, 1, direction).reshape(n, width)
    err = rel_rows(widen(y).T[:cols], ref.T[:cols])
    assert err.max() < TOL[storage], err.max()
    if width > cols:
        assert np.array_equal(y[:, cols:], m[:, cols:])


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("storage", ["fp32", "fp16"])
def test_in_place(api, n, storage):
    log(f"in-place n={n} {storage}")
    x = make_input(storage, (9, n), 300 + n)
    y = widen(run_plan(api, x, n, 9, 1, n, storage, -1, inplace=True))
    assert rel_rows(y, oracle.fft(x)).max() < TOL[storage]


@pytest.mark.parametrize("n", [8192, 16384])
@pytest.mark.parametrize("storage", ["fp32", "fp16"])
def test_long_columns_in_and_out_of_place(api, n, storage):
    """Long interleaved columns run as two passes of short columns out of
    place and as one pass in place; both against the oracle, ragged width."""
    log(f"long columns n={n} {storage}")
    cols, width = 70, 72
    m = make_input(storage, (n, width), 700 + n)
    ref = oracle.fft_layout(m, n, cols, width, 1, -1).reshape(n, width)
    for inplace in (False, True):
        y = run_plan(api, m, n, cols, width, 1, storage, -1, inplace=inplace)
        err = rel_rows(widen(y).T[:cols], ref.T[:cols])
        assert err.max() < TOL[storage], (inplace, err.max())
        assert np.array_equal(y[:, cols:], m[:, cols:])


@pytest.mark.parametrize("n", [1024, 4096, 16384])
def test_padded_rows_and_strided_blocks(api, n):
    """dist > n leaves the gaps alone; stride 3 with dist 3n uses the column kernel on blocks."""
    log(f"padded/strided n={n}")
    batch, dist = 5, n + 7
    buf = workloads.uniform_complex(1, batch * dist, 400 + n)[0]
    y = run_plan(api, buf, n, batch, 1, dist, "fp32", -1)
    ref = oracle.fft_layout(buf, n, batch, 1, dist, -1)
    yb, rb = y.reshape(batch, dist), ref.reshape(batch, dist)
    assert rel_rows(yb[:, :n], rb[:, :n]).max() < 1e-5
    assert np.array_equal(yb[:, n:], buf.reshape(batch, dist)[:, n:])
    buf = workloads.uniform_complex(1, batch * 3 * n, 500 + n)[0]
    y = run_plan(api, buf, n, batch, 3, 3 * n, "fp32", 1)
    ref = oracle.fft_layout(buf, n, batch, 3, 3 * n, 1)
    yb, rb = y.reshape(batch, n, 3), ref.reshape(batch, n, 3)
    assert rel_rows(yb[:, :, 0], rb[:, :, 0]).max() < 1e-5
    assert np.array_equal(yb[:, :, 1:], buf.reshape(batch, n, 3)[:, :, 1:])


@pytest.mark.parametrize("n", SIZES)
def test_closed_forms(api, n):
    """Impulse -> exp(-2 pi i k n0 / N); tone -> N delta[k - f]; constant -> N delta[k]."""
    log(f"closed forms n={n}")
    k = np.arange(n)
    n0, f = n // 3, n // 5
    x = np.zeros((3, n), np.complex64)
    x[0, n0] = 1
    x[1] = np.exp(2j * np.pi * ((f * k) % n) / n)
    x[2] = 1
    y = widen(run_plan(api, x, n, 3, 1, n, "fp32", -1))
    want = np.zeros((3, n), complex)
    want[0] = np.exp(-2j * np.pi * ((k * n0) % n) / n)
    want[1, f] = n
    want[2, 0] = n
    assert np.abs(y[0] - want[0]).max() < 1e-6
    assert np.abs(y[1] - want[1]).max() < 1e-6 * n
    assert np.abs(y[2] - want[2]).max() < 1e-6 * n


def test_non_default_stream(api):
    import torch

    log("non-default stream")
    x = workloads.uniform_complex(64, 4096, 7)
    xd = to_dev(x)
    out = torch.empty_like(xd)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        api.fft(xd, -1, out=out)
    s.synchronize()
    assert rel_rows(widen(to_host(out)), oracle.fft(x)).max() < 1e-5


def test_misaligned_pointer(api):
    import torch

    from paper_2609_32237_amd import _lib

    buf = torch.zeros(4096 * 2 + 1, dtype=torch.complex64, device="cuda")
    plan = _lib.fft_plan_create(4096, 1, 1, 4096, 0, -1)
    try:
        rc = _lib.lib.fft_execute(plan, buf.data_ptr() + 4, buf.data_ptr(), None)
        assert rc == _lib.FFT_EALIGN
        rc = _lib.lib.fft_execute(plan, buf.data_ptr(), buf.data_ptr() + 4, None)
        assert rc == _lib.FFT_EALIGN
    finally:
        _lib.fft_plan_destroy(plan)


# --------------------------------------------------------------------------
# The benchmark workloads at full size, in the launch configuration the
# benchmark times: every transform against the oracle, element by element
# (the pass criterion is the per-transform error maximised over the batch,
# Section III), with Parseval on every transform as an extra check.
# --------------------------------------------------------------------------

FULL = ["fft_n1024_b64_fp32", "fft_n4096_b32768_fp32", "fft_n8192_b16384_fp32", "fft_n16384_b8192_fp32",
        "fft_n16384_b16384_fp16"]


def parseval_ratio(x, y):
    """sum |Y|^2 / (N sum |x|^2) per transform, accumulated in fp64."""
    x, y = widen(x), widen(y)
    n = x.shape[-1]
    return (np.abs(y) ** 2).sum(-1) / (n * (np.abs(x) ** 2).sum(-1))


def compare_all(x, y, sign, chunk_points=1 << 24):
    """Per-transform relative L2 error of every transform of y against the
    oracle on x, in chunks of about 2^24 points (256 MiB of complex128)."""
    batch, n = x.shape[0], x.shape[1]
    step = max(1, chunk_points // n)
    err = np.empty(batch)
    num = den = 0.0
    for s in range(0, batch, step):
        ref = oracle.fft(x[s:s + step], sign)
        got = widen(y[s:s + step])
        d = (np.abs(got - ref) ** 2).sum(-1)
        r = (np.abs(ref) ** 2).sum(-1)
        err[s:s + step] = np.sqrt(d / r)
        num += d.sum()
        den += r.sum()
    return err, float(np.sqrt(num / den))


@pytest.mark.parametrize("name", FULL)
def test_full_size_workload(api, name):
    import torch

    w = workloads.FFT_WORKLOADS[name]
    n, batch, storage = w["n"], w["batch"], w["storage"]
    log(f"full-size {name}")
    x = workloads.fft_workload(name)
    xd = to_dev(x)
    out = torch.empty_like(xd)
    plan = api.Plan(n, batch, 1, n, storage_code(storage), -1)
    plan.execute(xd, out)
    torch.cuda.synchronize()
    y = to_host(out)
    err, glob = compare_all(x, y, -1)
    worst = int(err.argmax())
    log(f"  {name}: all {batch} transforms, max rel {err.max():.3e} (transform {worst}), "
        f"median {np.median(err):.3e}, global {glob:.3e}, SQNR {-20 * np.log10(glob):.1f} dB")
    assert err.max() < TOL[storage], (worst, err.max())
    # Parseval on every transform, in chunks
    tol = 2e-5 if storage == "fp32" else 5e-3
    for s in range(0, batch, 2048):
        r = parseval_ratio(x[s:s + 2048], y[s:s + 2048])
        assert np.abs(r - 1).max() < tol, (s, np.abs(r - 1).max())
    if name == "fft_n4096_b32768_fp32":
        # round trip: inverse of the forward output equals N x, every transform
        inv = api.Plan(n, batch, 1, n, 0, 1)
        back = torch.empty_like(xd)
        inv.execute(out, back)
        torch.cuda.synchronize()
        b = to_host(back)
        errs = np.empty(batch)
        for s in range(0, batch, 4096):
            errs[s:s + 4096] = rel_rows(widen(b[s:s + 4096]) / n, x[s:s + 4096].astype(np.complex128))
        log(f"  round trip: max rel {errs.max():.3e}")
        assert errs.max() < 1e-5
        # the inverse itself against the oracle on the forward output, every transform
        e_inv, _ = compare_all(y, b, 1)
        assert e_inv.max() < 1e-5, e_inv.max()
        inv.close()
    plan.close()


def test_columns_spanning_more_than_2gib(api):
    """Columns whose workgroup span exceeds 2 GiB take the 64-bit addressing path.
    A (16384, 16400) complex64 matrix (2.1 GB) on the GPU; three columns are
    transformed, the column next to them must stay untouched."""
    import torch

    n, width, cols = 16384, 16400, 3
    log("wide columns 16384 x 16400")
    m = torch.zeros(n, width, dtype=torch.complex64, device="cuda")
    data = workloads.uniform_complex(cols + 1, n, 901)  # column-major sample
    m[:, :cols + 1] = torch.from_numpy(np.ascontiguousarray(data.T)).cuda()
    plan = api.Plan(n, cols, width, 1, 0, -1)
    plan.execute(m, m)
    torch.cuda.synchronize()
    plan.close()
    got = m[:, :cols + 1].cpu().numpy().T
    del m
    torch.cuda.empty_cache()
    err = rel_rows(widen(got[:cols]), oracle.fft(data[:cols]))
    assert err.max() < 1e-5
    assert np.array_equal(got[cols], data[cols])


@pytest.mark.parametrize("order", ["range_first", "azimuth_first"])
def test_sar_reference_buffers_in_either_order(api, order):
    """The reference-spectrum launch addresses both references from one base with
    a signed gap; it must work whichever buffer comes first in memory."""
    import torch

    log(f"sar references {order}")
    sc = workloads.sar_scene(n_az=1024, n_rg=1024, n_targets=3, len_rg=128, len_az=64, min_sep=16, seed=12)
    both = torch.empty(2, 1024, dtype=torch.complex64, device="cuda")
    r_i, a_i = (0, 1) if order == "range_first" else (1, 0)
    both[r_i] = torch.from_numpy(sc.range_ref).cuda()
    both[a_i] = torch.from_numpy(sc.az_ref).cuda()
    img = api.sar_form_image(to_dev(sc.raw), both[r_i], both[a_i], 0)
    torch.cuda.synchronize()
    ref = oracle.sar_chain(sc.raw, sc.range_ref, sc.az_ref)
    got = to_host(img).astype(np.complex128)
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) < 1e-5


def test_one_plan_from_several_host_threads(api):
    """One plan executed concurrently from four host threads, each on its own
    stream and buffers (the plan is read-only after creation, the per-device
    tables are shared), against the oracle, while each thread also creates,
    uses and destroys a plan of its own."""
    import threading

    import torch

    n, batch = 4096, 256
    xs = [workloads.uniform_complex(batch, n, 600 + i) for i in range(4)]
    refs = [oracle.fft(x) for x in xs]
    p = api.Plan(n, batch, 1, n, 0, -1)
    results, errors = [None] * 4, []

    def work(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                xd = torch.from_numpy(xs[i]).to("cuda", non_blocking=False)
                yd = torch.empty_like(xd)
                for _ in range(5):
                    p.execute(xd, yd, stream=s)
                q = api.Plan(2048, 8, 1, 2048, 0, -1)
                q.execute(xd[:8, :2048].contiguous(), torch.empty(8, 2048, dtype=torch.complex64, device="cuda"),
                          stream=s)
                s.synchronize()
                q.close()
                results[i] = yd.cpu().numpy()
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(repr(e))

    log("plan from four host threads")
    ts = [threading.Thread(target=work, args=(i,)) for i in range(4)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    p.close()
    assert not errors, errors
    for i in range(4):
        assert rel_rows(results[i].astype(np.complex128), refs[i]).max() < TOL["fp32"], i
