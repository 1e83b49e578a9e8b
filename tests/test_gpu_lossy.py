"""The lossy steps of Sec. 5.4 on the GPU (lmgc_sparsify_topk,
lmgc_quantize_linear, lmgc_sign_pack) against the oracle, bit for bit: the
full 8M-value lossy workload at 50/25/10 percent and 16/8/1-bit, ragged and
tiny sizes, heavy ties across chunks, signed zeros, NaN/inf, in place, and
the error paths."""
import numpy as np
import pytest

from gpu_util import log
from oracle import lossy as olossy
from paper_2409_17836_amd import binding as B
from synth import get_workload, parse_lossy
from synth.gen import gen_values, workload_values

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _host(t, dtype=None):
    import torch
    torch.cuda.synchronize()
    a = t.cpu().numpy()
    return a.view(dtype) if dtype is not None else a


@pytest.fixture(scope="module")
def big():
    w = get_workload("lossy7b")
    return workload_values(w)                                  # 8M x N(0, 1e-3^2)


# ----------------------------------------------------------- sparsification --
@pytest.mark.parametrize("pct", [50, 25, 10])
def test_sparsify_full_size(big, pct):
    k = olossy.keep_count(big.size, pct)
    log(f"sparsify {big.size} values, keep {k}")
    got = _host(B.sparsify_topk(_dev(big), k))
    want = olossy.sparsify_topk(big, k)
    assert got.tobytes() == want.tobytes()


def _tie_vector(n, seed, levels=5):
    rng = np.random.default_rng(seed)
    v = (rng.integers(-levels, levels + 1, n) * 0.125).astype(np.float32)
    v[rng.random(n) < 0.05] = -0.0
    return v


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1023, 1024, 1025, 4097, 100003])
def test_sparsify_ties_and_ragged_sizes(n):
    v = _tie_vector(n, n)
    dv = _dev(v)
    for k in sorted({0, 1, n // 3, n // 2, max(n - 1, 0), n, n + 5}):
        got = _host(B.sparsify_topk(dv, k))
        assert got.tobytes() == olossy.sparsify_topk(v, k).tobytes(), (n, k)


def test_sparsify_tie_set_spanning_all_chunks():
    """3M values with 7 magnitudes: the threshold key is shared by ~430k
    values in every chunk, so the kept ones depend on the cross-chunk ranks."""
    n = 3 * (1 << 20) + 17
    v = _tie_vector(n, 11, levels=3)
    dv = _dev(v)
    for k in (1, n // 7, n // 2 + 1, n - 3):
        got = _host(B.sparsify_topk(dv, k))
        assert got.tobytes() == olossy.sparsify_topk(v, k).tobytes(), k


def test_sparsify_in_place_and_special_values():
    v = gen_values("laplace:1e-3", 50000, 2)
    v[[5, 77, 901]] = [np.inf, -np.inf, np.nan]
    v[[6, 7]] = [0.0, -0.0]
    for k in (1, 2, 3, 4, 25000):
        dv = _dev(v)
        out = B.sparsify_topk(dv, k, out=dv)                    # in place
        assert out.data_ptr() == dv.data_ptr()
        assert _host(dv).tobytes() == olossy.sparsify_topk(v, k).tobytes(), k


def test_sparsify_errors():
    import torch
    dv = _dev(np.ones(100, np.float32))
    with pytest.raises(B.LMGCError) as e:
        B.sparsify_topk(dv, -1)
    assert e.value.code == -1
    with pytest.raises(B.LMGCError) as e:
        B.sparsify_topk(dv[:50], 3, out=dv[4:54])               # overlapping, not equal
    assert e.value.code == -1
    ws = torch.empty(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.LMGCError) as e:
        B.sparsify_topk(dv, 3, ws=ws)
    assert e.value.code == -4


# ------------------------------------------------------------- quantisation --
@pytest.mark.parametrize("bits", [16, 8, 1, 3, 12])
def test_quantize_full_size(big, bits):
    v = olossy.sparsify_topk(big, olossy.keep_count(big.size, 10)) if bits == 8 else big
    q, mn, mx = B.quantize_linear(_dev(v), bits)
    dt = np.uint8 if bits <= 8 else np.uint16
    got = _host(q, dt)
    want, wmn, wmx = olossy.quantize_linear(v, bits)
    assert (mn, mx) == (wmn, wmx)
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]


@pytest.mark.parametrize("n", [1, 2, 5, 1027, 65537])
def test_quantize_ragged_sizes(n):
    v = gen_values("mixture:1e-4:0.05:1e-2", n, n)
    for bits in (8, 16):
        q, _, _ = B.quantize_linear(_dev(v), bits)
        got = _host(q, np.uint8 if bits <= 8 else np.uint16)
        assert np.array_equal(got, olossy.quantize_linear(v, bits)[0]), (n, bits)


def test_quantize_constant_vector_and_errors():
    q, mn, mx = B.quantize_linear(_dev(np.full(1000, 0.25, np.float32)), 8)
    assert not _host(q).any() and mn == mx == 0.25
    for bad in (np.nan, np.inf, -np.inf):
        v = np.ones(5000, np.float32)
        v[4321] = bad
        with pytest.raises(B.LMGCError) as e:
            B.quantize_linear(_dev(v), 8)
        assert e.value.code == -1
    for bits in (0, 17):
        with pytest.raises(B.LMGCError):
            B.quantize_linear(_dev(np.ones(8, np.float32)), bits)


# ------------------------------------------------------------- sign packing --
@pytest.mark.parametrize("n", [1, 7, 8, 9, 31, 1000003])
def test_sign_pack_sizes(n):
    v = gen_values("normal:1.0", n, n)
    v[: min(n, 3)] = [-0.0, 0.0, np.nan][: min(n, 3)]
    got = _host(B.sign_pack(_dev(v)))
    assert got.tobytes() == olossy.sign_pack(v).tobytes()


def test_sign_pack_full_size(big):
    got = _host(B.sign_pack(_dev(big)))
    assert got.tobytes() == olossy.sign_pack(big).tobytes()


# ---------------------------------------------------------------- workload --
def test_lossy_workload_preparation(big):
    """The 8M-value lossy workload: top 10 % then 8-bit indices, on the GPU."""
    w = get_workload("lossy7b")
    got = _host(B.lossy_prepare(_dev(big), parse_lossy(w.lossy)))
    want = olossy.prepare(big, w.lossy)
    assert got.dtype == want.dtype and got.tobytes() == want.tobytes()
