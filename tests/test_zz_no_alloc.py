"""lmgc_sparsify_topk_noalloc (the top-k of Sec. 5.4 on the library's own
device scratch, for callers that cannot allocate) against
lmgc_sparsify_topk with a caller workspace, through the C ABI: bitwise equal
on two calls in a row, the second on a smaller vector, so that what the
first call left in the shared scratch (state, histogram, tie counts) would
show if it leaked into the second.  Both vectors carry large tie sets at the
threshold spread over every chunk of the ordered write pass."""
import numpy as np
import pytest

from gpu_util import log
from oracle import lossy as olossy
from paper_2409_17836_amd import binding as B
from synth.gen import gen_values

pytestmark = pytest.mark.gpu


def _vector(n, seed):
    x = gen_values("laplace:1e-3", n, seed)
    # every 7th value shares one magnitude (both signs): a tie set that
    # straddles the threshold of the k chosen below
    t = np.float32(np.sort(np.abs(x))[int(0.9 * n)])
    x[::7] = t
    x[3::14] = -t
    return x


@pytest.mark.parametrize("calls", [[(3_000_017, 0.1, 11), (70_001, 0.25, 12)]])
def test_noalloc_topk_equals_workspace_entry_point(calls):
    import torch
    for n, frac, seed in calls:
        x = _vector(n, seed)
        k = int(frac * n)
        d = torch.from_numpy(x).cuda()
        log(f"noalloc top-k: n={n} k={k} seed={seed}")
        ref = B.sparsify_topk(d, k)
        out = torch.full_like(d, float("nan"))
        B.sparsify_topk_noalloc(d, k, out)
        torch.cuda.synchronize()
        assert torch.equal(ref.view(torch.int32), out.view(torch.int32))
        got = out.cpu().numpy()
        assert got.tobytes() == olossy.sparsify_topk(x, k).tobytes()
        assert int(np.count_nonzero(np.abs(got) > 0)) <= k


def test_noalloc_topk_in_place_and_edges():
    import torch
    x = _vector(5000, 13)
    d = torch.from_numpy(x).cuda()
    ref = B.sparsify_topk(d, 777)
    B.sparsify_topk_noalloc(d, 777, d)             # in place
    B.sparsify_topk_noalloc(d[:0], 3, d[:0])       # empty: nothing to do
    z = torch.from_numpy(x).cuda()
    B.sparsify_topk_noalloc(z, 0, z)               # k = 0 zeroes everything
    torch.cuda.synchronize()
    assert torch.equal(ref.view(torch.int32), d.view(torch.int32))
    assert int(z.view(torch.int32).abs().sum()) == 0
    with pytest.raises(B.LMGCError):
        B.sparsify_topk_noalloc(d, -1, d)
