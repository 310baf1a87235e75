"""gt_compare_noalloc (the comparison with its result words in a static
device array, for callers that cannot allocate) against gt_compare, through
the C ABI: identical results on two calls in a row, the second on a smaller
input, so the array's previous contents must not leak into the next call."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gt():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_1909_10616_amd import gemmtune
    gemmtune.lib()
    return gemmtune


def _pair(n, seed, bump):
    g = torch.Generator().manual_seed(seed)
    R = torch.randn(n, generator=g)
    C = R + 1e-4 * torch.randn(n, generator=g)
    C[n // 3] += bump
    return C.cuda(), R.cuda()


def test_noalloc_matches_compare_on_consecutive_calls(gt):
    cases = [(1 << 22, 0, 0.5), (1 << 12, 1, 0.0), (777, 2, 3.0), (1, 3, 0.0)]
    got = []
    for n, seed, bump in cases:
        C, R = _pair(n, seed, bump)
        want = gt.gt_compare(C, R)
        have = gt.gt_compare_noalloc(C, R)
        print(f"n={n}: gt_compare {want!r} gt_compare_noalloc {have!r}", flush=True)
        assert have == want
        got.append(have)
    # the large first call's maximum must not survive into the later ones
    assert got[0] > got[1] and got[2] > got[1]


def test_noalloc_rejects_bad_arguments(gt):
    import ctypes
    rel = ctypes.c_double()
    C = torch.zeros(4, device="cuda")
    GT_EINVAL = -1
    assert gt.lib().gt_compare_noalloc(C.data_ptr(), C.data_ptr(), 0, None,
                                       ctypes.byref(rel)) == GT_EINVAL
    assert gt.lib().gt_compare_noalloc(None, C.data_ptr(), 4, None, ctypes.byref(rel)) == GT_EINVAL
