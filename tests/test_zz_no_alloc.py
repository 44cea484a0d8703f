"""kkm_iterate_noalloc: the clustering loop on the library's static device
scratch, for callers that cannot allocate.  Checked through the C ABI against
kkm_iterate (same kernels, scratch the context allocates) on two calls in a
row, the second with a smaller input, in every storage mode; then the size
limit, refused on the host before anything is enqueued."""
import numpy as np
import pytest

from gpu_helpers import TOL, Engine
from paper_2601_17136_amd import datagen

pytestmark = pytest.mark.gpu


def _torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU test on a machine without a GPU")
    return torch


def _both(eng, cl0, k, iters, tol):
    """(final ids, done, J history) of kkm_iterate and of kkm_iterate_noalloc."""
    torch = _torch_cuda()
    kkm = eng.kkm
    Va = torch.from_numpy(cl0).cuda()
    Vb = torch.from_numpy(cl0).cuda()
    ita, ha = kkm.kkm_iterate(eng.ctx, Va, k, iters, tol)
    itb, hb = kkm.kkm_iterate_noalloc(eng.ctx, Vb, k, iters, tol)
    return (Va.cpu().numpy(), ita, ha), (Vb.cpu().numpy(), itb, hb)


# two calls in a row, the second smaller; the second pair with more than 16
# labels (the packed SpMM's 16-tile segments and two label blocks)
SIZES = [((2600, 24, 10, 6, -1.0, 41), (700, 9, 6, 5, 0.0, 42)),
         ((5000, 12, 24, 4, -1.0, 43), (4500, 12, 20, 3, -1.0, 44))]


@pytest.mark.parametrize("sizes", range(len(SIZES)))
@pytest.mark.parametrize("mode", ["resident", "packed", "onthefly"])
def test_noalloc_matches_iterate_twice_smaller_second(mode, sizes):
    _torch_cuda()
    for n, d, k, iters, tol, seed in SIZES[sizes]:
        X = datagen.make_points(2, n=n, d=d)[0]
        cl0 = datagen.random_init(n, k, seed)
        print(f"[gpu] noalloc {mode} n={n} d={d} k={k} iters={iters} tol={tol}", flush=True)
        with Engine(X, "gauss", 1.0 / d, mode=mode) as eng:
            (ca, ia, ha), (cb, ib, hb) = _both(eng, cl0, k, iters, tol)
        assert ia == ib >= 1
        np.testing.assert_array_equal(ca, cb)
        assert np.max(np.abs(ha - hb) / np.abs(ha)) <= TOL
        np.testing.assert_array_equal(ha, hb)     # the same kernels in the same order


def test_noalloc_leaves_the_context_scratch_alone():
    """kkm_iterate, then the static-scratch call with another k, then kkm_iterate
    again: the context's own scratch (sized for the first k) still serves."""
    _torch_cuda()
    X = datagen.make_points(5, n=1500, d=16)[0]
    cl5 = datagen.random_init(1500, 5, 43)
    cl3 = datagen.random_init(1500, 3, 44)
    with Engine(X, "gauss", 1.0 / 16, mode="packed") as eng:
        first = _both(eng, cl5, 5, 4, -1.0)
        other = _both(eng, cl3, 3, 4, -1.0)
        again = _both(eng, cl5, 5, 4, -1.0)
    for (ca, ia, ha), (cb, ib, hb) in (first, other, again):
        assert ia == ib and np.array_equal(ca, cb) and np.array_equal(ha, hb)
    np.testing.assert_array_equal(first[0][0], again[0][0])


def test_noalloc_refuses_what_does_not_fit():
    """Scratch beyond the static array is refused with KKM_ERR_ARG; the context
    stays usable and kkm_iterate still runs the same problem."""
    torch = _torch_cuda()
    X = datagen.make_points(2, n=20000, d=8)[0]
    cl0 = datagen.random_init(20000, 10, 45)
    with Engine(X, "gauss", 1.0 / 8, mode="onthefly") as eng:
        kkm = eng.kkm
        V = torch.from_numpy(cl0).cuda()
        with pytest.raises(kkm.KKMError) as e:   # k = 1024: each row-side segment partial is 1024 x 20096 floats (82 MB)
            kkm.kkm_iterate_noalloc(eng.ctx, V, 1024, 2, -1.0)
        assert e.value.code == kkm.KKM_ERR_ARG and "static" in str(e.value)
        np.testing.assert_array_equal(V.cpu().numpy(), cl0)      # untouched
        it, _ = kkm.kkm_iterate(eng.ctx, V, 10, 2, -1.0)
        assert it == 2
        V2 = torch.from_numpy(datagen.random_init(20000, 2, 46)).cuda()
        it, _ = kkm.kkm_iterate_noalloc(eng.ctx, V2, 2, 2, -1.0)   # k = 2 fits (about 31 MB)
        assert it == 2
