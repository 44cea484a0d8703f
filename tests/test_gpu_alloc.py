"""A large K (8.5 GB, allocated as contiguous memory) within a budget of
exactly what kkm_plan asks for, and with the default budget.  kkm_plan counts
K, the staged points and the iteration scratch; the Gaussian build's fix-up
list uses spare room while building and gives it up to the first update's
scratch when the budget has no room for both.  Both contexts must stay within
their budget, report the same fix-up count, and give the same matrix (sampled
rows against the oracle) and the same update, bitwise, also after a rebuild.
"""
import numpy as np
import pytest

from gpu_helpers import TOL, Engine, rowscaled_err
from paper_2601_17136_amd import datagen

pytestmark = pytest.mark.gpu

N, D, K = 46000, 8, 5  # full fp32 K: 46000 x 46016 x 4 B = 8.47 GB


def test_large_k_within_the_planned_budget(oracle):
    torch = pytest.importorskip("torch")
    assert torch.cuda.is_available()
    from paper_2601_17136_amd import kkm
    X = datagen.make_points(2, n=N, d=D)[0]
    cl = datagen.random_init(N, K, 31)
    gamma = 1.0 / D
    mode, need = kkm.kkm_plan(N, D, K, kkm.KKM_GAUSS, 1 << 40, kkm.KKM_MODE_RESIDENT)
    assert mode == kkm.KKM_MODE_RESIDENT and need > 8e9
    print(f"[gpu] large K: n={N} d={D}, planned {need} bytes", flush=True)
    kern = oracle.Kernel("gauss", gamma, 0.0, 1)
    rows = np.array([0, 1, 127, 128, 20011, N - 2, N - 1])
    outs, fix = [], []
    for budget in (need + 4096, 0):  # the plan, then the default
        with Engine(X, "gauss", gamma, mode="resident", mem_budget=budget) as eng:
            # with the planned budget the first update's scratch takes the room
            # of the build's fix-up list, which is released after its counts are read
            outs.append(eng.step(cl, K))
            info = eng.info()
            assert info["bytes_K"] == N * (-(-N // 64) * 64) * 4
            if budget:
                assert info["bytes_total"] <= budget
            fix.append(info["fixups"])
            Kr = np.stack([eng.K_rows(int(r), int(r) + 1)[0] for r in rows])
            err = rowscaled_err(Kr, kern.block(X, rows, None))
            assert err <= TOL, f"K rows error {err:.3e} (budget {budget})"
            # a rebuild on the same context makes the list again; the next update
            # releases it again and gives the same result
            kkm.kkm_build_kernel(eng.ctx, eng.X, N, D, kkm.KKM_GAUSS,
                                 kkm.make_params(gamma, 0.0, 1, kkm.KKM_MODE_RESIDENT))
            again = eng.step(cl, K)
            assert np.array_equal(again["E"], outs[-1]["E"]) and again["J"] == outs[-1]["J"]
            print(f"[gpu] budget {budget}: {info['bytes_total']} bytes held, fix-ups {info['fixups']}, "
                  f"K rows err {err:.2e}", flush=True)
    assert fix[0] == fix[1] >= 0
    a, b = outs
    for key in ("E", "D", "z", "cl", "counts"):
        assert np.array_equal(a[key], b[key]), key
    assert a["J"] == b["J"]
    assert int(a["counts"].sum()) == N
