"""The achievable-peak microbenchmarks behind `bench.py --peaks`, checked on
small inputs: the streaming read returns exact per-workgroup sums of what
the streaming write stored (integers in fp32, exact at these sizes), and
the MFMA loop reports its flop count and finite results."""
import math

import pytest

from paper_2601_17136_amd import kkm

pytestmark = pytest.mark.gpu


@pytest.fixture()
def ctx():
    import torch
    torch.cuda.set_device(0)
    c = kkm.kkm_create(kkm.current_stream_handle())
    yield c
    kkm.kkm_destroy(c)


@pytest.mark.parametrize("numel", [4, 1000, 1 << 24, (1 << 24) + 12])
def test_write_then_read_sums(ctx, numel):
    import torch
    print(f"[gpu] peaks write/read numel={numel}", flush=True)
    buf = torch.zeros(numel, dtype=torch.float32, device="cuda")
    sums = torch.full((kkm.PEAK_READ_GROUPS,), -1.0, dtype=torch.float32, device="cuda")
    assert kkm.kkm_peak_write(ctx, buf, 2.0, 2) > 0
    assert bool((buf == 2.0).all())
    assert kkm.kkm_peak_read(ctx, buf, sums, 2) > 0
    assert float(sums.double().sum().item()) == 2.0 * numel


def test_mfma_loop(ctx):
    import torch
    print("[gpu] peaks mfma", flush=True)
    out = torch.full((4096,), math.nan, dtype=torch.float32, device="cuda")
    ms, flops = kkm.kkm_peak_mfma(ctx, 64, out, 2)
    assert ms > 0 and flops == 1024 * 4 * 4 * 4096 * 64
    assert bool(torch.isfinite(out).all())


def test_rejects_unaligned_sizes(ctx):
    import torch
    buf = torch.zeros(5, dtype=torch.float32, device="cuda")
    sums = torch.zeros(kkm.PEAK_READ_GROUPS, dtype=torch.float32, device="cuda")
    with pytest.raises(kkm.KKMError):
        kkm.kkm_peak_read(ctx, buf, sums, 1)
