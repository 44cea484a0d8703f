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


@pytest.mark.parametrize("nchunks,ld,seg", [(1, 128, 128), (3, 1024, 256), (3, 1152, 512), (5, 2176, 2176), (12, 4096, 1024)])
def test_row_pattern_read_sums(ctx, nchunks, ld, seg):
    """Each workgroup's sum is exact (small integers in fp32) and covers exactly its
    chunk's rows over its segment; out-of-range indices read the clamped row."""
    import numpy as np
    import torch
    print(f"[gpu] peaks rows nchunks={nchunks} ld={ld} seg={seg}", flush=True)
    nrows = 300
    vals = (np.arange(nrows) % 5 + 1).astype(np.float32)
    A = torch.from_numpy(np.repeat(vals[:, None], ld, axis=1)).cuda()
    A[:, seg * (ld // seg):] = 1000.0  # columns past the last whole segment are not read
    rng = np.random.default_rng(nchunks)
    rows = rng.integers(0, nrows, nchunks * 128).astype(np.int32)
    rows[0], rows[-1] = -3, nrows + 7
    nseg = ld // seg
    sums = torch.full((nchunks * nseg,), -1.0, dtype=torch.float32, device="cuda")
    assert kkm.kkm_peak_read_rows(ctx, A, torch.from_numpy(rows).cuda(), seg, sums, 2) > 0
    clamped = np.clip(rows, 0, nrows - 1)
    want = np.repeat(vals[clamped].reshape(nchunks, 128).sum(axis=1) * seg, nseg)
    np.testing.assert_array_equal(sums.cpu().numpy(), want.astype(np.float32))


def test_row_pattern_rejects_bad_shapes(ctx):
    import torch
    A = torch.zeros((4, 256), dtype=torch.float32, device="cuda")
    rows = torch.zeros(128, dtype=torch.int32, device="cuda")
    sums = torch.zeros(8, dtype=torch.float32, device="cuda")
    for seg in (0, 100, 384):  # not a multiple of 128, or wider than a row
        with pytest.raises(kkm.KKMError):
            kkm.kkm_peak_read_rows(ctx, A, rows, seg, sums, 1)
