"""The MFMA-rate probe (a measurement aid): it runs, reports the operation
count of its closed form, and its clock stamps read a plausible shader clock."""
import pytest

from _util import announce

pytestmark = pytest.mark.gpu


def test_mfma_probe_runs_and_stamps_a_clock():
    import torch
    from paper_2202_06819_amd import qconv
    blocks, iters = 64, 256
    announce(f"mfma probe blocks={blocks} iters={iters}")
    dev = torch.device("cuda:0")
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=dev)
    stamps = torch.zeros(blocks * 4, dtype=torch.int64, device=dev)
    ops = qconv.probe_mfma_i8(blocks, iters, sink, stamps)
    torch.cuda.synchronize()
    assert ops == blocks * 4 * iters * 8 * 2 * 16 * 16 * 64
    st = stamps.view(blocks, 4).cpu()
    cycles = (st[:, 1] - st[:, 0]).double()
    ns = (st[:, 3] - st[:, 2]).double() * 10.0
    assert bool((cycles > 0).all()) and bool((ns > 0).all())
    ghz = (cycles / ns).median().item()
    assert 0.5 < ghz < 3.5, ghz
    # every wave ran its 8 * iters MFMAs: at most 2048 int8 ops per clock per SIMD
    assert cycles.min().item() >= iters * 8 * 16 * 0.5
