"""The measurement aids: the MFMA-rate probe runs, reports the operation
count of its closed form, and its clock stamps read a plausible shader clock;
the device-wide meeting probe counts every arrival and nobody gives up."""
import pytest

from _util import announce

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [0, 1], ids=["16x16x64", "32x32x32"])
def test_mfma_probe_runs_and_stamps_a_clock(shape):
    import torch
    from paper_2202_06819_amd import qconv
    blocks, iters = 64, 256
    announce(f"mfma probe shape={shape} blocks={blocks} iters={iters}")
    dev = torch.device("cuda:0")
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=dev)
    stamps = torch.zeros(blocks * 4, dtype=torch.int64, device=dev)
    ops = qconv.probe_mfma_i8(blocks, iters, sink, stamps, shape=shape)
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


@pytest.mark.parametrize("two_level", [False, True])
def test_grid_meet_probe_counts_every_arrival(two_level):
    # every workgroup arrives once per meeting and nobody gives up waiting; the
    # counters start from zero on each launch (a second launch ends at the same values)
    import torch
    from paper_2202_06819_amd import qconv
    dev = torch.device("cuda:0")
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    state = torch.zeros(qconv.ProbeGridMeetCall.STATE_ELEMS, dtype=torch.int32, device=dev)
    for blocks, rounds in ((4, 3), (13, 2), (cus, 5), (cus, 0)):
        announce(f"grid meeting probe blocks={blocks} rounds={rounds} two_level={two_level}")
        for _ in range(2):
            qconv.ProbeGridMeetCall(blocks, rounds, state, two_level)()
            torch.cuda.synchronize()
            s = state.cpu()
            assert int(s[0]) == rounds * (min(blocks, 8) if two_level else blocks)
            assert int(s[144]) == 0
            if two_level:
                for g in range(8):
                    assert int(s[16 * (g + 1)]) == rounds * len(range(g, blocks, 8))
    with pytest.raises(qconv.QConvError):
        qconv.ProbeGridMeetCall(cus + 1, 1, state)()
