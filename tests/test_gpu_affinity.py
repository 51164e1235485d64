"""GPU: the load-latency probes and the XCD <-> memory affinity they measure.

This is a measurement, not a computation with an oracle: the tests check that
the probes' output has the structure a two-die memory system gives and that
it repeats.  On MI355X in the partition mode nuna_init verifies (one device of
256 compute units in 8 XCDs) the XCDs form two groups (0-3, 4-7), each close
to half of the HBM; every 8 KiB block of memory is near one group.  On any
other device or partitioning the structural tests skip.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def nuna():
    from paper_2608_00867_amd import nuna as n
    n.init()
    info = n.device_info()
    if not (info["map_verified"] and info["cu_count"] == 256 and info["xcd_count"] == 8):
        pytest.skip(f"the two-die structure is asserted for one 8-XCD MI355X device only ({info})")
    return n


@pytest.fixture(scope="module")
def affinity(nuna):
    buf = torch.zeros(64 << 18, dtype=torch.int32, device="cuda")  # 64 MiB
    lat_a, near_a = nuna.memory_affinity(buf, stride=8192, xcds=(0, 4))
    lat_b, near_b = nuna.memory_affinity(buf, stride=8192, xcds=(0, 4))
    lat_c, near_c = nuna.memory_affinity(buf, stride=8192, xcds=(1, 5))
    return lat_a.numpy(), near_a.numpy(), near_b.numpy(), lat_c.numpy(), near_c.numpy()


def test_probe_covers_every_block_with_sane_latencies(affinity):
    lat_a = affinity[0]
    assert lat_a.shape == (2, 8192)
    # cold HBM loads: hundreds to a few thousand shader cycles, never zero
    assert np.all(lat_a > 100) and np.median(lat_a) < 5000


def test_near_group_repeats(affinity):
    _, near_a, near_b, _, _ = affinity
    assert np.mean(near_a == near_b) > 0.9


def test_two_groups_split_memory_with_a_clear_gap(affinity):
    lat_a, near_a, _, _, _ = affinity
    gap = np.abs(lat_a[0] - lat_a[1])
    assert np.median(gap) > 100
    assert 0.3 < near_a.mean() < 0.7


def test_group_members_agree(affinity):
    """XCD 1 sides with XCD 0 and XCD 5 with XCD 4: blocks near XCD 0 are also near XCD 1."""
    _, near_a, _, _, near_c = affinity
    assert np.mean(near_a == near_c) > 0.85


def test_probe_rejects_bad_arguments(nuna):
    buf = torch.zeros(1024, dtype=torch.int32, device="cuda")
    with pytest.raises(nuna.NunaError):
        nuna.probe_load_latency(buf, 4096, 4096, 0)   # line_offset + 4 > stride
    with pytest.raises(nuna.NunaError):
        nuna.probe_load_latency(buf, 256, 0, 8)       # xcd out of range
    with pytest.raises(nuna.NunaError):
        nuna.probe_load_latency(buf, 8192, 0, 0)      # no whole block


@pytest.fixture(scope="module")
def cu_map(nuna):
    buf = torch.zeros(16 << 18, dtype=torch.int32, device="cuda")  # 16 MiB: 2048 blocks of 8 KiB
    return nuna.cu_latency_map(buf, stride=8192, xcds=(0, 5))


def test_cu_probe_reaches_every_compute_unit(cu_map):
    """512 one-wave workgroups reach all 32 compute units of an XCD; each CU is probed once."""
    for x, (lat, keys, seen) in cu_map.items():
        assert seen == 32 and lat.shape == (32, 2048), (x, seen, tuple(lat.shape))
        assert np.unique(keys.numpy()).size == 32
        assert np.all(lat.numpy() > 100)


def test_cu_probe_sees_the_same_dies_as_the_xcd_probe(cu_map):
    """Every compute unit of XCD 0 ranks the blocks near and far the way XCD 5's compute units rank them
    the other way round: per block, the XCD-0 CUs' mean latency is below the XCD-5 CUs' mean latency on
    the near-to-XCD-0 blocks, and single CUs agree with that label on most blocks."""
    a = cu_map[0][0].numpy()
    b = cu_map[5][0].numpy()
    near0 = a.mean(axis=0) < b.mean(axis=0)
    assert 0.3 < near0.mean() < 0.7
    thr = (np.median(a[:, near0], axis=1) + np.median(a[:, ~near0], axis=1))[:, None] / 2
    agree = np.mean((a < thr) == near0[None, :], axis=1)
    assert np.median(agree) > 0.8, agree
