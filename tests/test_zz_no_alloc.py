"""The allocation-free forward entry point (sdnn_forward_dense_noalloc) against sdnn_forward_dense.

Both run the same kernels, so the outputs must be equal bit for bit: two calls in a row on the library's
fixed scratch array, the second on a smaller batch (the array still holds the first call's data), on both
arms, and a size above the array's capacity is refused."""

import numpy as np
import pytest

from workloads import make_config, tiny_random

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("arm", ["sparse", "dense"])
def test_noalloc_matches_workspace_entry_point(arm):
    import torch

    import paper_1708_02937_amd as sd

    a = sd.SDNN_ARM_SPARSE if arm == "sparse" else sd.SDNN_ARM_DENSE
    cases = [make_config(2, 0.01, L=3, batch=1024), make_config(2, 0.01, L=3, batch=300)]
    for p in cases:
        p.layers = cases[0].layers  # one net, two batch sizes
    net = sd.net_from_problem(cases[0], dense=(arm == "dense"))
    for p in cases:
        y = torch.from_numpy(p.y0_dense).cuda()
        want = net.forward_dense(y, arm=a).cpu().numpy()
        got = torch.full_like(y, float("nan"))
        _say("noalloc", arm, p.batch)
        sd.sdnn_forward_dense_noalloc(net.handle, 0, p.L, p.batch, y, got, a)
        torch.cuda.synchronize()
        assert got.cpu().numpy().tobytes() == want.tobytes()
    net.free()


def test_noalloc_blocked_layout():
    """At 4097-16384 neurons with short lists the forward runs on the sample-blocked layout: the same two
    calls in a row (batch 300, then 256) on the fixed array, bit for bit against the workspace entry point."""
    import torch

    import paper_1708_02937_amd as sd

    p = tiny_random(8, 4500, 2, 300, w_density=0.006, dense_input=True, y_density=0.5, bias_lo=-0.2, bias_hi=0.2)
    net = sd.net_from_problem(p)
    for batch in (300, 256):
        y = torch.from_numpy(np.ascontiguousarray(p.y0_dense[:batch])).cuda()
        want = net.forward_dense(y).cpu().numpy()
        got = torch.full_like(y, float("nan"))
        _say("noalloc blocked", batch)
        sd.sdnn_forward_dense_noalloc(net.handle, 0, p.L, batch, y, got, sd.SDNN_ARM_SPARSE)
        torch.cuda.synchronize()
        assert got.cpu().numpy().tobytes() == want.tobytes()
    net.free()


def test_noalloc_layer_range_and_limits():
    import torch

    import paper_1708_02937_amd as sd

    p = tiny_random(7, 700, 3, 130, w_density=0.05, dense_input=True, y_density=0.5, bias_lo=-0.2, bias_hi=0.2)
    net = sd.net_from_problem(p)
    y = torch.from_numpy(p.y0_dense).cuda()
    want = net.forward_dense(y, k0=1, k1=3).cpu().numpy()
    got = torch.empty_like(y)
    _say("noalloc range")
    sd.sdnn_forward_dense_noalloc(net.handle, 1, 3, p.batch, y, got, sd.SDNN_ARM_SPARSE)
    torch.cuda.synchronize()
    assert got.cpu().numpy().tobytes() == want.tobytes()
    # a workspace above the array's capacity is refused (nothing is launched)
    cap = sd.sdnn_noalloc_scratch_bytes()
    big = cap // (2 * 4 * p.n) + 64
    assert sd.sdnn_workspace_size(net.handle, big, 0) > cap
    with pytest.raises(sd.SdnnError) as e:
        sd.sdnn_forward_dense_noalloc(net.handle, 0, 3, big, y, got, sd.SDNN_ARM_SPARSE)
    assert e.value.status == 9
    net.free()
