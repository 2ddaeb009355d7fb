"""GPU results against the oracle, through the C ABI (binding in paper_1708_02937_amd).

Tolerance and pattern rule: see tests/parity.py (|g - o| <= 1e-6 + 1e-5 |o|; pattern equal
except entries at the ReLU threshold within the fp32 rounding allowance; integer-valued
problems bit for bit).
"""

import math

import numpy as np
import pytest

from tests import parity
from workloads import Layer, csr_rows, dense_to_csr, integer_shadow, make_config, paper_grid, tiny_random

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sd():
    import torch

    import paper_1708_02937_amd as sd

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return sd


def _say(*a):
    print("[case]", *a, flush=True)


def run_dense(sd, p, arm, y0=None, bias_mode=0):
    import torch

    net = sd.net_from_problem(p, dense={sd.SDNN_ARM_DENSE: 1, sd.SDNN_ARM_DENSE_F32: 2}.get(arm, 0), bias_mode=bias_mode)
    y = torch.from_numpy(p.y0_dense if y0 is None else y0).cuda()
    out = net.forward_dense(y, arm=arm).cpu().numpy()
    net.free()
    return out


def run_csr(sd, p, y0=None, k0=0, k1=None, bias_mode=0):
    net = sd.net_from_problem(p, bias_mode=bias_mode)
    rp, c, v = net.forward_csr(*(p.y0_as_csr() if y0 is None else y0), k0=k0, k1=k1)
    res = (rp.cpu().numpy(), c.cpu().numpy(), v.cpu().numpy())
    net.free()
    return res


ARMS = ["sparse", "dense"]


def _arm(sd, name):
    return {"sparse": sd.SDNN_ARM_SPARSE, "dense": sd.SDNN_ARM_DENSE, "dense32": sd.SDNN_ARM_DENSE_F32}[name]


# ------------------------------------------------------------------------------------------ small shapes

TINY = [(1, 1, 1, 1), (2, 7, 2, 3), (3, 63, 2, 64), (4, 64, 3, 65), (5, 65, 2, 130), (6, 200, 3, 257),
        (7, 333, 2, 129), (8, 130, 1, 2048)]


@pytest.mark.parametrize("arm", ARMS)
@pytest.mark.parametrize("seed,n,L,batch", TINY)
def test_tiny_dense_batch(sd, arm, seed, n, L, batch):
    ymax = [math.inf, 1.5][seed % 2]
    p = tiny_random(seed, n, L, batch, w_density=0.2, y_density=0.6, dense_input=True, ymax=ymax,
                    explicit_zeros=seed % 3 == 0)
    _say("tiny dense", arm, seed, n, L, batch)
    out = run_dense(sd, p, _arm(sd, arm))
    parity.compare(p, dense_to_csr(out))


@pytest.mark.parametrize("seed,n,L,batch,d", [(31, 1400, 2, 128, 0.97), (32, 1400, 2, 260, 0.95),
                                              (33, 2000, 2, 1028, 0.7), (34, 1500, 1, 516, 0.9),
                                              (35, 1290, 2, 132, 0.999), (36, 1503, 1, 388, 0.9),
                                              (40, 1500, 2, 256, 0.25)])
def test_high_fanin_lds_tiles(sd, seed, n, L, batch, d):
    """Density >= 2/9 selects the LDS-tiled product with scalar-register weights; ragged n (not a
    multiple of 4, 16 or 64) and batch exercise its edges; d = 0.25, just above the switch, leaves most slots
    empty."""
    p = tiny_random(seed, n, L, batch, w_density=d, y_density=0.7, dense_input=True,
                    ymax=[math.inf, 3.0][seed % 2], bias_lo=-1.0, bias_hi=1.0)
    _say("high fan-in", seed, n, L, batch, d)
    parity.compare(p, dense_to_csr(run_dense(sd, p, sd.SDNN_ARM_SPARSE)))
    q = integer_shadow(p)
    q.y0_dense = np.where(p.y0_dense != 0, q.y0_dense if q.y0_dense is not None else 1, 0).astype(np.float32)
    parity.compare(q, dense_to_csr(run_dense(sd, q, sd.SDNN_ARM_SPARSE)), exact=True)


@pytest.mark.parametrize("seed,n,L,batch,d", [(38, 1400, 2, 130, 0.95), (39, 1333, 1, 63, 0.99)])
def test_high_fanin_gather_fallback(sd, seed, n, L, batch, d):
    """Density >= 2/9 but a batch the LDS-tiled kernels do not take (not a multiple of 4, or below
    128): the layer falls back to the gather SpMM with two or one columns per lane over lists far longer
    than one 64-entry load; integer shadow bit for bit."""
    p = tiny_random(seed, n, L, batch, w_density=d, y_density=0.7, dense_input=True,
                    ymax=[math.inf, 3.0][seed % 2], bias_lo=-1.0, bias_hi=1.0)
    assert 9 * p.layers[0].nnz >= 2 * p.n * p.n
    _say("high fan-in gather fallback", seed, n, L, batch, d)
    parity.compare(p, dense_to_csr(run_dense(sd, p, sd.SDNN_ARM_SPARSE)))
    q = integer_shadow(p)
    q.y0_dense = np.where(p.y0_dense != 0, q.y0_dense if q.y0_dense is not None else 1, 0).astype(np.float32)
    parity.compare(q, dense_to_csr(run_dense(sd, q, sd.SDNN_ARM_SPARSE)), exact=True)


def test_high_fanin_beyond_slot_limit(sd):
    """n = 16448: the fp64 weight slots of every (input, output) pair would exceed 2 GiB, so a layer of
    density >= 0.3 takes the readlane-fed LDS-tiled kernel instead of the scalar-register one; sampled rows,
    ragged batch."""
    p = tiny_random(37, 16448, 1, 132, w_density=0.31, y_density=0.7, dense_input=True, bias_lo=-1.0, bias_hi=1.0)
    assert 10 * p.layers[0].nnz >= 3 * p.n * p.n
    rows = np.arange(0, 132, 12)
    _say("high fan-in beyond the slot limit")
    out = run_dense(sd, p, sd.SDNN_ARM_SPARSE)
    parity.compare(p, dense_to_csr(out[rows]), rows=rows)


@pytest.mark.parametrize("seed,n,L,batch", TINY + [(9, 5000, 2, 17), (10, 17000, 2, 9), (11, 40000, 1, 5)])
def test_tiny_csr_batch(sd, seed, n, L, batch):
    p = tiny_random(seed, n, L, batch, w_density=min(0.3, 8.0 / n + 0.001), y_density=0.3,
                    bias_lo=-0.3, bias_hi=0.05 if seed % 2 else 0.0, ymax=[math.inf, 2.0][seed % 2],
                    explicit_zeros=seed % 3 == 0)
    _say("tiny csr", seed, n, L, batch)
    parity.compare(p, run_csr(sd, p))


@pytest.mark.parametrize("arm", ARMS)
@pytest.mark.parametrize("m,S", [(256, 1), (512, 2), (512, 16), (1024, 4), (1024, 1024), (2048, 262144),
                                 (4096, 1), (4096, 64), (8192, 16)])
def test_paper_grid_points(sd, arm, m, S):
    """Single layers of the paper's own matrix family (Sec. V.B) on both arms, batch 64; from m = 4096 on the
    sparse arm takes the narrow-chunk gather (batch under 256), up to dense W (S = 1, fan-in 4096)."""
    p = paper_grid(m, S)
    _say("paper grid", arm, m, S)
    parity.compare(p, dense_to_csr(run_dense(sd, p, _arm(sd, arm))))


# ------------------------------------------------------------------ bias on the structural pattern only


@pytest.mark.parametrize("seed,n,L,batch,wd,yd", [(61, 300, 3, 40, 0.02, 0.05), (62, 3000, 2, 257, 0.003, 0.015),
                                                  (63, 40000, 2, 24, 0.0002, 0.0012), (64, 500, 3, 64, 0.05, 0.3),
                                                  (65, 2000, 2, 100, 0.016, 0.1), (72, 40000, 2, 700, 0.0002, 0.008),
                                                  (73, 40000, 2, 300, 0.0002, 0.0275)])
def test_pattern_bias_csr_path(sd, seed, n, L, batch, wd, yd):
    """SDNN_BIAS_PATTERN with positive biases through the CSR path: small-sample and workgroup SpGEMM
    (one and three windows; the last two cases give the pipelined instance several samples per workgroup,
    the last one samples of about 1100 entries, two per thread), and the density-driven switch to dense
    activations (denser cases)."""
    p = tiny_random(seed, n, L, batch, w_density=wd, y_density=yd, bias_lo=-0.2, bias_hi=0.6,
                    explicit_zeros=seed % 2 == 1, ymax=[math.inf, 2.0][seed % 2])
    _say("pattern csr", seed, n, L, batch)
    parity.compare(p, run_csr(sd, p, bias_mode=1), bias_mode=1)


@pytest.mark.parametrize("seed,n,L,batch,wd,yd,b", [(74, 40000, 2, 300, 0.0002, 0.0275, 0.25),
                                                    (75, 3000, 2, 257, 0.003, 0.015, 0.25),
                                                    (76, 40000, 2, 200, 0.0002, 0.008, -0.1)])
def test_uniform_bias_csr_path(sd, seed, n, L, batch, wd, yd, b):
    """One bias value for every neuron (read once by the small-sample and pipelined SpGEMM instances), on
    the structural pattern (a positive b) and everywhere (a negative b, so sums are cut at -b)."""
    pattern = 1 if b > 0 else 0
    p = tiny_random(seed, n, L, batch, w_density=wd, y_density=yd, bias_lo=b, bias_hi=b,
                    ymax=[math.inf, 2.0][seed % 2])
    assert np.all(p.layers[0].bias == np.float32(b))
    _say("uniform bias csr", seed, n, L, batch, b)
    parity.compare(p, run_csr(sd, p, bias_mode=pattern), bias_mode=pattern)


@pytest.mark.parametrize("seed,n,L,batch,d,yd", [(66, 200, 2, 130, 0.05, 0.3), (67, 1400, 2, 260, 0.95, 0.001),
                                                 (68, 333, 3, 3, 0.1, 0.5), (69, 4100, 1, 2048, 0.002, 0.01),
                                                 (71, 2000, 2, 516, 0.7, 0.002)])
def test_pattern_bias_dense_batch(sd, seed, n, L, batch, d, yd):
    """SDNN_BIAS_PATTERN on the sparse arm with dense batches: the gather SpMM (one, two and four columns
    per lane) and the LDS-tiled SpMM (density >= 2/9); sparse inputs leave many positions untouched."""
    p = tiny_random(seed, n, L, batch, w_density=d, y_density=yd, dense_input=True, bias_lo=-0.2, bias_hi=0.6)
    _say("pattern dense", seed, n, L, batch)
    parity.compare(p, dense_to_csr(run_dense(sd, p, sd.SDNN_ARM_SPARSE, bias_mode=1)), bias_mode=1)


def test_pattern_bias_integer_shadow_and_dense_arm(sd):
    """Integer shadow of the very wide workload (positive biases, scaled) matches bit for bit in pattern
    mode; the dense arm has no pattern and refuses it."""
    q = integer_shadow(make_config(5, n=20480, L=2, batch=12, block=4096))
    _say("pattern integer shadow")
    parity.compare(q, run_csr(sd, q, bias_mode=1), exact=True, bias_mode=1)
    p = tiny_random(70, 64, 1, 4, dense_input=True)
    with pytest.raises(sd.SdnnError) as ei:
        run_dense(sd, p, sd.SDNN_ARM_DENSE, bias_mode=1)
    assert ei.value.status == 9


# ------------------------------------------------------------------ semiring mxm (Sec. II)

SEMIRINGS = ["plus_times", "max_plus", "max_min", "min_max", "xor_and"]


@pytest.mark.parametrize("name", SEMIRINGS)
@pytest.mark.parametrize("seed,n,batch,d", [(81, 37, 3, 0.3), (82, 300, 130, 0.05), (83, 1000, 2048, 0.01),
                                            (84, 700, 64, 0.6)])
def test_semiring_mxm_dense(sd, name, seed, n, batch, d):
    """Z = Y (+).(x) W_k on the gather skeleton equals the oracle bit for bit (one order of reduction,
    exact products), for 1, 2 and 4 columns per lane and with explicit zeros stored in W."""
    import oracle
    import torch

    p = tiny_random(seed, n, 1, batch, w_density=d, dense_input=True, y_density=0.7, explicit_zeros=True)
    want = oracle.mxm(name, n, p.layers[0], p.y0_dense)
    net = sd.net_from_problem(p)
    _say("semiring dense", name, seed, n, batch)
    got = net.mxm(0, oracle.SEMIRINGS[name], torch.from_numpy(p.y0_dense).cuda()).cpu().numpy()
    net.free()
    assert got.tobytes() == want.tobytes()


@pytest.mark.parametrize("name", SEMIRINGS)
@pytest.mark.parametrize("seed,n,batch,wd,yd", [(85, 500, 97, 0.02, 0.05), (86, 3000, 40, 0.3, 0.2),
                                                (87, 40000, 9, 0.0005, 0.002), (88, 64, 5, 0.5, 0.0)])
def test_semiring_mxm_csr(sd, name, seed, n, batch, wd, yd):
    """The CSR form, row by row over the stored entries: entries Y does not store are the 0-element (they
    contribute nothing); one and three accumulator windows, long fan-out rows, empty rows, explicit zeros in
    W.  Every semiring but +.x is exact; +.x sums in fp64 in atomic order, so it is held to the tolerance, and
    an integer-valued +.x product (exact in any order) bit for bit."""
    import oracle

    p = tiny_random(seed, n, 1, batch, w_density=wd, y_density=yd, explicit_zeros=True)
    zero = {"max_plus": -math.inf, "max_min": -math.inf, "min_max": math.inf}.get(name, 0.0)
    ydn = np.full((batch, n), zero, np.float32)
    rp, c, v = p.y0_csr
    rows = np.repeat(np.arange(batch), np.diff(rp))
    ydn[rows, c] = v
    want = oracle.mxm(name, n, p.layers[0], ydn)
    net = sd.net_from_problem(p)
    _say("semiring csr", name, seed, n)
    got = net.mxm_csr(0, oracle.SEMIRINGS[name], rp, c, v).cpu().numpy()
    if name == "plus_times":
        assert np.all(np.abs(got.astype(np.float64) - want) <= 1e-6 + 1e-5 * np.abs(want.astype(np.float64)))
        q = integer_shadow(p)
        net2 = sd.net_from_problem(q)
        qrp, qc, qv = q.y0_csr
        qd = np.zeros((batch, n), np.float32)
        qd[np.repeat(np.arange(batch), np.diff(qrp)), qc] = qv
        got2 = net2.mxm_csr(0, 0, qrp, qc, qv).cpu().numpy()
        net2.free()
        assert got2.tobytes() == oracle.mxm(name, n, q.layers[0], qd).tobytes()
    else:
        assert got.tobytes() == want.tobytes()
    net.free()


@pytest.mark.parametrize("n,batch", [(1 << 20, 4098), (1 << 23, 1056)])
def test_blocked_product_very_wide(sd, n, batch):
    """Very wide layers on the sample-blocked layout: n = 2^20, batch 4098 (129 chunks of 32 samples, the
    last one partial) and n = 2^23, batch 1056 (33 chunks: more workgroups than one launch holds, so the
    product runs as two launches of whole chunks).  Y is drawn on the device from a seeded generator and the
    sampled rows are handed to the oracle; up to 145 GB of device memory."""
    import torch

    rng = np.random.default_rng(20170802)
    col = np.sort(rng.integers(0, n, size=(n, 2)), axis=1).astype(np.int32)
    col[:, 1] = np.where(col[:, 1] == col[:, 0], (col[:, 0] + 1) % n, col[:, 1])
    col.sort(axis=1)
    row_ptr = np.arange(0, 2 * n + 1, 2, dtype=np.int64)
    layer = Layer(row_ptr, col.reshape(-1), rng.uniform(-1, 1, size=2 * n).astype(np.float32),
                  rng.uniform(-0.1, 0.1, size=n).astype(np.float32))
    gen = torch.Generator(device="cuda").manual_seed(20170802)
    y = torch.rand((batch, n), generator=gen, device="cuda", dtype=torch.float32)
    net = sd.Net(n, 1, nnz_per_layer=layer.nnz)
    net.set_layer(0, layer.row_ptr, layer.col, layer.val, layer.bias)
    _say("blocked very wide", n, batch)
    out = net.forward_dense(y, arm=sd.SDNN_ARM_SPARSE)
    rows = [0, 1, 31, 32, 1023, batch - 2, batch - 1]
    got = out[rows].cpu().numpy()
    y_rows = y[rows].cpu().numpy()
    del out, y
    net.free()
    torch.cuda.empty_cache()
    from workloads import Problem
    p = Problem("segmented", n, 1, len(rows), math.inf, [layer], y0_dense=y_rows)
    parity.compare(p, dense_to_csr(got))


def _mixed_length_layer(rng, n, lengths):
    """W whose output neuron j gathers lengths[j % len(lengths)] distinct inputs (so the four neurons of a
    wave have very different list lengths); returns the Layer in its input-major CSR form."""
    ii, jj = [], []
    for j in range(n):
        k = min(lengths[j % len(lengths)], n)
        ii.append(rng.choice(n, size=k, replace=False))
        jj.append(np.full(k, j))
    i = np.concatenate(ii).astype(np.int64)
    j = np.concatenate(jj).astype(np.int64)
    order = np.lexsort((j, i))
    i, j = i[order], j[order]
    row_ptr = np.zeros(n + 1, np.int64)
    np.add.at(row_ptr, i + 1, 1)
    return Layer(np.cumsum(row_ptr), j.astype(np.int32), rng.uniform(-1, 1, size=len(i)).astype(np.float32),
                 rng.uniform(-0.3, 0.3, size=n).astype(np.float32))


@pytest.mark.parametrize("seed,n,batch,lengths,bias_mode", [
    (81, 4097, 36, [0, 1, 15, 16, 17, 40, 100], 0), (82, 5003, 96, [3, 0, 0, 33, 8, 9, 64, 1], 0),
    (83, 6144, 132, [16, 16, 16, 16, 32, 31, 48, 7], 1), (84, 4099, 4, [120, 0, 5, 17], 1),
    (85, 4500, 300, [2, 30, 31, 33, 0, 64, 120, 130], 0), (86, 16384, 512, [32, 25, 40, 32, 100, 120], 1),
    (87, 40000, 60, [33, 2, 0, 17, 64], 0), (88, 4099, 2, [120, 0, 5, 17], 0)])
def test_narrow_chunk_gather(sd, seed, n, batch, lengths, bias_mode):
    """Layers with n >= 4096 and a batch under 256 that is a multiple of 4, or n > 4096 up to 16384 with
    lists too long for the blocked product (over 48 entries per neuron on average; cases 85 and 86, at a
    batch of 256 or more), take the narrow-chunk gather (16 lanes and 64 columns, four per lane, per
    neuron): ragged n, partial last chunks, and list lengths from 0 to 130 side by side in one wave, which
    exercises the unpredicated prefix, the guarded tail and lists spanning several loads of 16 entries.  The
    last case (batch 2, not a multiple of 4) is the fan-in gather fallback with one column per lane."""
    rng = np.random.default_rng(seed)
    layers = [_mixed_length_layer(rng, n, lengths), _mixed_length_layer(rng, n, lengths[::-1])]
    y = rng.random((batch, n), dtype=np.float32)
    y[rng.random((batch, n)) < 0.3] = 0.0
    from workloads import Problem
    p = Problem(f"narrow-{seed}", n, 2, batch, math.inf, layers, y0_dense=y)
    _say("narrow gather", seed, n, batch, bias_mode)
    parity.compare(p, dense_to_csr(run_dense(sd, p, sd.SDNN_ARM_SPARSE, bias_mode=bias_mode)),
                   bias_mode=bias_mode)


@pytest.mark.parametrize("seed,n,batch,lengths,bias_mode", [
    (91, 16400, 256, [32, 25, 40, 32, 0, 1, 77, 33], 0), (92, 20000, 300, [3, 0, 0, 33, 8, 9, 64, 1], 1),
    (93, 17003, 257, [120, 0, 5, 17, 31, 32, 33], 0), (94, 24576, 512, [24, 24, 24, 24, 24, 24, 24, 25], 1),
    (95, 16900, 288, [100, 90, 110, 64], 0), (96, 18000, 256, [95, 0, 120, 101], 1),
    (97, 4500, 300, [2, 30, 31, 33, 0, 64], 0), (98, 16384, 512, [32, 25, 40, 32], 1),
    (99, 8192, 256, [0, 1, 15, 16, 17, 40, 100], 0), (100, 5000, 257, [3, 0, 17, 33, 64], 1)])
def test_blocked_product(sd, seed, n, batch, lengths, bias_mode):
    """Layers wider than 16384, or from 4097 to 16384 neurons with short lists (at most 48 entries per neuron
    on average: cases 97-100, whose 2 MiB or smaller chunks go whole to one XCD each, 10, 16, 8 and 9 chunks,
    the last of one sample),
    with batches of 256 or more take the product on the sample-blocked layout (chunks of 32 samples, eight
    neurons per wave walking their lists in step): ragged n, a partial last chunk, empty lists and list
    lengths from 0 to 120 side by side in one wave, both bias readings, every row compared.  Each workgroup stages its 64 neurons' lists in LDS while they fit (up to about 3968
    entries: the cases with lists of about 100 entries exceed it, and their layers read the staged copy
    entry by entry instead)."""
    rng = np.random.default_rng(seed)
    layers = [_mixed_length_layer(rng, n, lengths), _mixed_length_layer(rng, n, lengths[::-1])]
    y = rng.random((batch, n), dtype=np.float32)
    y[rng.random((batch, n)) < 0.3] = 0.0
    from workloads import Problem
    p = Problem(f"blocked-{seed}", n, 2, batch, [math.inf, 2.5][seed % 2], layers, y0_dense=y)
    _say("blocked product", seed, n, batch, bias_mode)
    parity.compare_in_chunks(p, dense_to_csr(run_dense(sd, p, sd.SDNN_ARM_SPARSE, bias_mode=bias_mode)),
                             bias_mode=bias_mode)


@pytest.mark.parametrize("longest,want", [(150, "spmm_narrow_kernel"), (120, "spmm_blocked_kernel")])
def test_mid_width_layout_choice(sd, longest, want):
    """From 4097 to 16384 neurons a forward takes the sample-blocked layout only when every layer stages its
    lists: layers of 20-entry lists with one longer list per 4096 neurons (which the schedule's sort puts in
    its run's first workgroup region, still small enough for LDS) stay neuron-major on the narrow-chunk
    gather when that list holds 150 entries (more than the staged product walks), and take the blocked
    product at 120; both paths (dense and CSR input) against the oracle, the kernel that ran read from the
    library's profiling log."""
    import torch

    rng = np.random.default_rng(71)
    n, batch = 6000, 300
    lengths = [20] * 4095 + [longest]
    layers = [_mixed_length_layer(rng, n, lengths), _mixed_length_layer(rng, n, lengths[::-1])]
    assert all(l.nnz <= 48 * n for l in layers)
    y = rng.random((batch, n), dtype=np.float32)
    y[rng.random((batch, n)) < 0.5] = 0.0
    from workloads import Problem
    p = Problem(f"mid-width-{longest}", n, 2, batch, math.inf, layers, y0_dense=y)
    net = sd.net_from_problem(p)
    net.set_profiling(True)
    _say("mid-width layout", longest)
    out = net.forward_dense(torch.from_numpy(y).cuda()).cpu().numpy()
    rp, c, v = net.forward_csr(*(torch.from_numpy(a).cuda() for a in p.y0_as_csr()))
    got_csr = (rp.cpu().numpy(), c.cpu().numpy(), v.cpu().numpy())
    torch.cuda.synchronize()
    ran = {k for _, k, _ in net.read_profile()}
    net.free()
    assert want in ran and ({"spmm_blocked_kernel", "spmm_narrow_kernel"} - {want}).isdisjoint(ran), ran
    parity.compare(p, dense_to_csr(out))
    parity.compare(p, got_csr)


@pytest.mark.parametrize("case", ["from_input", "after_sparse", "integer", "empty_layer", "unstaged"])
def test_blocked_csr_path(sd, case):
    """The CSR path's dense activations on the blocked layout: densify from the caller's CSR (positive bias
    from layer 0) or from slot rows after sparse layers, the layers, and the packing into CSR; an integer
    shadow of the very wide recipe (scaled, batch 260) bit for bit; a layer with no weights; a 2%-dense input
    whose first layer cannot stage its lists (one list of 150 entries), so densify stores every row, zero
    rows included, for a product that reads them all."""
    if case == "unstaged":
        rng = np.random.default_rng(97)
        n, batch = 17000, 288
        layers = [_mixed_length_layer(rng, n, [150, 10, 20, 30, 0, 33]), _mixed_length_layer(rng, n, [33, 2, 40])]
        for l in layers:
            l.bias = rng.uniform(0.0, 0.2, size=n).astype(np.float32)
        y = rng.random((batch, n), dtype=np.float32)
        y[rng.random((batch, n)) >= 0.02] = 0.0
        from workloads import Problem
        p = Problem("blocked-unstaged", n, 2, batch, math.inf, layers, y0_dense=y)
        _say("blocked csr", case)
        parity.compare_in_chunks(p, run_csr(sd, p))
        return
    if case == "integer":
        q = integer_shadow(make_config(5, n=20480, L=3, batch=260, block=4096))
        for l in q.layers:  # positive biases everywhere: dense activations from layer 0
            l.bias = np.ones(q.n, np.float32)
        _say("blocked csr integer")
        parity.compare(q, run_csr(sd, q), exact=True)
        return
    p = tiny_random(95, 20000, 3, 300, w_density=0.0016, y_density=0.02, bias_lo=-0.2,
                    bias_hi=0.0 if case == "after_sparse" else 0.3)
    if case == "after_sparse":
        p.layers[2].bias = np.full(p.n, 0.02, np.float32)
    if case == "empty_layer":
        p.layers[1] = Layer(np.zeros(p.n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32),
                            np.linspace(-0.5, 0.5, p.n).astype(np.float32))
    _say("blocked csr", case)
    parity.compare_in_chunks(p, run_csr(sd, p))


def test_long_fanin_lists(sd):
    """Fan-in lists longer than 8192 entries (the radix-sort transpose handles any length), n not a multiple
    of 4, on both dense arms; sampled rows."""
    p = tiny_random(51, 9001, 1, 132, w_density=0.97, y_density=0.6, dense_input=True, bias_lo=-1.0, bias_hi=1.0)
    rows = np.arange(0, 132, 11)
    for arm in (sd.SDNN_ARM_SPARSE, sd.SDNN_ARM_DENSE):
        _say("long fan-in", arm)
        out = run_dense(sd, p, arm)
        parity.compare(p, dense_to_csr(out[rows]), rows=rows)


@pytest.mark.parametrize("n", [3000, 20000])
def test_spgemm_negative_bias_threshold(sd, n):
    """Every b_j < 0 but of different sizes: an accumulated sum at most -max_j b_j is zero after h in every
    column, so the SpGEMM epilogues read no bias for it; integer weights, inputs and biases put sums exactly
    on both thresholds (-max_j b_j and the column's own -b_j), compared bit for bit, with samples short enough
    for the one-wave kernel and long ones for the workgroup kernels (one accumulator window at n = 3000, two
    at 20000, dense and bitmap epilogues)."""
    rng = np.random.default_rng(13 + n)
    batch = 300
    layers = []
    for _ in range(2):
        ii, jj = [], []
        for i in range(n):
            k = int(rng.integers(4, 24))
            ii.append(np.full(k, i))
            jj.append(np.sort(rng.choice(n, size=k, replace=False)))
        i = np.concatenate(ii).astype(np.int64)
        j = np.concatenate(jj).astype(np.int32)
        row_ptr = np.zeros(n + 1, np.int64)
        np.add.at(row_ptr, i + 1, 1)
        vals = rng.choice(np.array([1.0, 2.0], np.float32), size=len(j))
        bias = -rng.choice(np.array([1.0, 2.0, 3.0, 5.0], np.float32), size=n)
        layers.append(Layer(np.cumsum(row_ptr), j, vals, bias))
    rows, cols = [], []
    for r in range(batch):
        ylen = int(rng.integers(1, 12)) if r % 3 else int(rng.integers(60, 160))
        rows.append(np.full(ylen, r))
        cols.append(np.sort(rng.choice(n, size=ylen, replace=False)))
    r_all = np.concatenate(rows).astype(np.int64)
    c_all = np.concatenate(cols).astype(np.int32)
    y_ptr = np.zeros(batch + 1, np.int64)
    np.add.at(y_ptr, r_all + 1, 1)
    y_val = rng.choice(np.array([1.0, 2.0], np.float32), size=len(c_all))
    from workloads import Problem
    p = Problem(f"neg-bias-{n}", n, 2, batch, math.inf, layers, y0_csr=(np.cumsum(y_ptr), c_all, y_val))
    _say("negative bias threshold", n)
    parity.compare(p, run_csr(sd, p), exact=True)


def test_small_sample_sort_sizes(sd):
    """The one-wave small-sample kernel sorts each sample's products by column: in registers for up to 512
    products (64, 128, 256 or 512 slots), through LDS beyond.  A narrow layer (300 neurons, fan-out rows of
    8-40) gives samples of 1 to about 1000 products with many equal columns (ties inside the sort), integer
    weights of both signs, inputs and non-positive biases keep every sum exact: compared bit for bit."""
    rng = np.random.default_rng(29)
    n, batch = 300, 700
    ii, jj = [], []
    for i in range(n):
        k = int(rng.integers(8, 41))
        ii.append(np.full(k, i))
        jj.append(np.sort(rng.choice(n, size=k, replace=False)))
    i = np.concatenate(ii).astype(np.int64)
    j = np.concatenate(jj).astype(np.int32)
    row_ptr = np.zeros(n + 1, np.int64)
    np.add.at(row_ptr, i + 1, 1)
    vals = rng.choice(np.array([1.0, 2.0, -1.0, -3.0], np.float32), size=len(j))
    bias = rng.choice(np.array([0.0, -1.0, -2.0], np.float32), size=n)
    layer = Layer(np.cumsum(row_ptr), j, vals, bias)
    longest = int(np.diff(layer.row_ptr).max())
    rows, cols = [], []
    for r in range(batch):
        ylen = 1 + r % (1024 // longest)
        rows.append(np.full(ylen, r))
        cols.append(np.sort(rng.choice(n, size=ylen, replace=False)))
    r_all = np.concatenate(rows).astype(np.int64)
    c_all = np.concatenate(cols).astype(np.int32)
    y_ptr = np.zeros(batch + 1, np.int64)
    np.add.at(y_ptr, r_all + 1, 1)
    y_val = rng.choice(np.array([1.0, 2.0], np.float32), size=len(c_all))
    from workloads import Problem
    p = Problem("small-sort-sizes", n, 1, batch, math.inf, [layer], y0_csr=(np.cumsum(y_ptr), c_all, y_val))
    fan = np.diff(layer.row_ptr)
    products = np.array([fan[c].sum() for c in cols])
    assert products.min() <= 64 and products.max() > 512
    _say("small-sample sort sizes")
    parity.compare(p, run_csr(sd, p), exact=True)


@pytest.mark.parametrize("n,fan,lens,biases,batch", [(3000, (4, 24), (150, 300), (0.0, -1.0, -2.0), 160),
                                                     (40000, (4, 24), (450, 1000), (-1.0, -2.0, -3.0), 160),
                                                     (3000, (30, 50), (60, 300), (-1.0, -2.0), 160),
                                                     (40000, (4, 24), (300, 900), (0.0, -1.0), 1100),
                                                     (60000, (4, 24), (400, 1000), (-1.0, -2.0), 1500),
                                                     (40000, (4, 24), (20, 1000), (-2.0,), 400)])
def test_spgemm_crossing_marks(sd, n, fan, lens, biases, batch):
    """Every b_j <= 0 and samples too long for the bitmap epilogue: the scatter marks the columns whose sum
    rises above -max_j b_j and the epilogue reads only those.  Weights of both signs make sums cross the
    threshold and fall back in any order of the additions; integer values keep every sum exact, so the
    output is compared bit for bit.  Samples longer than the bitmap epilogue takes (one in eight beyond 1024
    entries) use the register-resident and the general workgroup instances (lane-walked segments with short
    fan-out rows, half-wave segments with long ones), over one, three and four accumulator windows, with the
    input sparse enough to stay on the SpGEMM; a threshold of 0 comes from b_j = 0.  With three or four
    windows the register-resident samples take the pipelined instance; the two larger batches give each
    workgroup several samples in turn, mixing samples short enough for the bitmap epilogue with longer
    ones (all rows compared bit for bit, in blocks).  A single bias value takes the instances that read b
    once instead of per column."""
    rng = np.random.default_rng(17 + n + fan[0] + batch)
    layers = []
    for _ in range(2):
        ii, jj = [], []
        for i in range(n):
            k = int(rng.integers(fan[0], fan[1]))
            ii.append(np.full(k, i))
            jj.append(np.sort(rng.choice(n, size=k, replace=False)))
        i = np.concatenate(ii).astype(np.int64)
        j = np.concatenate(jj).astype(np.int32)
        row_ptr = np.zeros(n + 1, np.int64)
        np.add.at(row_ptr, i + 1, 1)
        vals = rng.choice(np.array([1.0, 2.0, -1.0, -2.0, -3.0], np.float32), size=len(j))
        bias = rng.choice(np.array(biases, np.float32), size=n)
        layers.append(Layer(np.cumsum(row_ptr), j, vals, bias))
    rows, cols = [], []
    for r in range(batch):
        ylen = int(rng.integers(*lens)) if r % 8 else int(rng.integers(1025, 1100))
        rows.append(np.full(ylen, r))
        cols.append(np.sort(rng.choice(n, size=ylen, replace=False)))
    r_all = np.concatenate(rows).astype(np.int64)
    c_all = np.concatenate(cols).astype(np.int32)
    y_ptr = np.zeros(batch + 1, np.int64)
    np.add.at(y_ptr, r_all + 1, 1)
    y_val = rng.choice(np.array([1.0, 2.0], np.float32), size=len(c_all))
    from workloads import Problem
    p = Problem(f"crossing-{n}-{fan[0]}", n, 2, batch, math.inf, layers, y0_csr=(np.cumsum(y_ptr), c_all, y_val))
    _say("crossing marks", n, fan, biases, batch)
    if batch > 500:
        assert parity.compare_exact_csr(p, run_csr(sd, p)) > 0
    else:
        parity.compare(p, run_csr(sd, p), exact=True)


@pytest.mark.parametrize("seed,n,L,batch,wd,yd", [(41, 5000, 3, 300, 0.0024, 0.008), (42, 3000, 2, 257, 0.003, 0.015),
                                                  (43, 40000, 2, 64, 0.0002, 0.0012)])
def test_small_and_large_samples_mixed(sd, seed, n, L, batch, wd, yd):
    """Every b_j <= 0: samples with few products take the one-wave sort kernel, longer ones the workgroup
    kernel, empty ones neither; lengths straddle the split (and one net has three accumulator windows)."""
    p = tiny_random(seed, n, L, batch, w_density=wd, y_density=yd, bias_lo=-0.2, bias_hi=0.0,
                    explicit_zeros=seed % 2 == 0)
    _say("small/large mix", seed, n, L, batch)
    parity.compare(p, run_csr(sd, p))


@pytest.mark.parametrize("cfg,kw", [
    (1, dict(n=1024, L=4, batch=64)), (2, dict(n=512, L=3, batch=200)), (3, dict(n=2048, L=3, batch=100)),
    (4, dict(n=20000, L=3, batch=50, window=1024)), (5, dict(n=20480, L=2, batch=12, block=4096))])
def test_integer_shadows_bit_exact(sd, cfg, kw):
    p = integer_shadow(make_config(cfg, 0.1 if cfg == 2 else None, **kw))
    _say("integer shadow", cfg, kw)
    if p.y0_dense is not None:
        for arm in ARMS:
            parity.compare(p, dense_to_csr(run_dense(sd, p, _arm(sd, arm))), exact=True)
    parity.compare(p, run_csr(sd, p), exact=True)


# --------------------------------------------------------------- padded row pitch of the activations

# n > 4096 and batch >= 256: the neuron-major activations sit at a padded row pitch (batch 256 -> 320 floats,
# 300 -> 320), so every kernel that reads or writes them indexes rows by the pitch, not by the batch.
@pytest.mark.parametrize("case", ["gather", "slots", "dense_arm", "csr_switch"])
@pytest.mark.parametrize("batch", [256, 300])
def test_padded_pitch_every_kernel(sd, case, batch):
    """The narrow-chunk gather, the scalar-register SpMM (density >= 2/9), the dense-W arm (K split, then the
    split sum) and the CSR path's switch to dense activations (densify, gather, transpose and compaction) at a
    padded pitch, ragged in n and batch."""
    n = 4500
    # the gather case averages 67 entries per neuron: short lists would take the sample-blocked layout
    d = {"gather": 0.015, "slots": 0.3, "dense_arm": 0.05, "csr_switch": 0.02}[case]
    if case == "csr_switch":
        p = tiny_random(90, n, 3, batch, w_density=d, y_density=0.3, bias_lo=0.0, bias_hi=0.2)
        _say("padded pitch", case, batch)
        parity.compare(p, run_csr(sd, p))
        return
    p = tiny_random(91, n, 2, batch, w_density=d, y_density=0.6, dense_input=True, bias_lo=-0.3, bias_hi=0.3)
    if case == "slots":
        assert 9 * p.layers[0].nnz >= 2 * n * n
    arm = sd.SDNN_ARM_DENSE if case == "dense_arm" else sd.SDNN_ARM_SPARSE
    rows = np.arange(0, batch, 7)
    _say("padded pitch", case, batch)
    out = run_dense(sd, p, arm)
    parity.compare(p, dense_to_csr(out[rows]), rows=rows)


@pytest.mark.parametrize("name", ["plus_times", "max_min"])
def test_semiring_mxm_padded_pitch(sd, name):
    """Semiring products at a padded activation pitch (n 4500, batch 260 -> 320), dense and CSR input."""
    import oracle
    import torch

    n, batch = 4500, 260
    p = tiny_random(92, n, 1, batch, w_density=0.004, dense_input=True, y_density=0.5)
    net = sd.net_from_problem(p)
    _say("semiring padded", name)
    got = net.mxm(0, oracle.SEMIRINGS[name], torch.from_numpy(p.y0_dense).cuda()).cpu().numpy()
    assert got.tobytes() == oracle.mxm(name, n, p.layers[0], p.y0_dense).tobytes()
    zero = {"max_min": -math.inf}.get(name, 0.0)
    rp, c, v = dense_to_csr(p.y0_dense)
    yd = np.full((batch, n), zero, np.float32)
    yd[np.repeat(np.arange(batch), np.diff(rp)), c] = v
    got = net.mxm_csr(0, oracle.SEMIRINGS[name], rp, c, v).cpu().numpy()
    net.free()
    want = oracle.mxm(name, n, p.layers[0], yd)
    if name == "plus_times":  # summed in atomic order on the CSR path
        assert np.all(np.abs(got.astype(np.float64) - want) <= 1e-6 + 1e-5 * np.abs(want.astype(np.float64)))
    else:
        assert got.tobytes() == want.tobytes()


# ------------------------------------------------------------------------------------------ the workloads


@pytest.mark.parametrize("arm", ARMS)
def test_config1_full(sd, arm):
    p = make_config(1)
    _say("config 1", arm)
    st = parity.compare(p, dense_to_csr(run_dense(sd, p, _arm(sd, arm))))
    assert st["entries"] > 0


def test_config1_csr_path(sd):
    p = make_config(1)
    _say("config 1 csr")
    parity.compare(p, run_csr(sd, p))


@pytest.mark.parametrize("d", [0.5, 0.25, 0.1, 0.01, 0.001])
def test_config2_sparse_arm_all_rows(sd, d):
    """The density-sweep workload at full size through the CSR arm, every row of Y_16 compared; d = 0.25
    sits just above the switch to the scalar-register LDS-tiled SpMM."""
    p = make_config(2, d)
    _say("config 2 sparse arm", d)
    out = run_dense(sd, p, sd.SDNN_ARM_SPARSE)
    st = parity.compare_in_chunks(p, dense_to_csr(out))
    assert st["entries"] > 0


@pytest.mark.parametrize("d", [0.5, 0.01])
def test_config2_dense_arm_all_rows(sd, d):
    p = make_config(2, d)
    _say("config 2 dense arm", d)
    out = run_dense(sd, p, sd.SDNN_ARM_DENSE)
    parity.compare_in_chunks(p, dense_to_csr(out))


@pytest.mark.parametrize("n", [700, 701])
@pytest.mark.parametrize("sparse_layers", [0, 1, 2, 3])
def test_csr_path_switches_to_dense_activations(sd, sparse_layers, n):
    """Layers with mostly positive bias move the CSR path to dense activations; switch after 0..3 layers
    (the exit compaction with four columns per thread when 4 | n, one otherwise)."""
    p = tiny_random(40 + sparse_layers, n, 4, 37, w_density=0.02, y_density=0.05, bias_lo=-0.2, bias_hi=0.0)
    for k in range(sparse_layers, p.L):
        p.layers[k].bias = np.full(p.n, 0.02, np.float32)
    _say("format switch", sparse_layers)
    parity.compare(p, run_csr(sd, p))
    q = integer_shadow(p)
    for k in range(sparse_layers, p.L):
        q.layers[k].bias = np.ones(p.n, np.float32)
    parity.compare(q, run_csr(sd, q), exact=True)


def test_config3_scaled_full_compare(sd):
    p = make_config(3, n=4096, L=6, batch=300)
    _say("config 3 scaled")
    parity.compare(p, run_csr(sd, p))


def test_config3_full_size_all_rows(sd):
    """The sparse-activation workload at full size (n 16384, L 32, batch 4096): every row of Y_32."""
    p = make_config(3)
    _say("config 3 full size")
    st = parity.compare_in_chunks(p, run_csr(sd, p))
    assert st["entries"] > 0


@pytest.fixture(scope="module")
def config4():
    return make_config(4)


@pytest.fixture(scope="module")
def config5():
    return make_config(5)


def test_config4_scaled(sd):
    p = make_config(4, n=32768, L=6, batch=400)
    _say("config 4 scaled")
    parity.compare(p, run_csr(sd, p))


@pytest.mark.parametrize("case", ["dies", "survives", "positive_bias_later"])
def test_csr_forward_stops_at_empty_activation(sd, case):
    """forward_csr checks the output count after its 1st, 2nd, 4th ... sparse layer when at least 8 later
    layers keep an empty activation empty, and stops at an empty one.  The deep sparse recipe dies out after
    its second layer (the loop must stop there, with the oracle's empty Y_L); a denser net with non-positive
    biases keeps its entries (checked, no stop); one layer with positive biases among the later ones rules
    the check out.  Every case against the oracle."""
    import torch

    if case == "dies":
        p = make_config(4, n=32768, L=20, batch=300)
    else:
        p = tiny_random(75, 1500, 12, 120, w_density=0.02, y_density=0.05, bias_lo=-0.02, bias_hi=0.0)
        if case == "positive_bias_later":
            p.layers[9] = Layer(p.layers[9].row_ptr, p.layers[9].col, p.layers[9].val,
                                np.full(p.n, 0.01, np.float32))
    net = sd.net_from_problem(p)
    y = tuple(torch.from_numpy(a).cuda() for a in p.y0_as_csr())
    net.set_profiling(True)
    rp, c, v = net.forward_csr(*y)
    torch.cuda.synchronize()
    layers_run = sum(1 for _, name, _ in net.read_profile() if name == "spgemm_layer")
    net.set_profiling(False)
    got = (rp.cpu().numpy(), c.cpu().numpy(), v.cpu().numpy())
    net.free()
    _say("stop at empty activation", case, layers_run)
    parity.compare(p, got)
    if case == "dies":
        assert got[0][-1] == 0 and layers_run == 2
    else:
        assert got[0][-1] > 0
        assert layers_run <= p.L


def test_config4_layer0_bit_exact_all_rows(sd, config4):
    """Deep sparse, full size, the live layer: weights are exactly 1/16 and inputs binary, so every
    pre-activation is c/16 + b with an integer count c; c/16 is exact and the only rounding is the one to
    fp32 after the bias, so Y_1 must equal the oracle bit for bit in all 60000 rows (588k entries)."""
    p = config4
    _say("config 4 layer 0 exact")
    got = run_csr(sd, p, k0=0, k1=1)
    assert parity.compare_exact_csr(p, got, k0=0, k1=1) > 100000


def test_config4_two_layers_all_rows(sd, config4):
    """Layers 0 and 1 of the deep sparse network at full size, all rows, at the tolerance: layer 1 takes
    the SpGEMM on Y_1 (about 10 entries per sample), whose sums of a few c/16 - 0.3 values stay below the
    threshold -0.3 leaves, so Y_2 is empty in both."""
    p = config4
    _say("config 4 two layers")
    got = run_csr(sd, p, k0=0, k1=2)
    want = parity.oracle_rows(p, k1=2)
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
    assert np.all(np.abs(got[2].astype(np.float64) - want[2]) <= parity.ATOL + parity.RTOL * np.abs(want[2]))


def config5_rows(batch, seed=4):
    """One sampled row in each run of 32 consecutive samples: every batch chunk of the dense-Y kernels
    (32, 64 or 256 columns wide) holds at least one, eight per 256 columns."""
    rng = np.random.default_rng(seed)
    return np.arange(0, batch, 32) + rng.integers(0, 32, size=batch // 32)


def test_config5_full_size_sampled(sd, config5):
    """The very wide workload at full size: 256 rows of Y_8 spread over every 32-sample run of the batch."""
    p = config5
    _say("config 5 full size")
    rp, c, v = run_csr(sd, p)
    rows = config5_rows(p.batch)
    st = parity.compare_in_chunks(p, csr_rows((rp, c, v), rows), rows=rows, chunk=64)
    assert st["entries"] > 0


def test_config5_scaled(sd):
    p = make_config(5, n=32768, L=3, batch=24)
    _say("config 5 scaled")
    parity.compare(p, run_csr(sd, p))


# ------------------------------------------------------ per layer: the oracle's Y_k through one GPU layer


def _one_layer(p, k, y_csr, rows=None):
    """A one-layer problem: layer k of p applied to the CSR rows y_csr (the oracle's Y_k)."""
    from workloads import Problem

    nrows = len(y_csr[0]) - 1
    return Problem(f"{p.name}-layer{k}", p.n, 1, nrows, p.ymax, [p.layers[k]], y0_csr=y_csr)


@pytest.mark.parametrize("cfg,kw,k", [(1, {}, 2), (2, {"density": 0.1}, 9), (2, {"density": 0.5}, 15),
                                      (3, {}, 31)])
def test_per_layer_from_oracle_input(sd, cfg, kw, k):
    """The oracle's Y_k (all rows, full size) through GPU layer k alone, against the oracle's layer k:
    bounds one layer's error independently of the layers before it.  Dense workloads run on the dense-Y
    path (forward_dense), the sparse-activation one through forward_csr."""
    p = make_config(cfg, kw.get("density"))
    yk = parity.oracle_rows(p, k1=k)
    q = _one_layer(p, k, yk)
    _say("per layer", cfg, kw, k)
    if p.y0_dense is not None:
        got = dense_to_csr(run_dense(sd, q, sd.SDNN_ARM_SPARSE, y0=parity.to_dense(yk, p.n)))
    else:
        got = run_csr(sd, q)
    st = parity.compare_in_chunks(q, got)
    assert st["entries"] > 0


def test_per_layer_config4_and_5(sd, config4, config5):
    """Deep sparse layer 1 on the oracle's Y_1 (all rows, bit for bit: its inputs are c/16 - 0.3 values and
    the weights 1/16, so the products and their short sums are exact), and very wide layer 3 on the
    oracle's Y_3 of 256 sampled rows."""
    p = config4
    y1 = parity.oracle_rows(p, k1=1)
    q = _one_layer(p, 1, y1)
    _say("per layer config 4")
    parity.compare_exact_csr(q, run_csr(sd, q), k0=0, k1=1)
    p = config5
    rows = config5_rows(p.batch, seed=9)
    y3 = parity.oracle_rows(p, rows=rows, k1=3)
    q = _one_layer(p, 3, y3)
    _say("per layer config 5")
    st = parity.compare_in_chunks(q, run_csr(sd, q), chunk=64)
    assert st["entries"] > 0


# ------------------------------------------------------------------------------------------ structure


def test_identity_input_reads_back_weights(sd):
    """Y_0 = I gives row i of Y_1 = h(W(i,:) + b): pins the Y W orientation on both paths."""
    p = tiny_random(21, 150, 1, 150, w_density=0.1)
    eye = np.eye(150, dtype=np.float32)
    p.y0_dense = eye
    want = np.maximum(p.layers[0].to_dense(150).astype(np.float64) + p.layers[0].bias, 0).astype(np.float32)
    for arm in ARMS:
        assert run_dense(sd, p, _arm(sd, arm)).tobytes() == want.tobytes()
    got = parity.to_dense(run_csr(sd, p, y0=dense_to_csr(eye)), 150)
    assert got.tobytes() == want.tobytes()


@pytest.mark.parametrize("layers", ["gather", "slots", "narrow", "blocked"])
def test_graph_replay_matches_eager(sd, layers):
    """A HIP graph of forward_dense replays the eager result bit for bit, replay after replay, with new inputs
    written into the bound input and unrelated eager work between the replays (both arms); the layers take the
    gather SpMM (tiny MLP recipe), the scalar-register LDS-tiled SpMM (d = 0.5), the narrow-chunk gather at
    a padded activation pitch (n 4200, batch 256 -> 320, 63 entries per neuron) or the product on the
    sample-blocked layout (the same shape with 34 entries per neuron)."""
    import torch

    if layers == "gather":
        p = make_config(1, n=1000, L=3, batch=132)
    elif layers in ("narrow", "blocked"):
        p = tiny_random(46, 4200, 2, 256, w_density=0.015 if layers == "narrow" else 0.008, y_density=0.6,
                        dense_input=True, bias_lo=-0.3, bias_hi=0.3)
    else:
        p = tiny_random(45, 1300, 2, 128, w_density=0.5, y_density=0.7, dense_input=True, bias_lo=-1.0,
                        bias_hi=1.0)
        assert 9 * p.layers[0].nnz >= 2 * p.n * p.n
    for arm in ARMS:
        net = sd.net_from_problem(p, dense={"dense": 1, "dense32": 2}.get(arm, 0))
        rng = np.random.default_rng(5)
        inputs = [p.y0_dense] + [rng.random((p.batch, p.n), dtype=np.float32) for _ in range(3)]
        want = [net.forward_dense(torch.from_numpy(x).cuda(), arm=_arm(sd, arm)).cpu().numpy() for x in inputs]
        y = torch.from_numpy(inputs[0]).cuda()
        o = torch.empty_like(y)
        g = net.capture_forward_dense(y, o, arm=_arm(sd, arm))
        for rep, which in enumerate([0, 1, 2, 3, 3, 2, 1, 0]):
            _say("graph replay", arm, rep)
            y.copy_(torch.from_numpy(inputs[which]))
            g.replay()
            torch.cuda.synchronize()
            assert o.cpu().numpy().tobytes() == want[which].tobytes()
            # unrelated eager work on the same net and stream between replays
            net.forward_dense(torch.from_numpy(inputs[(rep + 1) % 4]).cuda(), arm=_arm(sd, arm))
            torch.cuda.synchronize()
        parity.compare(p, dense_to_csr(want[0]))
        net.free()


def test_run_twice_identical(sd):
    p = make_config(3, n=4096, L=4, batch=128)
    a, b = run_csr(sd, p), run_csr(sd, p)
    for x, y in zip(a, b):
        assert x.tobytes() == y.tobytes()
    q = make_config(2, 0.1, L=3, batch=256)
    assert run_dense(sd, q, sd.SDNN_ARM_SPARSE).tobytes() == run_dense(sd, q, sd.SDNN_ARM_SPARSE).tobytes()


def test_layer_ranges_compose(sd):
    import torch

    p = make_config(3, n=2048, L=5, batch=64)
    net = sd.net_from_problem(p)
    full = [x.cpu().numpy() for x in net.forward_csr(*p.y0_csr)]
    mid = [x.clone() for x in net.forward_csr(*p.y0_csr, k0=0, k1=2)]
    rest = [x.cpu().numpy() for x in net.forward_csr(*mid, k0=2, k1=5)]
    for x, y in zip(full, rest):
        assert x.tobytes() == y.tobytes()
    same = [x.cpu().numpy() for x in net.forward_csr(*p.y0_csr, k0=3, k1=3)]
    for x, y in zip(same, p.y0_csr):
        assert x.tobytes() == y.tobytes()
    q = make_config(2, 0.01, n=512, L=4, batch=128)
    net2 = sd.net_from_problem(q)
    y = torch.from_numpy(q.y0_dense).cuda()
    a = net2.forward_dense(y).cpu().numpy()
    b = net2.forward_dense(net2.forward_dense(y, k0=0, k1=1), k0=1, k1=4).cpu().numpy()
    assert a.tobytes() == b.tobytes()
    assert net2.forward_dense(y, k0=2, k1=2).cpu().numpy().tobytes() == q.y0_dense.tobytes()
    net.free()
    net2.free()


def test_degenerate_cases(sd):
    import torch

    n = 100
    empty = Layer(np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32),
                  np.linspace(-0.5, 0.5, n).astype(np.float32))
    p = tiny_random(3, n, 2, 10, dense_input=True)
    p.layers[1] = empty
    want = np.maximum(empty.bias.astype(np.float64), 0).astype(np.float32)
    for arm in ARMS:
        out = run_dense(sd, p, _arm(sd, arm))
        assert out.tobytes() == np.tile(want, (10, 1)).tobytes()
    # batch 0 and empty input rows
    net = sd.net_from_problem(p)
    y = torch.zeros((0, n), device="cuda")
    assert net.forward_dense(y).shape == (0, n)
    rp = np.zeros(5, np.int64)
    out = net.forward_csr(rp, np.zeros(0, np.int32), np.zeros(0, np.float32))
    p.y0_dense, p.y0_csr = None, (rp, np.zeros(0, np.int32), np.zeros(0, np.float32))
    parity.compare(p, [x.cpu().numpy() for x in out])  # empty samples: h(b) propagates
    net.free()
    # a CSR batch of no samples through layers, n a multiple of 4 and not
    for nn in (100, 101):
        q = tiny_random(5, nn, 2, 3, w_density=0.1)
        net = sd.net_from_problem(q)
        rp0 = np.zeros(1, np.int64)
        orp, oc, ov = net.forward_csr(rp0, np.zeros(0, np.int32), np.zeros(0, np.float32))
        assert orp.cpu().numpy().tolist() == [0] and oc.numel() == 0 and ov.numel() == 0
        net.free()


def test_errors_leave_net_usable(sd):
    import torch

    p = tiny_random(4, 50, 2, 6, w_density=0.2, dense_input=True)
    net = sd.Net(50, 2, nnz_per_layer=[l.nnz for l in p.layers])
    l = p.layers[0]
    bad_cols = l.col.copy()
    r = int(np.argmax(np.diff(l.row_ptr) >= 2))
    a = l.row_ptr[r]
    bad_cols[a], bad_cols[a + 1] = bad_cols[a + 1], bad_cols[a]  # unsorted row
    with pytest.raises(sd.SdnnError) as e:
        net.set_layer(0, l.row_ptr, bad_cols, l.val, l.bias)
    assert e.value.status == 3
    with pytest.raises(sd.SdnnError) as e:
        net.set_layer(0, l.row_ptr, np.where(l.col == l.col.max(), 50, l.col).astype(np.int32), l.val, l.bias)
    assert e.value.status == 3
    bad_rp = l.row_ptr.copy()
    bad_rp[-1] += 1
    with pytest.raises(sd.SdnnError) as e:
        net.set_layer(0, bad_rp, l.col, l.val, l.bias)
    assert e.value.status == 3
    nanb = l.bias.copy()
    nanb[3] = np.nan
    with pytest.raises(sd.SdnnError) as e:
        net.set_layer(0, l.row_ptr, l.col, l.val, nanb)
    assert e.value.status == 2
    y = torch.from_numpy(p.y0_dense).cuda()
    with pytest.raises(sd.SdnnError) as e:  # layers not set
        net.forward_dense(y)
    assert e.value.status == 5
    for k, lk in enumerate(p.layers):
        net.set_layer(k, lk.row_ptr, lk.col, lk.val, lk.bias)
    with pytest.raises(sd.SdnnError) as e:  # dense arm before build_dense
        net.forward_dense(y, arm=sd.SDNN_ARM_DENSE)
    assert e.value.status == 5
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    out = torch.empty_like(y)
    with pytest.raises(sd.SdnnError) as e:
        sd.sdnn_forward_dense(net.handle, 0, 2, 6, y, out, ws, 16, 0)
    assert e.value.status == 6
    with pytest.raises(sd.SdnnError) as e:
        sd.sdnn_forward_dense(net.handle, 1, 3, 6, y, out, ws, 16, 0)
    assert e.value.status == 4
    got = net.forward_dense(y).cpu().numpy()  # still usable
    parity.compare(p, dense_to_csr(got))
    net.free()


def test_profiling_log_names_each_launch(sd):
    """The profiling log holds one record per layer product and per format change, in launch order, with
    the kernel that ran and a positive GPU time; reading clears it, and nothing is recorded while off."""
    import torch

    p = make_config(1)
    net = sd.net_from_problem(p)
    y = torch.from_numpy(p.y0_dense).cuda()
    net.set_profiling(True)
    net.forward_dense(y)
    net.forward_csr(*p.y0_as_csr(), k0=0, k1=2)
    net.set_profiling(False)
    rec = net.read_profile()
    _say("profiling log", rec)
    names = [r[1] for r in rec]
    assert names[:6] == ["transpose_kernel"] + ["spmm_fanin_kernel"] * 4 + ["transpose_kernel"]
    assert [r[0] for r in rec[:6]] == [-1, 0, 1, 2, 3, -1]
    assert all(r[2] > 0 for r in rec)
    assert net.read_profile() == []
    net.forward_dense(y)
    assert net.read_profile() == []
    net.free()


# ------------------------------------------------------------------ fp32 dense arm (sgemm arithmetic)


@pytest.mark.parametrize("seed,n,batch,d", [(101, 1, 1, 1.0), (102, 63, 65, 0.3), (103, 130, 200, 0.2),
                                            (104, 1000, 300, 0.05), (105, 4096, 64, 0.5), (106, 700, 1024, 1.0)])
def test_fp32_dense_arm_one_layer(sd, seed, n, batch, d):
    """The fp32 matrix-core arm against the oracle within its derived bound: products and sums rounded to
    fp32 over n terms, |g - o| <= 1e-6 + 1e-5 |o| + gamma_{n+2} s (s = sum |y w| + |b|); ragged tiles, the
    split-K path at small batch and fully dense W."""
    p = tiny_random(seed, n, 1, batch, w_density=d, y_density=0.6, dense_input=True, bias_lo=-0.5, bias_hi=0.5)
    _say("fp32 dense arm", seed, n, batch, d)
    out = run_dense(sd, p, sd.SDNN_ARM_DENSE_F32)
    st = parity.compare_in_chunks(p, dense_to_csr(out), scale_tol=parity.fp32_sum_scale(n))
    assert st["entries"] > 0 or n == 1


@pytest.mark.parametrize("d", [0.5, 0.01])
def test_fp32_dense_arm_density_sweep_layer(sd, d):
    """One full-size density-sweep layer (n 4096, batch 1024) on the fp32 arm, every row, and the oracle's
    Y_9 through layer 9 (d = 0.01)."""
    p = make_config(2, d, L=1)
    _say("fp32 dense arm sweep", d)
    parity.compare_in_chunks(p, dense_to_csr(run_dense(sd, p, sd.SDNN_ARM_DENSE_F32)),
                             scale_tol=parity.fp32_sum_scale(p.n))
    if d == 0.01:
        q = make_config(2, d)
        yk = parity.oracle_rows(q, k1=9)
        one = _one_layer(q, 9, yk)
        got = dense_to_csr(run_dense(sd, one, sd.SDNN_ARM_DENSE_F32, y0=parity.to_dense(yk, q.n)))
        parity.compare_in_chunks(one, got, scale_tol=parity.fp32_sum_scale(q.n))


# ------------------------------------------------------------------ caller-owned arena


def test_arena_is_the_only_device_memory(sd):
    """The net keeps everything in the caller's arena: an arena one byte short is refused, a layer above
    its capacity is refused, and set-up, dense copies and forwards leave the device's free memory unchanged
    (the arena and workspace are allocated by the caller beforehand)."""
    import torch

    p = make_config(2, 0.01, n=20000, L=2, batch=256)
    caps = [l.nnz for l in p.layers]
    need = sd.sdnn_net_arena_size(p.n, p.L, caps, 3)
    assert need > sd.sdnn_net_arena_size(p.n, p.L, caps, 0)
    small = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(sd.SdnnError) as e:
        sd.sdnn_net_create(p.n, p.L, math.inf, caps, 3, small, need - 1)
    assert e.value.status == 6
    del small
    for rep in range(2):  # the first pass loads the code objects
        torch.cuda.synchronize()
        net = sd.Net(p.n, p.L, nnz_per_layer=caps, dense=3)
        y = torch.from_numpy(p.y0_dense).cuda()
        out = torch.empty_like(y)
        ws = net.workspace(p.batch, 0)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        for k, l in enumerate(p.layers):
            net.set_layer(k, l.row_ptr, l.col, l.val, l.bias)
        net.build_dense()
        for arm in (sd.SDNN_ARM_SPARSE, sd.SDNN_ARM_DENSE, sd.SDNN_ARM_DENSE_F32):
            net.forward_dense(y, arm=arm, out=out)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        _say("arena free memory", rep, free0, free1)
        if rep == 1:
            assert free0 - free1 < (2 << 20), "device memory was allocated outside the arena"
            l = p.layers[0]
            big = make_config(2, 0.02, n=20000, L=1, batch=8).layers[0]
            assert big.nnz > caps[0]
            with pytest.raises(sd.SdnnError) as e:
                net.set_layer(0, big.row_ptr, big.col, big.val, big.bias)
            assert e.value.status == 6
            parity.compare(p, dense_to_csr(net.forward_dense(y).cpu().numpy()))  # still usable
        net.free()
        del ws
