"""GPU parity of Distribute + PointNet + per-vertex max (the fused operation)
against the CPU oracle, through the C ABI.

Every output row x_v (64 channels) is compared with the oracle's float64
value within 1e-5 of its scale (the rows' magnitudes carried through each
block's normalisation, |W|, |b|, the max over the vertex's rows); the local
means within a few fp32 ulps of their magnitude.  Vertex order is
canonicalised by sorted key.  Two forms of the normalisation: the group
normalisation with its statistics computed per cloud on the device, and the
caller's fixed affine (a, s).
"""
import numpy as np
import pytest
import torch

from datagen.clouds import make_workload, pointnet_gn_weights, pointnet_weights, random_cloud, raw_point_features
from oracle import lattice_oracle as O
from tests.gpu_util import REL_F32, GpuLattice, assert_close_scaled, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2108_03917_amd import load_library

    load_library()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _run(pos, feat, sigma, batch=None, seed=0, out_dtype="f32", groups=None, eps=1e-5, repeat=1):
    """One lattice, the fused operation (``repeat`` times on the same
    lattice: the statistics are zeroed by every call), every vertex compared.
    ``groups``: None for the caller's affines, "default" for min(32, K) per
    block, or three group counts."""
    from paper_2108_03917_amd import Lattice

    d = pos.shape[1]
    f_d = 0 if feat is None else feat.shape[1]
    L = Lattice(d, sigma, max_points=max(pos.shape[0], 1))
    g = GpuLattice(L, pos, None, batch=batch)
    lat = O.build(pos, sigma, batch=batch)
    assert np.array_equal(g.keys, lat.keys)
    if groups is None:
        sig0 = float(np.asarray(sigma, dtype=np.float64).reshape(-1)[0])
        layers = pointnet_weights(d + f_d, d, sig0, seed=seed)
        og = None
    else:
        layers = pointnet_gn_weights(d + f_d, seed=seed)
        og = [min(32, k) for k in (d + f_d, 16, 32)] if groups == "default" else list(groups)
    params = Lattice.pack_pointnet(layers).to("cuda:0")
    for _ in range(repeat):
        out, mean = L.distribute_pointnet(to_dev(pos), None if feat is None else to_dev(feat), params,
                                          want_mean=True, out_dtype=out_dtype, groups=og, eps=eps)
    ref, scale, mu = O.distribute_pointnet(lat, pos, feat, layers, groups=og, eps=eps)
    got = g.from_gpu_order(out.float())
    gmu = g.from_gpu_order(mean)
    assert np.all(np.isfinite(got))
    assert_close_scaled(gmu, mu, 2.0 ** -22 * np.abs(mu) + 1e-7 * np.abs(pos).max(), 1.0, "local mean")
    tag = f"distribute+pointnet d={d} f_d={f_d} {out_dtype} groups={og}"
    if out_dtype == "bf16":
        # the fp32 max rounded once to nearest even: half a bf16 ulp of the value
        assert_close_scaled(got, ref, REL_F32 * scale + 2.0 ** -8 * np.abs(ref), 1.0, tag)
    else:
        assert_close_scaled(got, ref, scale, REL_F32, tag)
    return lat


@pytest.mark.parametrize("d,m,sigma,f_d", [(3, 6000, 0.15, 6), (3, 5000, 0.1, 0), (4, 5000, 0.3, 1),
                                           (2, 4000, 0.08, 3)])
def test_distribute_pointnet_parity(d, m, sigma, f_d):
    w = random_cloud(m, d, seed=500 + d + f_d, extent=1.0, C=max(f_d, 1))
    _run(w.pos, w.feat[:, :f_d] if f_d else None, sigma, seed=501 + d)


def test_distribute_pointnet_batched():
    w = random_cloud(6000, 3, seed=510, extent=1.0, C=3, n_batch=5)
    _run(w.pos, w.feat, 0.15, batch=w.batch, seed=511)


@pytest.mark.parametrize("d,f_d", [(3, 6), (4, 1)])
def test_distribute_pointnet_bf16_rows(d, f_d):
    """Output rows stored as bf16 (for a bf16 conv that reads them), the
    whole-list stores and the decoded crossing lists both."""
    w = random_cloud(6000, d, seed=515 + d, extent=1.0, C=f_d)
    _run(w.pos, w.feat[:, :f_d], 0.15 if d == 3 else 0.3, seed=516 + d, out_dtype="bf16")


def test_distribute_pointnet_long_lists():
    """Tight clusters: vertices with hundreds to thousands of rows, whose
    lists span many 64-entry chunks (atomic max and fp64 atomic mean) and
    are mapped in 32-entry parts."""
    rng = np.random.default_rng(520)
    centres = rng.uniform(-0.8, 0.8, size=(3, 3))
    dense = centres[rng.integers(0, 3, 6000)] + rng.normal(0, 0.01, size=(6000, 3))
    sparse = rng.uniform(-1, 1, size=(3000, 3))
    pos = np.concatenate([dense, sparse]).astype(np.float32)[rng.permutation(9000)]
    feat = rng.standard_normal((9000, 4)).astype(np.float32)
    for out_dtype in ("f32", "bf16"):
        lat = _run(pos, feat, 0.1, seed=521, out_dtype=out_dtype)
    n = np.bincount(lat.idx.ravel(), minlength=lat.V)
    assert n.max() > 500 and (n > 64).sum() >= 3


def test_distribute_pointnet_empty_and_rejects():
    from paper_2108_03917_amd import Lattice, LatticeError

    L = Lattice(3, 0.1, max_points=16)
    L.splat(torch.zeros((0, 3), device="cuda:0"), None)
    params = Lattice.pack_pointnet(pointnet_weights(3, 3, 0.1, seed=1)).to("cuda:0")
    L.distribute_pointnet(torch.zeros((0, 3), device="cuda:0"), None, params)   # m = 0: nothing to do
    torch.cuda.synchronize()
    import ctypes

    feat = torch.zeros((1, 16), device="cuda:0")
    ok_widths = (ctypes.c_int * 3)(16, 32, 64)
    with pytest.raises(LatticeError):        # d + f_d = 17 > 16
        L._check(L._lib.lattice_distribute_pointnet(L._h, None, feat.data_ptr(), 14, params.data_ptr(), 3,
                                                    ok_widths, None, 0.0, None, 0, None), "distribute_pointnet")
    with pytest.raises(LatticeError):        # widths other than 16, 32, 64
        L._check(L._lib.lattice_distribute_pointnet(L._h, None, None, 0, params.data_ptr(), 3,
                                                    (ctypes.c_int * 3)(16, 32, 32), None, 0.0, None, 0, None),
                 "distribute_pointnet")
    with pytest.raises(LatticeError):        # an output type other than fp32 and bf16
        L._check(L._lib.lattice_distribute_pointnet(L._h, None, None, 0, params.data_ptr(), 3, ok_widths, None,
                                                    0.0, None, 7, None), "distribute_pointnet")
    for bad_groups, eps in (((2, 16, 32), 1e-5), ((3, 5, 32), 1e-5), ((3, 16, 0), 1e-5), ((3, 16, 32), -1.0),
                            ((3, 16, 32), float("nan"))):
        with pytest.raises(LatticeError):    # groups that do not divide the widths; a bad eps
            L._check(L._lib.lattice_distribute_pointnet(L._h, None, None, 0, params.data_ptr(), 3, ok_widths,
                                                        (ctypes.c_int * 3)(*bad_groups), eps, None, 0, None),
                     "distribute_pointnet")


@pytest.mark.parametrize("config,out_dtype", [(3, "bf16"), (4, "f32")])
def test_distribute_pointnet_full_size(config, out_dtype):
    """The indoor room (200k points, rgb + normal; bf16 rows, as the bench's
    first conv reads them) and the LiDAR scan (about 1.04e5 points in scan
    order, dense near the sensor), every vertex compared."""
    w = make_workload(config)
    _run(w.pos, raw_point_features(w), w.sigma, seed=530 + config, out_dtype=out_dtype)


# --------------------------------------------------------------------------
# group normalisation with its statistics computed on the device
# --------------------------------------------------------------------------

@pytest.mark.parametrize("d,m,sigma,f_d,groups", [(3, 6000, 0.15, 6, "default"), (4, 5000, 0.3, 1, "default"),
                                                  (2, 4000, 0.08, 3, "default"), (3, 5000, 0.1, 5, (1, 4, 8)),
                                                  (3, 3000, 0.12, 0, (3, 2, 16))])
def test_distribute_pointnet_gn_parity(d, m, sigma, f_d, groups):
    w = random_cloud(m, d, seed=540 + d + f_d, extent=1.0, C=max(f_d, 1))
    _run(w.pos, w.feat[:, :f_d] if f_d else None, sigma, seed=541 + d, groups=groups, repeat=2)


def test_distribute_pointnet_gn_batched_clouds():
    """Five clouds in one lattice, points grouped by cloud (most 64-entry
    chunks hold one cloud; the chunks at the boundaries span two)."""
    w = random_cloud(6000, 3, seed=550, extent=1.0, C=3, n_batch=5)
    order = np.argsort(w.batch, kind="stable")
    _run(w.pos[order], w.feat[order], 0.15, batch=w.batch[order], seed=551, groups="default")


def test_distribute_pointnet_gn_interleaved_clouds():
    """Batch ids drawn per point, with gaps between the ids used (0, 3, 7,
    11): consecutive vertices belong to different clouds, so nearly every
    chunk spans several (each row then takes its own cloud's affines and
    adds its own statistics)."""
    w = random_cloud(5000, 3, seed=552, extent=1.0, C=4)
    batch = np.random.default_rng(553).choice(np.array([0, 3, 7, 11], dtype=np.int32), size=w.m)
    for out_dtype in ("f32", "bf16"):
        _run(w.pos, w.feat, 0.15, batch=batch, seed=554, groups="default", out_dtype=out_dtype)


def test_distribute_pointnet_gn_long_lists():
    """Tight clusters (lists of hundreds to thousands of rows) with group
    normalisation: the statistics of rows whose vertex spans many chunks."""
    rng = np.random.default_rng(560)
    centres = rng.uniform(-0.8, 0.8, size=(3, 3))
    dense = centres[rng.integers(0, 3, 6000)] + rng.normal(0, 0.01, size=(6000, 3))
    sparse = rng.uniform(-1, 1, size=(3000, 3))
    pos = np.concatenate([dense, sparse]).astype(np.float32)[rng.permutation(9000)]
    feat = (rng.standard_normal((9000, 4)) * 3 + 2).astype(np.float32)
    _run(pos, feat, 0.1, seed=561, groups="default")


@pytest.mark.parametrize("config,out_dtype", [(2, "f32"), (3, "bf16"), (4, "f32")])
def test_distribute_pointnet_gn_full_size(config, out_dtype):
    """The part-seg batch (16 clouds, statistics per object), the indoor room
    (200k points, bf16 rows) and the LiDAR scan, with group normalisation,
    every vertex compared."""
    w = make_workload(config)
    _run(w.pos, raw_point_features(w), w.sigma, batch=w.batch, seed=570 + config, out_dtype=out_dtype,
         groups="default")


def test_distribute_pointnet_gn_too_many_clouds_is_reported():
    """Per-cloud statistics cover batch ids 0..63: a lattice with batch id
    90 completes the call in bounds and reports LATTICE_E_RANGE through the
    device status; the next splat clears it, and batch ids up to 63 pass."""
    from paper_2108_03917_amd import Lattice
    from paper_2108_03917_amd.lattice import E_RANGE, OK

    w = random_cloud(3000, 3, seed=580, extent=1.0, C=3)
    batch = np.random.default_rng(581).integers(0, 91, size=w.m).astype(np.int32)
    batch[0] = 90
    L = Lattice(3, 0.15, max_points=w.m)
    pos, feat = to_dev(w.pos), to_dev(w.feat)
    L.splat(pos, None, to_dev(batch), want_weight=False)
    params = Lattice.pack_pointnet(pointnet_gn_weights(6, seed=582)).to("cuda:0")
    L.distribute_pointnet(pos, feat, params, groups="default")
    torch.cuda.synchronize()
    assert L.status() == E_RANGE
    L.splat(pos, None, to_dev(np.minimum(batch, 63)), want_weight=False)
    L.distribute_pointnet(pos, feat, params, groups="default")
    assert L.status() == OK
