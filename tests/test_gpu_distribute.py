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


# --------------------------------------------------------------------------
# backward: the gradients of every block's parameters
# --------------------------------------------------------------------------

def _unpack(flat, k0):
    """Split a packed parameter vector into (a, s, W, b) per block."""
    out, at, K = [], 0, k0
    for w in (16, 32, 64):
        a = flat[at:at + K]; at += K
        s = flat[at:at + K]; at += K
        W = flat[at:at + w * K].reshape(w, K); at += w * K
        b = flat[at:at + w]; at += w
        out.append((a, s, W, b))
        K = w
    return out


def _abs_backward(blocks, seg, seed, inject, use_gn, actual=False):
    """The backward's sum of |terms| per parameter: the oracle's backward
    with every quantity replaced by its magnitude (products of magnitudes,
    the group normalisation's mean terms added), seeded with ``seed``
    [E, 64] at the last block's output and ``inject[l]`` [E, K_l] added at
    each block's normalised input gradient.  The forward's activations enter
    by their forward scale (sum of |terms|), or with ``actual`` by their own
    magnitude: where the forward rounds to well within 1e-5 of its values
    (no large cancellation), the latter bounds the backward's rounding
    without multiplying the forward's cancellations into every term."""
    out = []
    dh = seed
    for li in range(len(blocks) - 1, -1, -1):
        blk = blocks[li]
        r_m = np.abs(blk["r"]) if actual else blk["r_s"]
        x_m = np.abs(blk["xhat"]) if actual else blk["xhat_s"]
        db = dh.sum(axis=0)
        dW = dh.T @ r_m
        dr = dh @ np.abs(blk["W"])
        dhn = dr * (blk["hn"] > 0) + inject[li]
        da = (dhn * x_m).sum(axis=0)
        ds = dhn.sum(axis=0)
        g = np.abs(blk["a"]) * dhn
        if use_gn:
            G = blk["G"]
            dh = blk["rstd"] * (g + O._group_mean(g, seg, G) + x_m * O._group_mean(g * x_m, seg, G))
        else:
            dh = g
        out.append((da, ds, dW, db))
    return out[::-1]


def _gn_layers_plain(k0, d, seed):
    """Group-normalisation parameters with gamma = 1 and beta = 0 (about half
    of the normalised inputs negative: both ReLU branches taken), block 1's
    weights of the position channels zero (a vertex with one row has its
    local mean at its point, so those channels are zero)."""
    out = []
    for li, (ga, be, W, b) in enumerate(pointnet_gn_weights(k0, seed=seed)):
        if li == 0:
            W = W.copy()
            W[:, :d] = 0.0
        out.append((np.ones_like(ga), np.zeros_like(be), W, b))
    return out


def _forward_scales(blocks, layers, h_s):
    """Per block the forward's sum-of-|terms| scale of xhat and of the ReLU
    input; returns the last block's output scale."""
    for li, blk in enumerate(blocks):
        a = np.abs(blk["a"])
        mean_abs = np.abs(blk["h"] - blk["xhat"] / blk["rstd"])
        xs = (h_s + mean_abs) * blk["rstd"]
        hn_s = a * xs + np.abs(blk["hn"] - blk["a"] * blk["xhat"])
        blk["xhat_s"], blk["r_s"] = xs, hn_s
        h_s = hn_s @ np.abs(blk["W"]).T + np.abs(np.asarray(layers[li][3], np.float64))
    return h_s


# A float32 evaluation of this graph rounds at most about 96 times along any
# path (h0; per block the affine's two operations and a dot product of up to
# 32 terms; the statistics' finalisation), so its error is at most gamma_96 =
# 96 u / (1 - 96 u), u = 2^-24, times the sum of |terms|: the band within
# which a float32 evaluation may decide a max or a ReLU the other way.
_U = 2.0 ** -24
_BAND = 96 * _U / (1 - 96 * _U)


def _setup_backward(pos, feat, sigma, layers, groups, batch=None, seed=0):
    from paper_2108_03917_amd import Lattice

    d = pos.shape[1]
    L = Lattice(d, sigma, max_points=max(pos.shape[0], 1))
    g = GpuLattice(L, pos, None, batch=batch)
    lat = O.build(pos, sigma, batch=batch)
    assert np.array_equal(g.keys, lat.keys)
    params = Lattice.pack_pointnet(layers).to("cuda:0")
    G = np.random.default_rng(seed + 1).standard_normal((lat.V, 64)).astype(np.float32)
    gp = L.distribute_pointnet_backward(to_dev(pos), None if feat is None else to_dev(feat), params,
                                        g.to_gpu_order(G), groups=groups, eps=1e-5)
    got = _unpack(gp.cpu().numpy().astype(np.float64), d + (0 if feat is None else feat.shape[1]))
    ref, am, h3, v, blocks, seg = O.distribute_pointnet_backward(lat, pos, feat, layers, G, groups=groups, eps=1e-5)
    h3_s = _forward_scales(blocks, layers, O.distribute_rows(lat, pos, feat)[5])
    return lat, G, got, ref, am, h3, h3_s, v, blocks, seg


@pytest.mark.parametrize("d,f_d,groups,batched", [(3, 3, "default", False), (4, 1, "default", False),
                                                  (2, 2, (2, 4, 8), False), (3, 2, "default", True)])
def test_distribute_pointnet_backward_parity(d, f_d, groups, batched):
    """Every block's parameter gradients (gamma, beta, W, b) with group
    normalisation against the oracle's float64 backward on a sparse cloud
    (every pair its own vertex: each vertex has one row, so the max decides
    nothing; the entry counts 12000, 15000 and 9000 leave the last chunk of
    64 lanes partly empty, whose lanes must add nothing although the group
    means give every row an input gradient).  Bar: 1e-5 of the backward's sum of |terms| at the forward's
    values, plus, for each ReLU input within float32 rounding of zero (a
    handful; the test counts them), the whole effect of the other branch.
    Batched: four clouds (batch ids 0, 3, 7, 11) drawn per point, so that
    most wavefronts' rows span clouds and their group sums go per cloud."""
    m = 3000
    rng = np.random.default_rng(580 + d + (10 if batched else 0))
    pos = rng.uniform(0.0, 1.0, (m, d)).astype(np.float32)
    feat = rng.standard_normal((m, f_d)).astype(np.float32)
    batch = rng.choice(np.array([0, 3, 7, 11], dtype=np.int32), size=m) if batched else None
    k0 = d + f_d
    og = [min(32, k) for k in (k0, 16, 32)] if groups == "default" else list(groups)
    layers = _gn_layers_plain(k0, d, seed=581 + d)
    sigma = 0.0001 if d == 2 else 0.0005      # small enough that no two points share a vertex
    lat, G, got, ref, am, h3, h3_s, v, blocks, seg = _setup_backward(pos, feat, sigma, layers, og, batch=batch,
                                                                     seed=582)
    assert np.bincount(v).max() == 1                                      # one row per vertex
    if batched:
        assert len(np.unique(seg)) == 4
    E = h3.shape[0]
    seed_abs = np.zeros((E, 64))
    vv, cc = np.nonzero(am >= 0)
    np.add.at(seed_abs, (am[vv, cc], cc), np.abs(G[vv, cc]))
    scale = _abs_backward(blocks, seg, seed_abs, [np.zeros_like(b["hn"]) for b in blocks], True, actual=True)
    # the real input gradient of each block's ReLU, for the branches in doubt
    dh = np.zeros((E, 64))
    np.add.at(dh, (am[vv, cc], cc), G[vv, cc])
    inj, n_doubt = [None] * 3, 0
    for li in range(2, -1, -1):
        blk = blocks[li]
        dr = dh @ blk["W"]
        doubt = (np.abs(blk["hn"]) <= _BAND * blk["r_s"]) & (blk["hn"] != 0.0)   # exact zeros decide alike
        inj[li] = np.where(doubt, np.abs(dr), 0.0)
        n_doubt += int(doubt.sum())
        gn_ = blk["a"] * (dr * (blk["hn"] > 0))
        Gc = blk["G"]
        dh = blk["rstd"] * (gn_ - O._group_mean(gn_, seg, Gc) - blk["xhat"] * O._group_mean(gn_ * blk["xhat"], seg, Gc))
    assert n_doubt <= 100, n_doubt
    allow = _abs_backward(blocks, seg, np.zeros((E, 64)), inj, True, actual=True)
    names = ("gamma", "beta", "W", "b")
    for li in range(3):
        for q in range(4):
            assert_close_scaled(got[li][q], ref[li][q], REL_F32 * scale[li][q] + allow[li][q], 1.0,
                                f"pointnet backward d={d} block {li + 1} d{names[q]}")


def _sites_cloud(d, n_sites, per, seed, sigma):
    """Sites far apart (no two share a lattice vertex), each ``per`` points
    within one simplex, point i of a site with features 1 + i + U(0, 0.5):
    every vertex's rows are its site's points, one per point, and with
    positive weights the last point wins every channel by a wide margin."""
    rng = np.random.default_rng(seed)
    side = int(np.ceil(n_sites ** (1.0 / d)))
    grid = np.stack(np.meshgrid(*[np.arange(side)] * d, indexing="ij"), -1).reshape(-1, d)[:n_sites]
    centres = grid * 40.0 * sigma + rng.uniform(0, 10 * sigma, size=(n_sites, d))
    pos = np.repeat(centres, per, axis=0) + rng.normal(0, 0.002 * sigma, size=(n_sites * per, d))
    base = np.tile(np.arange(per, dtype=np.float64), n_sites)[:, None]
    feat = 1.0 + base + rng.uniform(0, 0.5, size=(n_sites * per, 4))
    return pos.astype(np.float32), feat.astype(np.float32)


def _positive_affine_layers(k0, d, seed):
    """Fixed-affine parameters with a = 1, s = 0 (s = 3 on the position
    channels, whose weights are zero), W ~ U(0.05, 0.3), b ~ U(0, 0.1): with
    positive features every activation is positive, far from the ReLU's
    kink, and free of cancellation."""
    rng = np.random.default_rng(seed)
    out, K = [], k0
    for w in (16, 32, 64):
        a = np.ones(K, np.float32)
        s_ = np.zeros(K, np.float32)
        W = rng.uniform(0.05, 0.3, size=(w, K)).astype(np.float32)
        if K == k0:
            s_[:d] = 3.0
            W[:, :d] = 0.0
        b = rng.uniform(0.0, 0.1, size=w).astype(np.float32)
        out.append((a, s_, W, b))
        K = w
    return out


@pytest.mark.parametrize("d,per", [(2, 3), (3, 3), (4, 3), (3, 150), (4, 150)])
def test_distribute_pointnet_backward_routing(d, per):
    """Several rows per vertex (the points of a site: three, or 150 so that
    every list crosses 64-row chunks and its winner is found from the runs
    of several chunks) with the fixed affine: the max routes each g[v][c] to
    the winning row, then every block's parameter gradients (a, s, W, b)
    match the oracle within 1e-5 of their sum of |terms|.  Positive weights
    and features keep every decision far outside float32 rounding, which the
    test checks first."""
    sigma = 0.05
    pos, feat = _sites_cloud(d, 400 if per == 3 else 60, per, 600 + d + per, sigma)
    k0 = d + 4
    layers = _positive_affine_layers(k0, d, 601)
    lat, G, got, ref, am, h3, h3_s, v, blocks, seg = _setup_backward(pos, feat, sigma, layers, None, seed=602)
    cnt = np.bincount(v)
    assert (cnt == per).mean() > 0.9
    order = np.argsort(v, kind="stable")
    starts = np.searchsorted(v[order], np.arange(lat.V))
    ends = np.searchsorted(v[order], np.arange(lat.V), side="right")
    for u in range(lat.V):
        rows = order[starts[u]:ends[u]]
        top = h3[am[u], np.arange(64)]
        other = rows[:, None] != am[u][None, :]
        gap = top[None, :] - h3[rows]
        bound = _BAND * (h3_s[rows] + h3_s[am[u], np.arange(64)][None, :])
        assert not np.any(other & (gap <= bound)), "a maximum within rounding of another row"
    for blk in blocks:
        assert np.all(np.abs(blk["hn"]) > _BAND * blk["r_s"]), "a ReLU input within rounding of zero"
    E = h3.shape[0]
    seed_abs = np.zeros((E, 64))
    vv, cc = np.nonzero(am >= 0)
    np.add.at(seed_abs, (am[vv, cc], cc), np.abs(G[vv, cc]))
    scale = _abs_backward(blocks, seg, seed_abs, [np.zeros_like(b["hn"]) for b in blocks], False)
    for li in range(3):
        for q, name in enumerate(("a", "s", "W", "b")):
            assert_close_scaled(got[li][q], ref[li][q], scale[li][q], REL_F32,
                                f"pointnet backward routing d={d} block {li + 1} d{name}")


def test_distribute_pointnet_backward_repeatable_and_checks():
    """Five clouds drawn per point (several rows per vertex, waves spanning
    clouds) with group normalisation: two calls give identical bits (every
    sum in a fixed order), the gradients are finite and not all zero.  A
    missing output or too few rows of grad_out are refused before any
    launch."""
    from paper_2108_03917_amd import Lattice, LatticeError

    w = random_cloud(6000, 3, seed=620, extent=1.0, C=3, n_batch=5)
    L = Lattice(3, 0.15, max_points=w.m)
    g = GpuLattice(L, w.pos, None, batch=w.batch)
    layers = pointnet_gn_weights(6, seed=621)
    params = Lattice.pack_pointnet(layers).to("cuda:0")
    G = to_dev(np.random.default_rng(622).standard_normal((L.max_vertices(), 64)).astype(np.float32))
    pos, feat = to_dev(w.pos), to_dev(w.feat)
    a = L.distribute_pointnet_backward(pos, feat, params, G, groups="default")
    b = L.distribute_pointnet_backward(pos, feat, params, G, groups="default")
    assert torch.equal(a, b)
    assert torch.isfinite(a).all() and a.abs().max() > 0
    with pytest.raises(ValueError):
        L.distribute_pointnet_backward(pos, feat, params, G[:10], groups="default")
    import ctypes
    from paper_2108_03917_amd.lattice import load_library
    lib = load_library()
    widths = (ctypes.c_int * 3)(16, 32, 64)
    st = lib.lattice_distribute_pointnet_backward(L._h, ctypes.c_void_p(pos.data_ptr()),
                                                  ctypes.c_void_p(feat.data_ptr()), 3,
                                                  ctypes.c_void_p(params.data_ptr()), 3, widths, None,
                                                  ctypes.c_float(1e-5), ctypes.c_void_p(G.data_ptr()), None)
    assert st != 0
    bad = (ctypes.c_int * 3)(16, 32, 32)
    out = torch.empty_like(params)
    st = lib.lattice_distribute_pointnet_backward(L._h, ctypes.c_void_p(pos.data_ptr()),
                                                  ctypes.c_void_p(feat.data_ptr()), 3,
                                                  ctypes.c_void_p(params.data_ptr()), 3, bad, None,
                                                  ctypes.c_float(1e-5), ctypes.c_void_p(G.data_ptr()),
                                                  ctypes.c_void_p(out.data_ptr()))
    assert st != 0
