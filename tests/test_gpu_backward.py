"""GPU parity of the backward passes (slice, splat, conv) against the CPU
oracle, through the C ABI.

Each gradient is compared element by element with the oracle's float64
definition on the same seeded inputs: vertex-side inputs are generated in
canonical (sorted-key) order and permuted into the GPU's vertex order, so the
oracle never sees a value produced by the HIP path.  Bar: |gpu - ref| <= rel *
A, A the oracle's sum of |terms| of that element; rel = 1e-5 for fp32, and for
bf16 computations 1e-5 against the oracle fed the same bf16-rounded inputs and
2e-2 against the unrounded ones.
"""
import numpy as np
import pytest
import torch

from datagen.clouds import conv_weight, deform_weights, make_workload, random_cloud, random_rows
from oracle import lattice_oracle as O
from tests.gpu_util import REL_BF16, REL_F32, GpuLattice, assert_close_scaled, to_dev

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


def _lattice(d, sigma, m, **kw):
    from paper_2108_03917_amd import Lattice

    return Lattice(d, sigma, max_points=max(m, 1), **kw)


def _setup(d, m, sigma, seed, C=4, pos=None):
    if pos is None:
        w = random_cloud(m, d, seed=seed, extent=1.0, C=C)
        pos = w.pos
    L = _lattice(d, sigma, pos.shape[0])
    g = GpuLattice(L, pos, None)
    lat = O.build(pos, sigma)
    assert g.V == lat.V and np.array_equal(g.keys, lat.keys)
    return L, g, lat


def _clustered(seed, m_dense=6000, m_sparse=3000):
    """Tight clusters (vertices with thousands of pairs: the split gather)
    plus a sparse background."""
    rng = np.random.default_rng(seed)
    centres = rng.uniform(-0.8, 0.8, size=(3, 3))
    dense = centres[rng.integers(0, 3, m_dense)] + rng.normal(0, 0.01, size=(m_dense, 3))
    sparse = rng.uniform(-1, 1, size=(m_sparse, 3))
    return np.concatenate([dense, sparse]).astype(np.float32)[rng.permutation(m_dense + m_sparse)]


# ---------------------------------------------------------------------------
# slice backward = Eq. (splat) of the point gradients
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,m,sigma,C,out_dtype", [(3, 6000, 0.15, 64, "f32"), (4, 5000, 0.3, 16, "f32"),
                                                   (2, 4000, 0.08, 5, "f32"), (3, 5000, 0.15, 64, "bf16")])
def test_slice_backward_parity(d, m, sigma, C, out_dtype):
    L, g, lat = _setup(d, m, sigma, seed=300 + d)
    gout = random_rows(m, C, seed=301 + d)
    got = L.slice_backward(to_dev(gout), out_dtype=out_dtype)
    ref, scale = O.slice_backward(lat, gout)
    tol = REL_F32 * scale
    if out_dtype == "bf16":
        tol = tol + 2.0 ** -8 * np.abs(ref)
    assert_close_scaled(g.from_gpu_order(got.float()), ref, tol, 1.0, f"slice backward d={d} C={C}")


def test_slice_backward_long_pair_lists():
    """Vertices hit by thousands of points: their lists are summed in parts."""
    pos = _clustered(60)
    L, g, lat = _setup(3, pos.shape[0], 0.1, 0, pos=pos)
    counts = np.bincount(lat.idx.reshape(-1), minlength=lat.V)
    assert counts.max() > 500
    gout = random_rows(pos.shape[0], 96, seed=61)
    got = L.slice_backward(to_dev(gout))
    ref, scale = O.slice_backward(lat, gout)
    assert_close_scaled(g.from_gpu_order(got), ref, scale, REL_F32, "slice backward, split lists")


# ---------------------------------------------------------------------------
# splat backward = Eq. (slice) of the vertex gradients
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,m,sigma,C,normalize,gv_dtype", [(3, 6000, 0.15, 64, False, "f32"),
                                                            (3, 6000, 0.15, 64, True, "f32"),
                                                            (4, 4000, 0.3, 8, True, "f32"),
                                                            (3, 3000, 0.12, 7, False, "f32"),
                                                            (3, 4000, 0.15, 32, False, "bf16")])
def test_splat_backward_parity(d, m, sigma, C, normalize, gv_dtype):
    w = random_cloud(m, d, seed=320 + d, extent=1.0, C=3)
    L = _lattice(d, sigma, m)
    g = GpuLattice(L, w.pos, w.feat, normalize=normalize)
    lat = O.build(w.pos, sigma)
    assert np.array_equal(g.keys, lat.keys)
    _, wref, _ = O.splat(lat, w.feat)
    gv = random_rows(lat.V, C, seed=321 + d)
    if gv_dtype == "bf16":
        gv = O.round_bf16(gv.astype(np.float32))
    gv_dev = g.to_gpu_order(gv).to(torch.bfloat16 if gv_dtype == "bf16" else torch.float32)
    got = L.splat_backward(gv_dev, normalize=normalize, weight=g.weight_dev if normalize else None)
    ref, scale = O.splat_backward(lat, gv, normalize=normalize, weight=wref)
    # the normalised form adds the rounding of w_v and of b / w_v
    rel = (3 if normalize else 1) * REL_F32
    assert_close_scaled(got.cpu().numpy(), ref, scale, rel, f"splat backward d={d} normalize={normalize}")


# ---------------------------------------------------------------------------
# conv backward: input gradient (flipped weights on the forward kernels) and
# weight / bias gradients (chunked product over the vertices)
# ---------------------------------------------------------------------------

def _conv_case(L, g, lat, c_in, c_out, dtype, seed, x_dtype="f32", g_dtype="f32", want_bias=True):
    nbr = O.neighbors(lat)
    x = random_rows(lat.V, c_in, seed=seed)
    go = random_rows(lat.V, c_out, seed=seed + 1)
    W = conv_weight(c_in, c_out, lat.d, seed=seed + 2)
    if x_dtype == "bf16":
        x = O.round_bf16(x.astype(np.float32))
    if g_dtype == "bf16":
        go = O.round_bf16(go.astype(np.float32))
    xd = g.to_gpu_order(x).to(torch.bfloat16 if x_dtype == "bf16" else torch.float32)
    gd = g.to_gpu_order(go).to(torch.bfloat16 if g_dtype == "bf16" else torch.float32)
    Wd = to_dev(W)
    if dtype == "bf16":
        Wd = L.weights_to_bf16(Wd)
    gi, gw, gb = L.conv_backward(gd, Wd, xd, dtype=dtype, want_bias=want_bias)
    gi = g.from_gpu_order(gi.float())
    gw = gw.cpu().numpy()
    gb = gb.cpu().numpy() if gb is not None else None
    if dtype == "bf16":
        xr, gr, Wr = O.round_bf16(x.astype(np.float32)), O.round_bf16(go.astype(np.float32)), \
            O.round_bf16(W.astype(np.float32))
    else:
        xr, gr, Wr = x, go, W
    rx, rw, rb, sx, sw, sb = O.conv_backward(xr, nbr, Wr, gr)
    tag = f"{c_in}->{c_out} {dtype} d={lat.d}"
    assert_close_scaled(gi, rx, sx, REL_F32, "conv grad_in " + tag)
    assert_close_scaled(gw, rw, sw, REL_F32, "conv grad_w " + tag)
    if gb is not None:
        # the bias gradient sums the unrounded output gradient
        rbu = go.astype(np.float64).sum(axis=0)
        assert_close_scaled(gb, rbu, np.abs(go).sum(axis=0), REL_F32, "conv grad_bias " + tag)
    if dtype == "bf16":
        fx, fw, _, fsx, fsw, _ = O.conv_backward(x, nbr, W, go)
        assert_close_scaled(gi, fx, fsx, REL_BF16, "conv grad_in vs fp32 " + tag)
        assert_close_scaled(gw, fw, fsw, REL_BF16, "conv grad_w vs fp32 " + tag)


@pytest.mark.parametrize("d,c_in,c_out,dtype", [(3, 64, 64, "f32"), (3, 64, 128, "bf16"), (3, 128, 128, "bf16"),
                                                (4, 64, 64, "bf16"), (3, 8, 16, "f32"), (2, 5, 7, "f32"),
                                                (3, 96, 32, "f32")])
def test_conv_backward_parity(d, c_in, c_out, dtype):
    sigma = {2: 0.1, 3: 0.15, 4: 0.3}[d]
    L, g, lat = _setup(d, 5000, sigma, seed=340 + d)
    _conv_case(L, g, lat, c_in, c_out, dtype, seed=341 + c_in + c_out)


def test_conv_backward_bf16_storage():
    """bf16-stored input rows and output gradients (as a bf16 network keeps them)."""
    L, g, lat = _setup(3, 5000, 0.15, seed=350)
    _conv_case(L, g, lat, 64, 64, "bf16", seed=351, x_dtype="bf16", g_dtype="bf16")


def test_conv_backward_empty_lattice():
    L = _lattice(3, 0.1, 16)
    L.splat(torch.zeros((0, 3), device="cuda:0"), None)
    assert L.num_vertices() == 0
    W = torch.randn((16, L.taps, 8), device="cuda:0")
    gi, gw, gb = L.conv_backward(torch.zeros((1, 16), device="cuda:0"), W, torch.zeros((1, 8), device="cuda:0"),
                                 want_bias=True)
    torch.cuda.synchronize()
    assert torch.count_nonzero(gw) == 0 and torch.count_nonzero(gb) == 0


@pytest.mark.parametrize("d,C,n_cls,bf16", [
    (3, 64, 20, False), (3, 64, 0, False), (4, 64, 26, True), (2, 16, 3, False), (3, 200, 0, False),
    (3, 1024, 5, False), (1, 5, 0, False), (3, 128, 64, True), (4, 16, 7, False), (3, 4, 0, False)])
def test_deform_slice_backward_parity(d, C, n_cls, bf16):
    """Every gradient of DeformSlice (and its classifier): the vertex values
    (pulled over the pair lists), the offsets' weights and bias, the
    classifier's weights and bias, against the oracle's float64 backward
    (the max routed to the first float32 maximum, the decision the kernel
    takes).  Shapes: one to sixteen channel chunks per lane, bf16 rows, d = 1..4."""
    sigma = {1: 0.05, 2: 0.1, 3: 0.15, 4: 0.3}[d]
    L, g, lat = _setup(d, 5000, sigma, seed=380 + d + C)
    y = random_rows(lat.V, C, seed=381 + C)
    if bf16:
        y = O.round_bf16(y.astype(np.float32)).astype(np.float32)
    yd = g.to_gpu_order(y)
    if bf16:
        yd = yd.to(torch.bfloat16)
    dw = deform_weights(C, max(n_cls, 1), seed=382 + C)
    with_cls = n_cls > 0
    G = random_rows(L.m, n_cls if with_cls else C, seed=383 + C)
    wc = to_dev(dw.w_cls) if with_cls else None
    gv, gwd, gbd, gwc, gbc = L.deform_slice_backward(yd, to_dev(dw.w_delta), dw.b_delta, to_dev(G), wc)
    (rX, rw, rb, rWc, rbc), (sX, sw, sb, sWc, sbc) = O.deform_slice_backward(
        lat.idx, lat.bary, y, dw.w_delta, dw.b_delta, G, lat.V, dw.w_cls if with_cls else None)
    tag = f"deform backward d={d} C={C} n_cls={n_cls} bf16={bf16}"
    assert_close_scaled(g.from_gpu_order(gv), rX, sX, REL_F32, tag + " values")
    assert_close_scaled(gwd.cpu().numpy(), rw, sw, REL_F32, tag + " w_delta")
    assert_close_scaled(gbd.cpu().numpy(), np.array([rb]), np.array([sb]), REL_F32, tag + " b_delta")
    if with_cls:
        assert_close_scaled(gwc.cpu().numpy(), rWc, sWc, REL_F32, tag + " w_cls")
        assert_close_scaled(gbc.cpu().numpy(), rbc, sbc, REL_F32, tag + " b_cls")
    else:
        assert gwc is None and gbc is None


@pytest.mark.parametrize("C,n_cls,bf16", [(64, 20, False), (128, 7, True), (16, 0, False)])
def test_deform_slice_backward_long_pair_lists(C, n_cls, bf16):
    """DeformSlice backward on clustered clouds: vertices with thousands of
    pairs are summed in parts of 32 entries (part rows added in part order),
    next to short lists; twice on one lattice, the second cloud smaller, so
    that no part record or list entry of the first splat leaks into the
    second."""
    L = _lattice(3, 0.1, 9000)
    for rep, (md, ms) in enumerate([(6000, 3000), (2500, 700)]):
        pos = _clustered(70 + rep, md, ms)
        g = GpuLattice(L, pos, None)
        lat = O.build(pos, 0.1)
        assert g.V == lat.V and np.array_equal(g.keys, lat.keys)
        counts = np.bincount(lat.idx.reshape(-1), minlength=lat.V)
        assert counts.max() > 500 and (counts > 32).sum() >= 3 and (counts <= 32).sum() > 100
        y = random_rows(lat.V, C, seed=71 + C + rep)
        if bf16:
            y = O.round_bf16(y.astype(np.float32)).astype(np.float32)
        yd = g.to_gpu_order(y)
        if bf16:
            yd = yd.to(torch.bfloat16)
        dw = deform_weights(C, max(n_cls, 1), seed=72 + C)
        with_cls = n_cls > 0
        G = random_rows(pos.shape[0], n_cls if with_cls else C, seed=73 + C + rep)
        gv, gwd, gbd, gwc, gbc = L.deform_slice_backward(yd, to_dev(dw.w_delta), dw.b_delta, to_dev(G),
                                                          to_dev(dw.w_cls) if with_cls else None)
        (rX, rw, rb, rWc, rbc), (sX, sw, sb, sWc, sbc) = O.deform_slice_backward(
            lat.idx, lat.bary, y, dw.w_delta, dw.b_delta, G, lat.V, dw.w_cls if with_cls else None)
        tag = f"deform backward, split lists C={C} n_cls={n_cls} rep={rep}"
        assert_close_scaled(g.from_gpu_order(gv), rX, sX, REL_F32, tag + " values")
        assert_close_scaled(gwd.cpu().numpy(), rw, sw, REL_F32, tag + " w_delta")
        if with_cls:
            assert_close_scaled(gwc.cpu().numpy(), rWc, sWc, REL_F32, tag + " w_cls")
            assert_close_scaled(gbc.cpu().numpy(), rbc, sbc, REL_F32, tag + " b_cls")


@pytest.mark.parametrize("n_cls", [0, 20])
def test_deform_slice_backward_empty_cloud(n_cls):
    """An empty cloud after a non-empty one on the same lattice: no pairs, so
    the offsets' and the classifier's gradients are zero (sums of no
    points); the per-list work reads nothing of the earlier splat's lists."""
    L = _lattice(3, 0.15, 4000)
    pos = random_cloud(4000, 3, seed=395, extent=1.0, C=1).pos
    L.splat(to_dev(pos), None)
    L.splat(torch.zeros((0, 3), device="cuda:0"), None)
    assert L.num_vertices() == 0 and L.m == 0
    C = 64
    dw = deform_weights(C, max(n_cls, 1), seed=396)
    y = torch.randn((L.max_vertices(), C), device="cuda:0")
    G = torch.zeros((1, n_cls if n_cls else C), device="cuda:0")
    wc = to_dev(dw.w_cls) if n_cls else None
    _, gwd, gbd, gwc, gbc = L.deform_slice_backward(y, to_dev(dw.w_delta), dw.b_delta, G, wc)
    torch.cuda.synchronize()
    assert torch.count_nonzero(gwd) == 0 and torch.count_nonzero(gbd) == 0
    if n_cls:
        assert torch.count_nonzero(gwc) == 0 and torch.count_nonzero(gbc) == 0


def test_deform_slice_backward_without_offsets_is_slice_backward():
    """Zero offset weights and bias: db = 0, so the vertex gradient of the
    point features is the slice's backward (the splat of grad_out), and the
    offsets' weight gradient is sum_pk (gf . x_k)(q_pk - mx_p)."""
    L, g, lat = _setup(3, 5000, 0.15, seed=390)
    y = random_rows(lat.V, 32, seed=391)
    G = random_rows(L.m, 32, seed=392)
    z = torch.zeros(32, device="cuda:0")
    gv, _, _, _, _ = L.deform_slice_backward(g.to_gpu_order(y), z, 0.0, to_dev(G))
    ref = L.slice_backward(to_dev(G))
    V = g.V
    assert torch.allclose(gv[:V], ref[:V], rtol=1e-5, atol=1e-6)


def test_deform_slice_backward_argument_checks():
    from paper_2108_03917_amd import LatticeError

    L, g, lat = _setup(3, 2000, 0.15, seed=393)
    y = torch.zeros((L.max_vertices(), 8), device="cuda:0")
    G = torch.zeros((L.m, 8), device="cuda:0")
    with pytest.raises(LatticeError):     # no output requested
        L.deform_slice_backward(y, torch.zeros(8, device="cuda:0"), 0.0, G, want_values=False, want_w_delta=False,
                                want_b_delta=False)


def test_backward_repeatable_bits():
    """The weight gradient adds its vertex chunks in a fixed order: two calls
    give identical bits."""
    L, g, lat = _setup(3, 6000, 0.15, seed=360)
    x = g.to_gpu_order(random_rows(lat.V, 64, seed=361))
    go = g.to_gpu_order(random_rows(lat.V, 64, seed=362))
    W = to_dev(conv_weight(64, 64, 3, seed=363))
    a = L.conv_backward(go, W, x, want_bias=True)
    b = L.conv_backward(go, W, x, want_bias=True)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_backward_stages_at_partseg_size():
    """Every backward stage of the part-segmentation step (16 x 2500 points,
    d = 3, sigma = 0.04; slice -> conv 64->64 bf16 -> conv 64->64 fp32 ->
    splat) at full size, in the benchmark's launch configuration.  Each stage
    takes the oracle's own input for that stage (laid out in GPU order), so
    the rounding of one stage does not feed the next; every point gradient
    and every weight gradient is compared."""
    w = make_workload(2)
    L = _lattice(3, w.sigma, w.m)
    g = GpuLattice(L, w.pos, w.feat, batch=w.batch)
    lat = O.build(w.pos, w.sigma, batch=w.batch)
    assert np.array_equal(g.keys, lat.keys)
    nbr = O.neighbors(lat)
    W0, W1 = w.convs[0].weight, w.convs[1].weight
    vals, _, _ = O.splat(lat, w.feat)
    y0, _ = O.conv(vals, nbr, W0)
    y0r = O.round_bf16(y0.astype(np.float32))
    gout = random_rows(w.m, W1.shape[0], seed=370)

    gy1, gy1_s = O.slice_backward(lat, gout)
    gy1_d = L.slice_backward(to_dev(gout))
    assert_close_scaled(g.from_gpu_order(gy1_d), gy1, gy1_s, REL_F32, "partseg slice backward")

    gy1r = O.round_bf16(gy1.astype(np.float32))
    W1r = O.round_bf16(W1.astype(np.float32))
    gx1, gw1, _, gx1_s, gw1_s, _ = O.conv_backward(y0r, nbr, W1r, gy1r)
    gx1_d, gw1_d, _ = L.conv_backward(g.to_gpu_order(gy1r).to(torch.bfloat16), L.weights_to_bf16(to_dev(W1)),
                                      g.to_gpu_order(y0r).to(torch.bfloat16), dtype="bf16")
    assert_close_scaled(g.from_gpu_order(gx1_d), gx1, gx1_s, REL_F32, "partseg conv1 (bf16) grad_in")
    assert_close_scaled(gw1_d.cpu().numpy(), gw1, gw1_s, REL_F32, "partseg conv1 (bf16) grad_w")

    gx0, gw0, _, gx0_s, gw0_s, _ = O.conv_backward(vals, nbr, W0, gx1)
    gx0_d, gw0_d, _ = L.conv_backward(g.to_gpu_order(gx1), to_dev(W0), g.to_gpu_order(vals), dtype="f32")
    assert_close_scaled(g.from_gpu_order(gx0_d), gx0, gx0_s, REL_F32, "partseg conv0 (fp32) grad_in")
    assert_close_scaled(gw0_d.cpu().numpy(), gw0, gw0_s, REL_F32, "partseg conv0 (fp32) grad_w")

    gf, gf_s = O.splat_backward(lat, gx0)
    gf_d = L.splat_backward(g.to_gpu_order(gx0))
    assert_close_scaled(gf_d.cpu().numpy(), gf, gf_s, REL_F32, "partseg splat backward")
