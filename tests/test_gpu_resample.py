"""GPU parity of downsampling (strided conv onto the coarse lattice) and
upsampling (transposed conv onto the fine lattice) against the CPU oracle,
through the C ABI.

The coarse lattice is the cloud's lattice at twice the scale.  Its key set
must match the oracle's bit for bit; vertex-side inputs are generated in
canonical order and laid out in each lattice's GPU vertex order; outputs are
compared on every vertex within 1e-5 of the sum of |terms| (fp32), and for
bf16 within 1e-5 against the oracle fed the same bf16-rounded inputs and 2e-2
against the unrounded ones.
"""
import numpy as np
import pytest
import torch

from datagen.clouds import conv_weight, make_workload, random_cloud, random_rows
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


def _pair(pos, sigma, batch=None, alpha=0.0):
    """Fine and coarse lattices of one cloud on one stream, splatted."""
    from paper_2108_03917_amd import Lattice

    s = torch.cuda.current_stream()
    sig = np.broadcast_to(np.asarray(sigma, dtype=np.float32), (pos.shape[1],))
    Lf = Lattice(pos.shape[1], sig, alpha=alpha, max_points=pos.shape[0], stream=s)
    Lc = Lattice(pos.shape[1], 2 * sig, alpha=alpha, max_points=pos.shape[0], stream=s)
    gf = GpuLattice(Lf, pos, None, batch=batch)
    gc = GpuLattice(Lc, pos, None, batch=batch)
    fine = O.build(pos, sig, alpha=alpha or None, batch=batch)
    coarse = O.coarsen(pos, sig, alpha=alpha or None, batch=batch)
    assert gf.V == fine.V and np.array_equal(gf.keys, fine.keys)
    assert gc.V == coarse.V and np.array_equal(gc.keys, coarse.keys)
    return Lf, Lc, gf, gc, fine, coarse


def _check(Lf, Lc, gf, gc, fine, coarse, c_in, c_out, dtype, seed, with_bias=False, out_dtype="f32"):
    T = Lf.taps
    W = conv_weight(c_in, c_out, fine.d, seed=seed)
    bias = random_rows(1, c_out, seed=seed + 9)[0] if with_bias else None
    Wd = to_dev(W)
    if dtype == "bf16":
        Wd = Lf.weights_to_bf16(Wd)
    bd = None if bias is None else to_dev(bias)
    tag = f"{c_in}->{c_out} {dtype} d={fine.d}"
    tol_out = (lambda ref: 2.0 ** -8 * np.abs(ref)) if out_dtype == "bf16" else (lambda ref: 0.0)

    # downsample: fine values -> coarse vertices
    x = random_rows(fine.V, c_in, seed=seed + 1)
    xin = gf.to_gpu_order(x)
    if dtype == "bf16":
        xin = xin.to(torch.bfloat16)
    y = Lf.downsample(Lc, xin, Wd, dtype=dtype, bias=bd, out_dtype=out_dtype)
    got = gc.from_gpu_order(y.float())
    if dtype == "bf16":
        xr = O.round_bf16(x.astype(np.float32))
        Wr = O.round_bf16(W.astype(np.float32))
        ref, sc = O.downsample(fine, coarse, xr, Wr, bias)
        assert_close_scaled(got, ref, REL_F32 * sc + tol_out(ref), 1.0, "downsample " + tag)
        ref32, sc32 = O.downsample(fine, coarse, x, W, bias)
        assert_close_scaled(got, ref32, REL_BF16 * sc32, 1.0, "downsample vs fp32 " + tag)
    else:
        ref, sc = O.downsample(fine, coarse, x, W, bias)
        assert_close_scaled(got, ref, REL_F32 * sc + tol_out(ref), 1.0, "downsample " + tag)

    # upsample: coarse values -> fine vertices
    yc = random_rows(coarse.V, c_in, seed=seed + 2)
    yin = gc.to_gpu_order(yc)
    if dtype == "bf16":
        yin = yin.to(torch.bfloat16)
    z = Lc.upsample(Lf, yin, Wd, dtype=dtype, bias=bd, out_dtype=out_dtype)
    got = gf.from_gpu_order(z.float())
    if dtype == "bf16":
        ref, sc = O.upsample(coarse, fine, O.round_bf16(yc.astype(np.float32)), O.round_bf16(W.astype(np.float32)),
                             bias)
    else:
        ref, sc = O.upsample(coarse, fine, yc, W, bias)
    assert_close_scaled(got, ref, REL_F32 * sc + tol_out(ref), 1.0, "upsample " + tag)
    # most fine vertices receive something: the test is not vacuous
    assert (np.abs(ref).sum(axis=1) > 0).mean() > 0.3


@pytest.mark.parametrize("d,sigma,c_in,c_out,dtype", [(3, 0.15, 64, 64, "f32"), (3, 0.15, 64, 64, "bf16"),
                                                      (3, 0.15, 64, 128, "bf16"), (4, 0.3, 64, 64, "bf16"),
                                                      (2, 0.08, 8, 16, "f32"), (3, 0.15, 5, 7, "f32"),
                                                      (1, 0.05, 4, 4, "f32")])
def test_resample_parity(d, sigma, c_in, c_out, dtype):
    w = random_cloud(6000, d, seed=400 + d, extent=1.0, C=2)
    Lf, Lc, gf, gc, fine, coarse = _pair(w.pos, sigma)
    _check(Lf, Lc, gf, gc, fine, coarse, c_in, c_out, dtype, seed=401 + c_in + c_out)


def test_resample_batched_with_bias_and_bf16_output():
    w = random_cloud(6000, 3, seed=410, extent=1.0, C=2, n_batch=4)
    Lf, Lc, gf, gc, fine, coarse = _pair(w.pos, 0.15, batch=w.batch)
    _check(Lf, Lc, gf, gc, fine, coarse, 64, 64, "bf16", seed=411, with_bias=True, out_dtype="bf16")


def test_resample_tables_follow_a_new_splat():
    """A second cloud splatted on the same two lattices rebuilds the cached
    cross-lattice tables (the tables of the first cloud would be wrong)."""
    from paper_2108_03917_amd import Lattice

    s = torch.cuda.current_stream()
    Lf = Lattice(3, 0.15, max_points=6000, stream=s)
    Lc = Lattice(3, 0.3, max_points=6000, stream=s)
    for rep in range(2):
        w = random_cloud(6000 - 2000 * rep, 3, seed=420 + rep, extent=1.0, C=2)
        gf = GpuLattice(Lf, w.pos, None)
        gc = GpuLattice(Lc, w.pos, None)
        fine, coarse = O.build(w.pos, 0.15), O.coarsen(w.pos, 0.15)
        assert np.array_equal(gf.keys, fine.keys) and np.array_equal(gc.keys, coarse.keys)
        _check(Lf, Lc, gf, gc, fine, coarse, 64, 64, "f32", seed=421 + rep)


def test_resample_rejects_mismatched_lattices():
    from paper_2108_03917_amd import Lattice, LatticeError

    s = torch.cuda.current_stream()
    pos = to_dev(random_cloud(500, 3, seed=430).pos)
    L3 = Lattice(3, 0.1, max_points=500, stream=s)
    L3b = Lattice(3, 0.2, max_points=500, stream=s)
    x = torch.zeros((L3.max_vertices(500), 8), device="cuda:0")
    W = torch.zeros((8, 9, 8), device="cuda:0")
    with pytest.raises(LatticeError):        # coarse not splatted yet
        L3.splat(pos)
        L3.downsample(L3b, x, W)
    L3b.splat(pos)
    # The two lattices in the wrong order, and a coarse scale that is not
    # twice the fine one, are refused before any launch.  (Buffers hold the
    # row bound of either lattice, so even a launch would stay in bounds.)
    xb = torch.zeros((2000, 8), device="cuda:0")
    with pytest.raises(LatticeError):
        L3.upsample(L3b, xb, W)           # source must be the coarse lattice
    with pytest.raises(LatticeError):
        L3b.downsample(L3, xb, W)         # source must be the fine lattice
    L4 = Lattice(3, 0.25, max_points=500, stream=s)
    L4.splat(pos)
    with pytest.raises(LatticeError):
        L3.downsample(L4, xb, W)          # sigma ratio 2.5, not 2
    y = L3.downsample(L3b, xb, W)         # the right pair works
    Vc = L3b.num_vertices()               # rows 0..V-1 are written
    assert Vc > 0 and torch.count_nonzero(y[:Vc]) == 0
    other = torch.cuda.Stream()
    L3c = Lattice(3, 0.2, max_points=500, stream=other)
    L3c.splat(pos)
    with pytest.raises(LatticeError):        # another stream
        L3.downsample(L3c, x, W)
    other.synchronize()


@pytest.mark.parametrize("config", [2, 5])
def test_resample_full_size(config):
    """The part-segmentation batch (16 x 2500 points, d = 3) and the four-scan
    space-time cloud (d = 4, about 4.2e5 points) at full size: every coarse
    and every fine vertex is compared."""
    w = make_workload(config)
    Lf, Lc, gf, gc, fine, coarse = _pair(w.pos, w.sigma, batch=w.batch)
    dtype = "f32" if config == 2 else "bf16"
    _check(Lf, Lc, gf, gc, fine, coarse, 64, 64, dtype, seed=440 + config)


# ---------------------------------------------------------------------------
# backward: the adjoints of both resamplings (input, weight and bias gradients)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,c_in,c_out,dtype,up", [
    (3, 64, 64, "f32", False), (3, 64, 64, "f32", True), (3, 64, 128, "bf16", False),
    (3, 128, 64, "bf16", True), (4, 64, 64, "bf16", False), (4, 32, 16, "f32", True),
    (2, 5, 7, "f32", False),
])
def test_resample_backward_parity(d, c_in, c_out, dtype, up):
    """Every input-row, weight and bias gradient of downsample (fine ->
    coarse) and upsample (coarse -> fine) against the oracle's conv_backward
    over the forward's cross table: within 1e-5 of the sum of |terms| against
    the oracle fed the same rounded operands (bf16: the operands rounded to
    bf16), and 2e-2 against the unrounded ones."""
    sigma = {2: 0.08, 3: 0.15, 4: 0.3}[d]
    w = random_cloud(6000, d, seed=400 + d + 10 * up, extent=1.0, C=1)
    Lf, Lc, gf, gc, fine, coarse = _pair(w.pos, sigma)
    src, dst = (coarse, fine) if up else (fine, coarse)
    gsrc, gdst = (gc, gf) if up else (gf, gc)
    Lsrc, Ldst = (Lc, Lf) if up else (Lf, Lc)
    seed = 410 + c_in + c_out
    x = random_rows(src.V, c_in, seed=seed)
    go = random_rows(dst.V, c_out, seed=seed + 1)
    W = conv_weight(c_in, c_out, d, seed=seed + 2)
    Wd = to_dev(W)
    if dtype == "bf16":
        Wd = Lsrc.weights_to_bf16(Wd)
    xd, gd = gsrc.to_gpu_order(x), gdst.to_gpu_order(go)
    fn = Lsrc.upsample_backward if up else Lsrc.downsample_backward
    gi, gw, gb = fn(Ldst, gd, Wd, xd, dtype=dtype, want_bias=True)
    gi = gsrc.from_gpu_order(gi.float())
    gw, gb = gw.cpu().numpy(), gb.cpu().numpy()
    bwd = O.upsample_backward if up else O.downsample_backward
    if dtype == "bf16":
        r = lambda a: O.round_bf16(a.astype(np.float32))
        xr, gr, Wr = r(x), r(go), r(W)
    else:
        xr, gr, Wr = x, go, W
    rx, rw, _, sx, sw, _ = bwd(src, dst, xr, Wr, gr)
    tag = f"{'up' if up else 'down'}sample {c_in}->{c_out} {dtype} d={d}"
    # a good share of the input rows receive a gradient (38% for d = 4
    # downsampling, whose strided taps reach fewer fine vertices; 63-100% else)
    assert (np.abs(rx).sum(axis=1) > 0).mean() > 0.3
    assert_close_scaled(gi, rx, sx, REL_F32, "grad_in " + tag)
    assert_close_scaled(gw, rw, sw, REL_F32, "grad_w " + tag)
    assert_close_scaled(gb, go.astype(np.float64).sum(axis=0), np.abs(go).sum(axis=0), REL_F32, "grad_bias " + tag)
    if dtype == "bf16":
        fx, fw, _, fsx, fsw, _ = bwd(src, dst, x, W, go)
        assert_close_scaled(gi, fx, fsx, REL_BF16, "grad_in vs fp32 " + tag)
        assert_close_scaled(gw, fw, fsw, REL_BF16, "grad_w vs fp32 " + tag)


def test_resample_backward_argument_checks():
    """Lattices in the wrong order and an input gradient aliasing the output
    gradient are refused before any launch."""
    from paper_2108_03917_amd import LatticeError

    w = random_cloud(2000, 3, seed=420, extent=1.0, C=1)
    Lf, Lc, gf, gc, fine, coarse = _pair(w.pos, 0.15)
    W = to_dev(conv_weight(8, 8, 3, seed=421))
    go = torch.zeros((fine.V, 8), device="cuda:0")
    x = torch.zeros((fine.V, 8), device="cuda:0")
    with pytest.raises(LatticeError):
        Lc.downsample_backward(Lf, go, W, x)          # coarse passed as the fine lattice
    import ctypes
    from paper_2108_03917_amd.lattice import F32, load_library
    lib = load_library()
    p = ctypes.c_void_p(go.data_ptr())
    st = lib.lattice_downsample_backward(Lf._h, Lc._h, p, F32, 8, ctypes.c_void_p(W.data_ptr()), 8, F32,
                                         ctypes.c_void_p(x.data_ptr()), F32, p, F32, None, None)
    assert st != 0
