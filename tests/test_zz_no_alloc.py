"""The allocation-free conv backward (lattice_conv_backward_noalloc) against
the allocating one (lattice_conv_backward), through the C ABI.

Both run the same kernels with the same vertex chunking; the no-alloc entry
point keeps its flipped weights and weight-gradient partials in the
library's fixed per-GPU workspace.  So the input, weight and bias gradients
must be bit-identical to the allocating entry point's (which is checked
against the oracle in the backward parity tests).  Two calls in a row share
the workspace, the second on a smaller lattice with another shape, so that
what the first left behind must not leak into the second.  A shape whose
scratch exceeds the workspace is refused before anything is enqueued.
"""
import numpy as np
import pytest
import torch

from datagen.clouds import conv_weight, random_cloud, random_rows

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


def _case(d, m, sigma, c_in, c_out, dtype, seed):
    from paper_2108_03917_amd import Lattice

    dev = "cuda:0"
    w = random_cloud(m, d, seed=seed, extent=1.0, C=4)
    L = Lattice(d, sigma, max_points=m)
    L.splat(torch.from_numpy(w.pos).to(dev), None, want_weight=False)
    V = L.num_vertices()
    rows = L.max_vertices(m)
    x = torch.from_numpy(random_rows(rows, c_in, seed=seed + 1)).to(dev)
    g = torch.from_numpy(random_rows(rows, c_out, seed=seed + 2)).to(dev)
    W = torch.from_numpy(conv_weight(c_in, c_out, d, seed=seed + 3)).to(dev)
    if dtype == "bf16":
        W = L.weights_to_bf16(W)
    T = 2 * (d + 1) + 1
    outs = []
    for noalloc in (False, True):
        gi = torch.full((rows, c_in), float("nan"), device=dev)
        gw = torch.full((c_out, T, c_in), float("nan"), device=dev)
        gb = torch.full((c_out,), float("nan"), device=dev)
        L.conv_backward(g, W, x, dtype=dtype, grad_in=gi, grad_w=gw, grad_bias=gb, noalloc=noalloc)
        torch.cuda.synchronize()
        outs.append((gi[:V].cpu(), gw.cpu(), gb.cpu()))
    for a, b, name in zip(outs[0], outs[1], ("grad_in", "grad_w", "grad_bias")):
        assert torch.isfinite(a).all(), name
        assert torch.equal(a, b), f"{name}: no-alloc differs from the allocating entry point (d={d}, {c_in}->{c_out})"
    return L


def test_noalloc_conv_backward_matches_allocating_entry_point():
    # a 20k-point lattice, 128 -> 128 fp32 (the largest partial buffers) ...
    L1 = _case(3, 20000, 0.1, 128, 128, "f32", seed=900)
    # ... then, sharing the workspace, a smaller d = 4 lattice (11 taps), 64 -> 32 in bf16
    L2 = _case(4, 4000, 0.3, 64, 32, "bf16", seed=910)
    L1.close()
    L2.close()


def test_noalloc_conv_backward_refuses_shapes_above_the_workspace():
    from paper_2108_03917_amd import Lattice, LatticeError

    dev = "cuda:0"
    w = random_cloud(2000, 3, seed=920, extent=1.0, C=4)
    L = Lattice(3, 0.1, max_points=w.m)
    L.splat(torch.from_numpy(w.pos).to(dev), None, want_weight=False)
    rows = L.max_vertices(w.m)
    g = torch.zeros((rows, 512), device=dev)
    x = torch.zeros((rows, 512), device=dev)
    W = torch.zeros((512, 9, 512), device=dev)
    with pytest.raises(LatticeError):   # 512 x 9 x 512 fp32 weights alone exceed 24 MiB with the partials
        L.conv_backward(g, W, x, dtype="f32", want_bias=True, noalloc=True)
    torch.cuda.synchronize()
    L.close()
