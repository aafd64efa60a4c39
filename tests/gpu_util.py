"""Helpers for GPU parity tests: run the HIP path, canonicalise its vertex
order by sorted key, and compare against the CPU oracle.

The GPU assigns vertex indices in hash-insertion order, which is not
deterministic.  Every comparison first maps GPU vertex g to its canonical
index rank[g] (ascending (batch, c_0, .., c_{d-1}), the oracle's order).
Inputs that feed a single stage (conv, slice) are generated in canonical
order from a seed and permuted into GPU order, so the oracle never sees a
value produced by the HIP path.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import lattice_oracle as O

REL_F32 = 1e-5     # fp32 splat / slice / conv, relative to the sum of |terms|
REL_BF16 = 2e-2    # bf16 MFMA conv against the fp32-input oracle
BARY_ABS = 1e-5    # barycentric weights, absolute


def dev():
    return torch.device("cuda:0")


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).to(dev())
    return t if dtype is None else t.to(dtype)


def canonical_perm(keys: np.ndarray, vbatch, d: int):
    """perm: canonical position -> GPU row;  rank: GPU row -> canonical position."""
    cols = [keys[:, i] for i in reversed(range(d))]
    if vbatch is not None:
        cols.append(vbatch)
    perm = np.lexsort(cols) if len(keys) else np.zeros(0, dtype=np.int64)
    rank = np.empty_like(perm)
    rank[perm] = np.arange(len(perm))
    return perm, rank


class GpuLattice:
    """Splat a workload on the GPU and read back the canonicalised lattice."""

    def __init__(self, L, pos, feat=None, batch=None, normalize=False):
        self.L = L
        d = L.d
        self.values_dev, self.weight_dev = L.splat(to_dev(pos), None if feat is None else to_dev(feat),
                                                   None if batch is None else to_dev(batch), normalize=normalize)
        self.V = L.num_vertices()
        if batch is not None:
            k, vb = L.keys(with_batch=True)
            self.keys_raw = k.cpu().numpy().astype(np.int64)
            self.vb_raw = vb.cpu().numpy().astype(np.int64)
        else:
            self.keys_raw = L.keys().cpu().numpy().astype(np.int64)
            self.vb_raw = None
        self.perm, self.rank = canonical_perm(self.keys_raw, self.vb_raw, d)
        self.keys = self.keys_raw[self.perm]
        self.vbatch = None if self.vb_raw is None else self.vb_raw[self.perm]
        idx, bary = L.point_simplex()
        idx = idx.cpu().numpy().astype(np.int64)
        self.idx_raw = idx
        self.idx = np.where(idx >= 0, self.rank[np.maximum(idx, 0)], -1)
        self.bary = bary.cpu().numpy().astype(np.float64)

    def values(self):
        if self.values_dev is None:
            return None
        return self.values_dev[: self.V].cpu().numpy().astype(np.float64)[self.perm]

    def weight(self):
        return self.weight_dev[: self.V].cpu().numpy().astype(np.float64)[self.perm]

    def neighbors(self):
        nbr = self.L.neighbors().cpu().numpy().astype(np.int64)[self.perm]
        return np.where(nbr >= 0, self.rank[np.maximum(nbr, 0)], -1)

    def to_gpu_order(self, canon: np.ndarray) -> torch.Tensor:
        """Rows given in canonical order, laid out in GPU vertex order (fp32)."""
        return to_dev(np.ascontiguousarray(canon[self.rank], dtype=np.float32))

    def from_gpu_order(self, t: torch.Tensor) -> np.ndarray:
        return t[: self.V].cpu().numpy().astype(np.float64)[self.perm]


def assert_close_scaled(got, ref, scale, rel, what, atol=1e-30):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    err = np.abs(got - ref)
    bound = rel * np.asarray(scale, dtype=np.float64) + atol
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {err.size} elements out of tolerance; worst at {i}: "
                             f"got {got[i]!r} ref {ref[i]!r} scale {np.asarray(scale)[i]!r} rel {rel}")
    ratio = float((err / (np.asarray(scale) + 1e-300)).max()) if err.size else 0.0
    return ratio


def check_lattice(g: GpuLattice, lat: O.Lattice):
    """Bit-exact key set, per-point vertices; weights within BARY_ABS."""
    assert g.V == lat.V, (g.V, lat.V)
    assert np.array_equal(g.keys, lat.keys)
    assert np.all(g.keys.sum(axis=1) == 0)
    if lat.vbatch is not None:
        assert np.array_equal(g.vbatch, lat.vbatch)
    assert np.array_equal(g.idx, lat.idx)
    assert np.abs(g.bary - lat.bary).max(initial=0.0) <= BARY_ABS

