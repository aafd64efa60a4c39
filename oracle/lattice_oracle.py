"""Plain CPU oracle of the sparse permutohedral-lattice hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module: only the tests, the smoke check and the CPU-baseline leg of the
benchmark use it.  It shares no code with the HIP library.

It follows the paper (Rosu et al., "LatticeNet", arXiv 2108.03917):

* Sec. "Permutohedral Lattice": the lattice is (d+1)Z^{d+1} projected along
  the all-ones vector onto the hyperplane H_d; vertex coordinates sum to zero;
  the enclosing simplex of a point comes from a simple rounding algorithm
  (cited there to Baek & Adams); each vertex has 2(d+1) neighbours at
  +-[-1,..,-1,d,-1,..,-1]; vertices are stored sparsely in a hash map.
* Sec. "Method": positions are scaled as G / sigma.
* Sec. "Common Operations on Permutohedral Lattice": splat (barycentric
  weighting onto the d+1 simplex vertices, summed), convolve over the 1-hop
  ring of 2(d+1)+1 vertices (an unallocated neighbour counts as zero, caption
  of the convolution figure), slice (the inverse of splat with the same
  weights).
* Eq. (splat): x_v = sum_{p in J_v} b_pv f_p.   Eq. (slice): f_p = sum_{v in I_p} b_pv x_v.

Precision.  Where floating point decides an integer (which simplex encloses a
point, hence every lattice key), this oracle takes that decision in float32
with one fixed sequence of individually rounded operations, no fused
multiply-add, exactly as the HIP kernel does: the paper fixes no precision,
and bit-exact keys need both sides to round the same way.  Everything that is
an output value (barycentric weights, splat, conv, slice) is computed in
float64 from those float32 elevated coordinates.

Readings of the paper taken here (the paper is silent on them):

* Elevation: x = alpha * E * (g / sigma), with E the orthonormal basis of H_d
  whose j-th column is (1,..,1,-j,0,..,0)/sqrt(j(j+1)) (j ones).  Default
  alpha = (d+1) sqrt(2/3), the scale of the lattice-filtering work the paper
  builds on.  alpha is a parameter.
* Rounding to the remainder-0 point uses round-half-to-even on x * fl(1/(d+1)).
* Rank ties: the lower coordinate index ranks first (rank 0 = largest).
* All d+1 vertices of every point's simplex are allocated, zero weight or not.
* Splat output is the raw sum of Eq. (splat) plus the weight channel
  w_v = sum b_pv; the optional normalised form divides by w_v (0 where w_v=0).
* Tap order of the 1-ring: tap 0 is the vertex itself, tap 1+j is c + n_j and
  tap d+2+j is c - n_j (j = 0..d), with n_j = (d+1) e_j - 1.
* Conv weight layout [C_out][T][C_in]: y_v[o] = sum_t sum_i x_{nbr(v,t)}[i] W[o,t,i].
* Batched clouds are independent lattices; canonical vertex order is
  ascending (batch, c_0, .., c_{d-1}).
* Distribute + PointNet: each block normalises its input rows with a group
  normalisation (Sec. "Implementation": 32 groups by default) whose
  statistics are taken over all the rows of one cloud (one batch id); with
  fewer than 32 channels, or a count that 32 does not divide, the group count
  is the largest divisor of the channel count not above 32.

Parity unpinned: alpha, the rounding-tie rule and the rank-tie rule are
conventions that the paper does not fix; both sides adopt the ones above.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import scipy.sparse as sp

F32 = np.float32


def default_alpha(d: int) -> float:
    """Default elevation scale (d+1) sqrt(2/3) (reading of Sec. "Permutohedral Lattice")."""
    return (d + 1) * np.sqrt(2.0 / 3.0)


def scale_factors(d: int, sigma, alpha: Optional[float] = None) -> np.ndarray:
    """Per-axis float32 factors f_j = alpha / (sigma_{j-1} sqrt(j(j+1))), j = 1..d.

    Folds the position scaling G / sigma (Sec. "Method") into the orthonormal
    elevation basis.  Computed in float64, rounded once to float32."""
    if alpha is None or alpha <= 0:
        alpha = default_alpha(d)
    sig = np.broadcast_to(np.asarray(sigma, dtype=F32), (d,))
    out = np.empty(d, dtype=F32)
    for j in range(1, d + 1):
        out[j - 1] = F32(float(alpha) / (np.float64(sig[j - 1]) * np.sqrt(np.float64(j * (j + 1)))))
    return out


def elevate(pos: np.ndarray, factors: np.ndarray) -> np.ndarray:
    """Elevate d-dim points onto H_d in float32 (Sec. "Permutohedral Lattice").

    x_d = -d s_d ;  x_i = (s_{i+1} + .. + s_d) - i s_i ;  x_0 = s_1 + .. + s_d,
    with s_j = g_{j-1} f_j.  The running sum goes from j = d down to 1 and
    every product and sum is rounded to float32 on its own."""
    pos = np.asarray(pos, dtype=F32)
    m, d = pos.shape
    x = np.empty((m, d + 1), dtype=F32)
    S = np.zeros(m, dtype=F32)
    for j in range(d, 0, -1):
        s = pos[:, j - 1] * F32(factors[j - 1])          # float32 product
        t = F32(j) * s                                   # float32 product
        x[:, j] = S - t                                  # float32 difference
        S = S + s                                        # float32 sum
    x[:, 0] = S
    return x


def enclosing_simplex(x: np.ndarray):
    """Remainder-0 point and ranks of the enclosing simplex (Sec. "Permutohedral Lattice").

    Steps of the rounding algorithm the paper cites:
      1. r_i = (d+1) * round(x_i / (d+1))                       (remainder-0 point)
      2. rank_i = position of Delta_i = x_i - r_i in descending order (ties: lower i first)
      3. s = sum r_i / (d+1); rank += s, and coordinates whose rank leaves
         [0, d] wrap around by -+(d+1) with r_i moved by -+(d+1).
    Returns (r int64 [m, d+1], rank int64 [m, d+1]); sum(r) == 0 afterwards."""
    x = np.asarray(x, dtype=F32)
    m, dp1 = x.shape
    inv = F32(1.0 / dp1)
    q = np.rint(x * inv)                                 # float32 product, round-half-even
    r = q.astype(np.int64) * dp1
    delta = x - r.astype(F32)                            # float32 difference
    gt = delta[:, None, :] > delta[:, :, None]           # [p, i, j]: Delta_j > Delta_i
    eq = delta[:, None, :] == delta[:, :, None]
    lower = np.arange(dp1)[None, :] < np.arange(dp1)[:, None]   # [i, j]: j < i
    rank = gt.sum(axis=2) + (eq & lower[None]).sum(axis=2)
    rank = rank.astype(np.int64)
    s = r.sum(axis=1) // dp1
    rank = rank + s[:, None]
    neg = rank < 0
    big = rank > dp1 - 1
    rank[neg] += dp1
    r[neg] += dp1
    rank[big] -= dp1
    r[big] -= dp1
    return r, rank


def barycentric(x: np.ndarray, r: np.ndarray, rank: np.ndarray) -> np.ndarray:
    """Barycentric weights b_k of the d+1 simplex vertices, in float64.

    With delta_i = (x_i - r_i) / (d+1) and z_q the delta whose rank is q
    (z_0 >= .. >= z_d):  b_k = z_{d-k} - z_{d+1-k} for k = 1..d and
    b_0 = 1 - (z_0 - z_d).  Vertex k is the one with remainder k (see
    ``simplex_keys``).  The weights are >= 0 and sum to 1."""
    x = np.asarray(x, dtype=np.float64)
    m, dp1 = x.shape
    d = dp1 - 1
    delta = (x - r) / dp1
    z = np.empty_like(delta)
    np.put_along_axis(z, rank, delta, axis=1)            # z[p, rank_i] = delta_i
    b = np.empty((m, dp1))
    for k in range(1, d + 1):
        b[:, k] = z[:, d - k] - z[:, d + 1 - k]
    b[:, 0] = 1.0 - (z[:, 0] - z[:, d])
    return b


def simplex_keys(r: np.ndarray, rank: np.ndarray) -> np.ndarray:
    """Integer keys of the d+1 simplex vertices: [m, k, i] (Sec. "Permutohedral Lattice").

    Vertex k has c_i = r_i + k when rank_i <= d - k, else r_i + k - (d+1);
    every coordinate of vertex k is congruent to k mod (d+1) and each key
    sums to zero."""
    m, dp1 = r.shape
    d = dp1 - 1
    keys = np.empty((m, dp1, dp1), dtype=np.int64)
    for k in range(dp1):
        keys[:, k, :] = r + k - dp1 * (rank > d - k)
    return keys


@dataclass
class Lattice:
    d: int
    keys: np.ndarray            # int64 [V, d+1], canonical order
    vbatch: Optional[np.ndarray]  # int64 [V] batch id of each vertex, or None
    idx: np.ndarray             # int64 [m, d+1]: vertex of remainder k for point p
    bary: np.ndarray            # float64 [m, d+1]
    x: np.ndarray               # float32 [m, d+1] elevated positions
    B: sp.csr_matrix            # [m, V] barycentric weight matrix

    @property
    def V(self) -> int:
        return int(self.keys.shape[0])

    @property
    def m(self) -> int:
        return int(self.idx.shape[0])


def _single(pos, factors):
    x = elevate(pos, factors)
    r, rank = enclosing_simplex(x)
    b = barycentric(x, r, rank)
    keys = simplex_keys(r, rank)
    return x, b, keys


def build(pos: np.ndarray, sigma, alpha: Optional[float] = None,
          batch: Optional[np.ndarray] = None) -> Lattice:
    """Allocate the sparse lattice of a cloud: vertex set V, I_p and b_pv (Sec. "Notation").

    The vertex set is the set of distinct keys over all points' simplices;
    with ``batch`` each batch id is its own lattice and the vertex lists are
    concatenated in batch order."""
    pos = np.asarray(pos, dtype=F32)
    m, d = pos.shape
    fac = scale_factors(d, sigma, alpha)
    x, b, keys = _single(pos, fac)
    flat = keys.reshape(m * (d + 1), d + 1)[:, :d]      # c_d is implied by the zero sum
    if batch is not None:
        bcol = np.repeat(np.asarray(batch, dtype=np.int64), d + 1)[:, None]
        flat = np.concatenate([bcol, flat], axis=1)
    uniq, inv = np.unique(flat, axis=0, return_inverse=True)
    inv = inv.reshape(m, d + 1)
    if batch is not None:
        vbatch = uniq[:, 0].copy()
        coords = uniq[:, 1:]
    else:
        vbatch = None
        coords = uniq
    full = np.concatenate([coords, -coords.sum(axis=1, keepdims=True)], axis=1)
    V = full.shape[0]
    B = sp.csr_matrix((b.ravel(), (np.repeat(np.arange(m), d + 1), inv.ravel())), shape=(m, V))
    return Lattice(d, full, vbatch, inv, b, x, B)


def splat(lat: Lattice, feat: np.ndarray, normalize: bool = False):
    """Eq. (splat): x_v = sum_{p in J_v} b_pv f_p, in float64.

    Returns (values [V, C], weight [V], scale [V, C]) where weight is
    w_v = sum_p b_pv and scale = sum_p |b_pv f_p| (the magnitude against which
    rounding error of any summation order is measured).  With ``normalize``
    the values are x_v / w_v (0 where w_v = 0)."""
    f = np.asarray(feat, dtype=np.float64)
    Bt = lat.B.T.tocsr()
    values = Bt @ f
    weight = np.asarray(Bt.sum(axis=1)).ravel()
    scale = abs(Bt) @ np.abs(f)
    if normalize:
        with np.errstate(divide="ignore", invalid="ignore"):
            nz = weight != 0
            values = np.where(nz[:, None], values / np.where(nz, weight, 1.0)[:, None], 0.0)
            scale = np.where(nz[:, None], scale / np.where(nz, weight, 1.0)[:, None], 0.0)
    return values, weight, scale


def neighbor_offsets(d: int) -> np.ndarray:
    """Tap offsets [T, d+1]: 0, then +n_j, then -n_j, n_j = (d+1) e_j - 1 (Sec. "Permutohedral Lattice")."""
    n = (d + 1) * np.eye(d + 1, dtype=np.int64) - 1
    return np.concatenate([np.zeros((1, d + 1), dtype=np.int64), n, -n], axis=0)


def neighbors(lat: Lattice) -> np.ndarray:
    """1-ring table [V, T]: vertex index of key + offset_t, -1 when not allocated."""
    d = lat.d
    cols = ([("b", np.int64)] if lat.vbatch is not None else []) + [(f"c{i}", np.int64) for i in range(d)]
    dt = np.dtype(cols)

    def pack(coords, vb):
        rec = np.empty(coords.shape[0], dtype=dt)
        if vb is not None:
            rec["b"] = vb
        for i in range(d):
            rec[f"c{i}"] = coords[:, i]
        return rec

    table = pack(lat.keys, lat.vbatch)                  # canonical order is sorted
    offs = neighbor_offsets(d)
    nbr = np.full((lat.V, offs.shape[0]), -1, dtype=np.int64)
    for t, o in enumerate(offs):
        q = pack(lat.keys + o, lat.vbatch)
        pos = np.searchsorted(table, q)
        hit = pos < lat.V
        hit[hit] = table[pos[hit]] == q[hit]
        nbr[hit, t] = pos[hit]
    return nbr


def conv(values: np.ndarray, nbr: np.ndarray, weight: np.ndarray, bias: Optional[np.ndarray] = None):
    """1-ring lattice convolution in float64 (Sec. "Common Operations": Convolving).

    y_v = sum_t x_{nbr(v,t)} W_t^T (+ bias), with an absent neighbour
    contributing zero.  ``weight`` is [C_out][T][C_in].  Returns (y, scale)
    with scale = sum_t |x_{nbr(v,t)}| |W_t|^T."""
    x = np.asarray(values, dtype=np.float64)
    W = np.asarray(weight, dtype=np.float64)
    V = nbr.shape[0]            # one output row per table row (the input rows may be another lattice's)
    c_out, T, c_in = W.shape
    y = np.zeros((V, c_out))
    scale = np.zeros((V, c_out))
    for t in range(T):
        present = nbr[:, t] >= 0
        g = np.zeros((V, c_in))
        g[present] = x[nbr[present, t]]
        y += g @ W[:, t, :].T
        scale += np.abs(g) @ np.abs(W[:, t, :]).T
    if bias is not None:
        y += np.asarray(bias, dtype=np.float64)[None, :]
        scale += np.abs(np.asarray(bias, dtype=np.float64))[None, :]
    return y, scale


def slice_(lat: Lattice, values: np.ndarray):
    """Eq. (slice): f_p = sum_{v in I_p} b_pv x_v, in float64.  Returns (out, scale)."""
    y = np.asarray(values, dtype=np.float64)
    return lat.B @ y, abs(lat.B) @ np.abs(y)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even), returned as float32.

    Standard bit method: add 0x7FFF plus the lowest kept bit, then clear the
    low 16 bits.  Inputs here are finite."""
    u = np.ascontiguousarray(a, dtype=F32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    return u.view(F32)


def deform_slice(idx: np.ndarray, bary: np.ndarray, values: np.ndarray, w_delta: np.ndarray, b_delta: float,
                 w_cls: Optional[np.ndarray] = None, b_cls: Optional[np.ndarray] = None,
                 with_delta_scale: bool = False):
    """DeformSlice (Sec. "Proposed Operations", DeformSlicing; Eq. deformSlice),
    optionally followed by the final linear classifier (Sec. "Implementation":
    the two are one fused operation).  float64 throughout.

    For point p with simplex vertices v = idx[p, k] and weights b_pk, in the
    paper's order:
      Gather       q_pk = b_pk x_v                                  [m, d+1, C]
      MaxPool      mx_p = max over the d+1 vertices of q_pk, per channel
      SubtractMax  q_pk - mx_p
      Linear+Tanh  db_pk = tanh(b_delta + (q_pk - mx_p) . w_delta)  [m, d+1]
      slice        f_p = sum_k (b_pk + db_pk) x_v                   [m, C]
      classifier   logits_p = f_p W_cls^T + b_cls                   [m, n_cls]
    The max runs over all d+1 vertices, v included (the formula; the prose
    says "the other vertices").  The nonlinearity is tanh (the network
    figure's Linear+Tanh).

    Returns (out, delta, scale): out is f or the logits, delta the offsets,
    and scale the magnitude against which a float32 evaluation's rounding is
    measured: for f, sum_k (|b| + |db|)|x| plus sum_k |x| times the tanh
    argument's sum of |terms| (tanh has slope at most 1); for the logits,
    that scale and |f| carried through |W_cls| plus |b_cls|.  With
    with_delta_scale a fourth item follows: the tanh argument's sum of
    |terms| [m, d+1], the scale of the offsets' rounding (plus tanh's own
    few ulps)."""
    idx = np.asarray(idx, dtype=np.int64)
    b = np.asarray(bary, dtype=np.float64)
    X = np.asarray(values, dtype=np.float64)
    w = np.asarray(w_delta, dtype=np.float64)
    m, dp1 = idx.shape
    C = X.shape[1]
    rows = np.zeros((m, dp1, C))
    valid = idx >= 0
    rows[valid] = X[idx[valid]]
    q = b[:, :, None] * rows                                  # Gather
    mx = q.max(axis=1)                                        # MaxPool
    diff = q - mx[:, None, :]                                 # SubtractMax
    arg = b_delta + diff @ w                                  # Linear
    delta = np.tanh(arg)                                      #   + Tanh
    f = ((b + delta)[:, :, None] * rows).sum(axis=1)          # slice with b + db
    arg_scale = abs(b_delta) + (np.abs(q) + np.abs(mx)[:, None, :]) @ np.abs(w)
    absrows = np.abs(rows)
    f_scale = ((np.abs(b) + np.abs(delta))[:, :, None] * absrows).sum(axis=1) \
        + (arg_scale[:, :, None] * absrows).sum(axis=1)
    extra = (arg_scale,) if with_delta_scale else ()
    if w_cls is None:
        return (f, delta, f_scale) + extra
    Wc = np.asarray(w_cls, dtype=np.float64)                  # [n_cls, C]
    logits = f @ Wc.T
    scale = (f_scale + np.abs(f)) @ np.abs(Wc).T
    if b_cls is not None:
        bc = np.asarray(b_cls, dtype=np.float64)
        logits = logits + bc
        scale = scale + np.abs(bc)
    return (logits, delta, scale) + extra


def deform_slice_backward(idx: np.ndarray, bary: np.ndarray, values: np.ndarray, w_delta: np.ndarray,
                          b_delta: float, grad_out: np.ndarray, V: int, w_cls: Optional[np.ndarray] = None,
                          b_cls: Optional[np.ndarray] = None):
    """Gradients of deform_slice (with or without the classifier) given
    grad_out = dL/dout [m, n_cls or C], float64, written from the forward's
    steps in reverse:
      classifier   gf_p = grad_out_p W_cls, dW_cls = grad_out^T f, db_cls = sum_p grad_out_p
      slice        dx_pk += (b_pk + db_pk) gf_p,  ddb_pk = gf_p . x_pk
      Tanh         darg_pk = ddb_pk (1 - db_pk^2)
      Linear       dw_delta = sum_pk darg_pk (q_pk - mx_p),  db_delta = sum_pk darg_pk,
                   d(q_pk - mx_p) = darg_pk w_delta
      SubtractMax  dq_pk += darg_pk w_delta,  dmx_p = -(sum_k darg_pk) w_delta
      MaxPool      dq_{p,k*,c} += dmx_{p,c} for k* the maximising vertex of channel c
      Gather       dx_pk += b_pk dq_pk, and dX_v = sum of dx_pk over the pairs with v_pk = v
    The max routes its gradient to one vertex per channel, a decision that
    rounding can flip near a tie, so it is taken in float32 as a float32
    evaluation makes it: on the products float32(b_pk) * float32(x_pk), the
    first (lowest k) of equal maxima winning.  Invalid vertices (index -1)
    read a zero row and receive nothing.
    Returns (dX [V, C], dw_delta [C], db_delta, dW_cls or None, db_cls or
    None) and their scales (dX_scale, dw_scale, db_scale, dW_cls_scale,
    db_cls_scale): sums of |terms|, with the offsets' rounding (the forward's
    tanh-argument scale) carried through b + db and 1 - db^2."""
    idx = np.asarray(idx, dtype=np.int64)
    b = np.asarray(bary, dtype=np.float64)
    X = np.asarray(values, dtype=np.float64)
    w = np.asarray(w_delta, dtype=np.float64)
    G = np.asarray(grad_out, dtype=np.float64)
    m, dp1 = idx.shape
    C = X.shape[1]
    valid = idx >= 0
    rows = np.zeros((m, dp1, C))
    rows[valid] = X[idx[valid]]
    # forward quantities
    q = b[:, :, None] * rows
    mx = q.max(axis=1)
    diff = q - mx[:, None, :]
    delta = np.tanh(b_delta + diff @ w)
    f = ((b + delta)[:, :, None] * rows).sum(axis=1)
    _, _, f_scale, arg_scale = deform_slice(idx, bary, values, w_delta, b_delta, with_delta_scale=True)
    # the maximising vertex of each channel, decided in float32
    q32 = np.asarray(bary, dtype=np.float32)[:, :, None] * rows.astype(np.float32)
    am = q32.argmax(axis=1)                                   # first of equal maxima
    onehot = am[:, None, :] == np.arange(dp1)[None, :, None]  # [m, dp1, C]
    # classifier
    if w_cls is not None:
        Wc = np.asarray(w_cls, dtype=np.float64)
        gf = G @ Wc
        gs = np.abs(G) @ np.abs(Wc)
        dWc = G.T @ f
        dWc_s = np.abs(G).T @ (f_scale + np.abs(f))
        dbc = G.sum(axis=0)
        dbc_s = np.abs(G).sum(axis=0)
    else:
        gf, gs = G, np.abs(G)
        dWc = dWc_s = dbc = dbc_s = None
    # slice, Tanh
    ddelta = np.einsum("pkc,pc->pk", rows, gf)
    darg = ddelta * (1.0 - delta ** 2)
    S = darg.sum(axis=1)
    # Linear
    dw = np.einsum("pk,pkc->c", darg, diff)
    dbd = darg.sum()
    # SubtractMax, MaxPool, Gather: the gradient of each pair's row
    dx = ((b + delta)[:, :, None] * gf[:, None, :]
          + (b * darg)[:, :, None] * w[None, None, :]
          - (b * S[:, None])[:, :, None] * onehot * w[None, None, :])
    dX = np.zeros((V, C))
    np.add.at(dX, idx[valid], dx[valid])
    # scales
    absrows = np.abs(rows)
    dds = np.einsum("pkc,pc->pk", absrows, gs)
    darg_s = dds + np.abs(ddelta) * 2.0 * np.abs(delta) * arg_scale
    S_s = darg_s.sum(axis=1)
    dx_s = ((np.abs(b) + np.abs(delta) + arg_scale)[:, :, None] * gs[:, None, :]
            + (np.abs(b) * (darg_s + S_s[:, None]))[:, :, None] * np.abs(w)[None, None, :])
    dX_s = np.zeros((V, C))
    np.add.at(dX_s, idx[valid], dx_s[valid])
    dw_s = np.einsum("pk,pkc->c", darg_s, np.abs(q) + np.abs(mx)[:, None, :])
    return (dX, dw, dbd, dWc, dbc), (dX_s, dw_s, darg_s.sum(), dWc_s, dbc_s)


# ---------------------------------------------------------------------------
# Backward passes (Sec. "Implementation": the network is trained end to end,
# so every lattice operation needs the gradient of a loss with respect to its
# inputs).  Each one is the transpose of the forward linear map, written out
# as its own definition: the derivative of a scalar loss L through
# y = forward(x) is dL/dx = J^T dL/dy, with J the forward's Jacobian.
# ---------------------------------------------------------------------------

def slice_backward(lat: Lattice, grad_out: np.ndarray):
    """Gradient of Eq. (slice) with respect to the vertex values, float64.

    f_p = sum_k b_pk y_{idx[p,k]}  gives  dL/dy_v = sum over the (p, k) with
    idx[p, k] = v of b_pk dL/df_p: each point scatters its gradient onto its
    d+1 simplex vertices with the barycentric weights.  Returns (grad [V, C],
    scale = the same sum of |terms|)."""
    g = np.asarray(grad_out, dtype=np.float64)
    m, dp1 = lat.idx.shape
    out = np.zeros((lat.V, g.shape[1]))
    scale = np.zeros_like(out)
    for k in range(dp1):
        v = lat.idx[:, k]
        b = lat.bary[:, k][:, None]
        np.add.at(out, v, b * g)
        np.add.at(scale, v, np.abs(b * g))
    return out, scale


def splat_backward(lat: Lattice, grad_values: np.ndarray, normalize: bool = False,
                   weight: Optional[np.ndarray] = None):
    """Gradient of Eq. (splat) with respect to the point features, float64.

    Raw splat x_v = sum_p b_pv f_p gives dL/df_p = sum_k b_pk dL/dx_{idx[p,k]}.
    The normalised splat x_v / w_v (w_v = sum_p b_pv does not depend on f)
    divides each vertex's gradient by w_v first (0 where w_v = 0, where the
    forward value is the constant 0).  Returns (grad [m, C], scale)."""
    g = np.asarray(grad_values, dtype=np.float64)
    if normalize:
        w = np.asarray(weight, dtype=np.float64)
        inv = np.zeros_like(w)
        inv[w != 0] = 1.0 / w[w != 0]
        g = g * inv[:, None]
    m, dp1 = lat.idx.shape
    out = np.zeros((m, g.shape[1]))
    scale = np.zeros_like(out)
    for k in range(dp1):
        b = lat.bary[:, k][:, None]
        rows = g[lat.idx[:, k]]
        out += b * rows
        scale += np.abs(b * rows)
    return out, scale


def conv_backward(values: np.ndarray, nbr: np.ndarray, weight: np.ndarray, grad_out: np.ndarray):
    """Gradients of the 1-ring convolution (Sec. "Common Operations":
    Convolving), float64.

    y_v[o] = sum_t sum_i x_{nbr(v,t)}[i] W[o,t,i] (+ bias[o]) gives
      dL/dx_u[i]   = sum over (v, t) with nbr(v,t) = u of sum_o g_v[o] W[o,t,i]
                     (each output row scatters back along the tap it read);
      dL/dW[o,t,i] = sum_v g_v[o] x_{nbr(v,t)}[i]   (absent taps read zero);
      dL/dbias[o]  = sum_v g_v[o].
    Returns (grad_x, grad_w, grad_bias) and their sum-of-|terms| scales
    (grad_x_scale, grad_w_scale, grad_bias_scale)."""
    x = np.asarray(values, dtype=np.float64)
    W = np.asarray(weight, dtype=np.float64)
    g = np.asarray(grad_out, dtype=np.float64)
    V = x.shape[0]
    c_out, T, c_in = W.shape
    gx = np.zeros((V, c_in))
    gx_s = np.zeros((V, c_in))
    gw = np.zeros((c_out, T, c_in))
    gw_s = np.zeros((c_out, T, c_in))
    for t in range(T):
        present = nbr[:, t] >= 0
        src = nbr[present, t]
        np.add.at(gx, src, g[present] @ W[:, t, :])
        np.add.at(gx_s, src, np.abs(g[present]) @ np.abs(W[:, t, :]))
        gw[:, t, :] = g[present].T @ x[src]
        gw_s[:, t, :] = np.abs(g[present]).T @ np.abs(x[src])
    return gx, gw, g.sum(axis=0), gx_s, gw_s, np.abs(g).sum(axis=0)


# ---------------------------------------------------------------------------
# Downsampling and upsampling (Sec. "Proposed Operations": Downsampling,
# Upsampling, and the caption of the Coarsen figure).
#
# A coarse lattice is the lattice of the same cloud with the positions
# divided by 2 (the same as doubling sigma: halving is exact in float32).
# Downsampling: coarse vertex c' is embedded in the fine lattice as 2c' and
# convolves over the fine vertices 2c' + offset_t (the 1-ring offsets), a
# strided convolution.  Upsampling: fine vertex u is embedded in the coarse
# lattice as u/2 and convolves over the coarse vertices (u + offset_t)/2; a
# tap whose key has a fractional coordinate (it lies inside a coarse
# simplex) contributes nothing, as does a tap whose vertex is not allocated.
# This makes upsampling a transposed convolution.
# ---------------------------------------------------------------------------

def lookup(lat: Lattice, keys: np.ndarray, vbatch: Optional[np.ndarray] = None) -> np.ndarray:
    """Vertex index of each key [n, d+1] (with batch ids [n] on a batched
    lattice) in ``lat``, -1 where the key is not a vertex of it."""
    d = lat.d
    cols = ([("b", np.int64)] if lat.vbatch is not None else []) + [(f"c{i}", np.int64) for i in range(d)]
    dt = np.dtype(cols)

    def pack(coords, vb):
        rec = np.empty(coords.shape[0], dtype=dt)
        if lat.vbatch is not None:
            rec["b"] = vb
        for i in range(d):
            rec[f"c{i}"] = coords[:, i]
        return rec

    table = pack(lat.keys, lat.vbatch)                  # canonical order is sorted
    q = pack(np.asarray(keys, dtype=np.int64), vbatch)
    pos = np.searchsorted(table, q)
    out = np.full(q.shape[0], -1, dtype=np.int64)
    hit = pos < lat.V
    hit[hit] = table[pos[hit]] == q[hit]
    out[hit] = pos[hit]
    return out


def coarsen(pos: np.ndarray, sigma, alpha: Optional[float] = None, batch: Optional[np.ndarray] = None) -> Lattice:
    """The coarse lattice of a cloud: its lattice with the positions divided by 2."""
    return build(np.asarray(pos, dtype=F32) / F32(2), sigma, alpha, batch)


def down_neighbors(fine: Lattice, coarse: Lattice) -> np.ndarray:
    """[V_coarse, T]: the fine vertex at 2c' + offset_t for each coarse vertex c', or -1."""
    offs = neighbor_offsets(coarse.d)
    out = np.empty((coarse.V, offs.shape[0]), dtype=np.int64)
    for t, o in enumerate(offs):
        out[:, t] = lookup(fine, 2 * coarse.keys + o, coarse.vbatch)
    return out


def up_neighbors(coarse: Lattice, fine: Lattice) -> np.ndarray:
    """[V_fine, T]: the coarse vertex at (u + offset_t)/2 for each fine vertex u,
    or -1 when that key is fractional or not a coarse vertex."""
    offs = neighbor_offsets(fine.d)
    out = np.full((fine.V, offs.shape[0]), -1, dtype=np.int64)
    for t, o in enumerate(offs):
        q = fine.keys + o
        even = np.all(q % 2 == 0, axis=1)
        if even.any():
            vb = None if fine.vbatch is None else fine.vbatch[even]
            out[even, t] = lookup(coarse, q[even] // 2, vb)
    return out


def downsample(fine: Lattice, coarse: Lattice, values: np.ndarray, weight: np.ndarray,
               bias: Optional[np.ndarray] = None):
    """Strided convolution from the fine lattice's values [V_fine, C_in] onto the
    coarse vertices: y_c' = sum_t x_{fine(2c' + offset_t)} W_t^T (+ bias).
    Returns (y [V_coarse, C_out], scale)."""
    return conv(values, down_neighbors(fine, coarse), weight, bias)


def upsample(coarse: Lattice, fine: Lattice, values: np.ndarray, weight: np.ndarray,
             bias: Optional[np.ndarray] = None):
    """Transposed convolution from the coarse lattice's values [V_coarse, C_in]
    onto the fine vertices: z_u = sum_t x_{coarse((u + offset_t)/2)} W_t^T (+ bias),
    fractional or absent taps contributing nothing.  Returns (z [V_fine, C_out], scale)."""
    return conv(values, up_neighbors(coarse, fine), weight, bias)


def downsample_backward(fine: Lattice, coarse: Lattice, values: np.ndarray, weight: np.ndarray,
                        grad_out: np.ndarray):
    """Gradients of downsample (a linear map of the fine values and of the
    weights): conv_backward over the coarse vertices' table into the fine
    lattice.  values [V_fine, C_in] is the forward input, grad_out
    [V_coarse, C_out].  Returns conv_backward's six arrays (grad_x has the
    fine lattice's V rows)."""
    return conv_backward(values, down_neighbors(fine, coarse), weight, grad_out)


def upsample_backward(coarse: Lattice, fine: Lattice, values: np.ndarray, weight: np.ndarray,
                      grad_out: np.ndarray):
    """Gradients of upsample: conv_backward over the fine vertices' table into
    the coarse lattice (values [V_coarse, C_in], grad_out [V_fine, C_out])."""
    return conv_backward(values, up_neighbors(coarse, fine), weight, grad_out)


# ---------------------------------------------------------------------------
# Distribute and PointNet (Sec. "Proposed Operations": Distribute, Eq.
# distribute; the network figure's PointNet block; Sec. "Performance"
# suggests fusing the two into one operation).
#
# Every (point, simplex vertex) pair p in J_v hands the vertex the point's
# position minus the mean position of all points of J_v, and the point's
# features, concatenated: h_0 = [g_p - mu_v ; f_p].  A PointNet embeds each
# such row: blocks of normalisation, ReLU and a 1x1 (fully connected) layer,
# h_l = W_l relu(a_l * h_{l-1} + s_l) + b_l, where the normalisation enters as
# the per-channel affine (a_l, s_l) that a group normalisation with known
# statistics reduces to.  A max over the rows of each vertex (scatter-max)
# gives its value x_v.
# ---------------------------------------------------------------------------

def local_mean(lat: Lattice, pos: np.ndarray) -> np.ndarray:
    """mu_v = (1/|J_v|) sum_{p in J_v} g_p, float64 [V, d]: the mean position of
    the points whose simplex contains v (every pair counts, whatever its weight)."""
    g = np.asarray(pos, dtype=np.float64)
    m, dp1 = lat.idx.shape
    v = lat.idx.ravel()
    p = np.repeat(np.arange(m), dp1)
    s = np.zeros((lat.V, g.shape[1]))
    np.add.at(s, v, g[p])
    n = np.bincount(v, minlength=lat.V).astype(np.float64)
    return s / n[:, None]


def default_groups(K: int, max_groups: int = 32) -> int:
    """Group count of a group normalisation over K channels: the default of 32
    groups (Sec. "Implementation"), reduced, where K is smaller than 32 or not
    a multiple of it, to the largest divisor of K that is at most 32 (the
    groups must split the channels evenly).  Below 32 channels every channel
    is then its own group."""
    return max(g for g in range(1, min(max_groups, K) + 1) if K % g == 0)


def group_norm(h: np.ndarray, seg: np.ndarray, groups: int, gamma, beta, eps: float = 1e-5):
    """Group normalisation (Wu and He, the method Sec. "Implementation" cites),
    float64, of rows h [N, K] that belong to samples seg [N].

    The K channels are cut into ``groups`` groups of K / groups consecutive
    channels.  Within one sample (here one cloud, the rows of one batch id),
    each group is centred by its mean and divided by sqrt(var + eps), the mean
    and the variance (the biased one, dividing by the count) taken over every
    row of the sample and every channel of the group; then channel c is
    scaled by gamma_c and shifted by beta_c.

    Returns (out [N, K], mean [S, groups], var [S, groups], samples [S]) with
    the samples in ascending order."""
    h = np.asarray(h, dtype=np.float64)
    N, K = h.shape
    assert K % groups == 0, (K, groups)
    gamma = np.asarray(gamma, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    samples = np.unique(seg)
    out = np.empty_like(h)
    means = np.zeros((len(samples), groups))
    varis = np.zeros((len(samples), groups))
    for i, s in enumerate(samples):
        rows = seg == s
        x = h[rows].reshape(-1, groups, K // groups)
        mu = x.mean(axis=(0, 2))
        var = ((x - mu[None, :, None]) ** 2).mean(axis=(0, 2))
        xn = (x - mu[None, :, None]) / np.sqrt(var + eps)[None, :, None]
        out[rows] = xn.reshape(-1, K) * gamma + beta
        means[i], varis[i] = mu, var
    return out, means, varis, samples


def distribute_rows(lat: Lattice, pos: np.ndarray, feat: Optional[np.ndarray]):
    """The distributed rows of Eq. (distribute), float64: one row per pair
    (point p, vertex v of p's simplex), h_0 = [g_p - mu_v ; f_p].

    Returns (h0 [E, d + f_d], v [E], p [E], seg [E], mu [V, d]) where seg is
    the cloud of each row (its vertex's batch id, 0 for an unbatched lattice),
    plus the magnitudes |g_p| + |mu_v|, |f_p| of the row's terms [E, d + f_d]."""
    g = np.asarray(pos, dtype=np.float64)
    m, dp1 = lat.idx.shape
    mu = local_mean(lat, pos)
    v = lat.idx.ravel()
    p = np.repeat(np.arange(m), dp1)
    dg = g[p] - mu[v]                                        # D_G: positions minus the local mean
    sg = np.abs(g[p]) + np.abs(mu[v])
    if feat is not None and np.asarray(feat).shape[1] > 0:
        f = np.asarray(feat, dtype=np.float64)[p]            # D_F: the features as they are
        h = np.concatenate([dg, f], axis=1)
        sc = np.concatenate([sg, np.abs(f)], axis=1)
    else:
        h, sc = dg, sg
    seg = lat.vbatch[v] if lat.vbatch is not None else np.zeros(len(v), dtype=np.int64)
    return h, v, p, seg, mu, sc


def distribute_pointnet(lat: Lattice, pos: np.ndarray, feat: Optional[np.ndarray], layers, groups=None,
                        eps: float = 1e-5):
    """Distribute + PointNet + per-vertex max, float64.

    Each block of the PointNet (the network figure) is a normalisation, a
    ReLU and a fully connected 1x1 layer: h_l = W_l relu(N_l(h_{l-1})) + b_l;
    then x_v is the channel-wise max over the rows of v.

    * ``groups`` given (one group count per block): N_l is the group
      normalisation of ``group_norm`` over all the rows of one cloud (per
      batch id), and ``layers`` holds (gamma, beta, W, b) per block.
    * ``groups`` None: N_l is the fixed per-channel affine a h + s (a
      normalisation whose statistics are already folded in), and ``layers``
      holds (a, s, W, b).

    W is [w_l, K_l]; K_0 = d + f_d.  Returns (out [V, w_L], scale [V, w_L],
    mu [V, d]).  ``scale`` bounds the rounding of a float32 evaluation: per
    row, the magnitudes |g_p| + |mu_v| and |f_p| carried through each block
    (the normalisation as |a| (|h| + |mean|) + |beta| with a = gamma /
    sqrt(var + eps); ReLU is 1-Lipschitz; then |W|, |b|), and the max over
    the vertex's rows."""
    h, v, p, seg, mu, sc = distribute_rows(lat, pos, feat)
    for li, (a, s, W, b) in enumerate(layers):
        a = np.asarray(a, dtype=np.float64)
        s = np.asarray(s, dtype=np.float64)
        W = np.asarray(W, dtype=np.float64)
        b = np.asarray(b, dtype=np.float64)
        if groups is None:
            hn = a * h + s
            scn = np.abs(a) * sc + np.abs(s)
        else:
            G = groups[li]
            hn, means, varis, samples = group_norm(h, seg, G, a, s, eps)
            K = h.shape[1]
            row = np.searchsorted(samples, seg)
            gmean = np.repeat(means, K // G, axis=1)[row]               # [E, K] the group's mean
            ga = a / np.sqrt(np.repeat(varis, K // G, axis=1)[row] + eps)
            scn = np.abs(ga) * (sc + np.abs(gmean)) + np.abs(s)
        h = np.maximum(hn, 0.0) @ W.T + b
        sc = scn @ np.abs(W).T + np.abs(b)
    out = np.full((lat.V, h.shape[1]), -np.inf)
    np.maximum.at(out, v, h)
    scale = np.zeros_like(out)
    np.maximum.at(scale, v, sc)
    return out, scale, mu


def _pointnet_forward_cache(lat: Lattice, pos, feat, layers, groups, eps):
    """The forward of distribute_pointnet keeping what its backward needs,
    float64: per block l the input h, the normalised xhat (h itself for the
    fixed affine), the per-row normalisation factor 1/sqrt(var + eps) (1 for
    the fixed affine), hn, the ReLU output r; the rows' vertices, clouds, and
    the last block's output."""
    h, v, p, seg, mu, _ = distribute_rows(lat, pos, feat)
    blocks = []
    for li, (a, s, W, b) in enumerate(layers):
        a = np.asarray(a, dtype=np.float64)
        s = np.asarray(s, dtype=np.float64)
        W = np.asarray(W, dtype=np.float64)
        b = np.asarray(b, dtype=np.float64)
        K = h.shape[1]
        if groups is None:
            xhat, rstd, G = h, np.ones_like(h), None
        else:
            G = groups[li]
            _, means, varis, samples = group_norm(h, seg, G, a, s, eps)
            row = np.searchsorted(samples, seg)
            mean = np.repeat(means, K // G, axis=1)[row]
            rstd = 1.0 / np.sqrt(np.repeat(varis, K // G, axis=1)[row] + eps)
            xhat = (h - mean) * rstd
        hn = a * xhat + s
        r = np.maximum(hn, 0.0)
        blocks.append(dict(h=h, xhat=xhat, rstd=rstd, hn=hn, r=r, a=a, W=W, G=G))
        h = r @ W.T + b
    return blocks, h, v, seg


def _group_mean(x: np.ndarray, seg: np.ndarray, G: int) -> np.ndarray:
    """Per row, the mean of x over its cloud's rows and its group's channels."""
    N, K = x.shape
    out = np.empty_like(x)
    for s_ in np.unique(seg):
        rows = seg == s_
        m = x[rows].reshape(-1, G, K // G).mean(axis=(0, 2))
        out[rows] = np.repeat(m, K // G)[None, :]
    return out


def pointnet_backward_rows(blocks, seg, dh: np.ndarray):
    """Backward of the PointNet blocks given dL/dh of the last block's rows
    [E, w_L], float64.  Per block, from the last:
      db = sum_rows dh,  dW = dh^T r,  dr = dh W,  dhn = dr [hn > 0];
      normalisation hn = a xhat + s (a = gamma, s = beta with groups):
        da = sum_rows dhn xhat,  ds = sum_rows dhn,
        dh_prev = a dhn (fixed affine), or with group normalisation
        (xhat = (h - mean) rstd over a cloud's rows and a group's channels)
        dh_prev = rstd (g - mean(g) - xhat mean(g xhat)),  g = a dhn,
        the means over the same rows and channels.
    Returns [(da, ds, dW, db)] per block, in block order."""
    out = []
    for blk in reversed(blocks):
        db = dh.sum(axis=0)
        dW = dh.T @ blk["r"]
        dr = dh @ blk["W"]
        dhn = dr * (blk["hn"] > 0)
        da = (dhn * blk["xhat"]).sum(axis=0)
        ds = dhn.sum(axis=0)
        g = blk["a"] * dhn
        if blk["G"] is None:
            dh = g
        else:
            G = blk["G"]
            dh = blk["rstd"] * (g - _group_mean(g, seg, G) - blk["xhat"] * _group_mean(g * blk["xhat"], seg, G))
        out.append((da, ds, dW, db))
    return out[::-1]


def distribute_pointnet_backward(lat: Lattice, pos: np.ndarray, feat: Optional[np.ndarray], layers,
                                 grad_out: np.ndarray, groups=None, eps: float = 1e-5):
    """Gradients of distribute_pointnet with respect to every block's
    parameters (gamma and beta, or a and s; W; b) given grad_out = dL/dx
    [V, w_L], float64.  The max sends grad_out[v, c] to the row of v whose
    channel c is largest (the first such row in row order).  The positions
    and features are the network's raw inputs and get no gradient.
    Returns ([(da, ds, dW, db)] per block, argmax [V, w_L] row indices,
    last-block rows [E, w_L], the rows' vertices [E], the forward cache,
    the rows' clouds)."""
    blocks, h3, v, seg = _pointnet_forward_cache(lat, pos, feat, layers, groups, eps)
    E, w = h3.shape
    g = np.asarray(grad_out, dtype=np.float64)
    order = np.argsort(v, kind="stable")                   # rows grouped by vertex, row order kept
    am = np.full((lat.V, w), -1, dtype=np.int64)
    starts = np.searchsorted(v[order], np.arange(lat.V))
    ends = np.searchsorted(v[order], np.arange(lat.V), side="right")
    for vv in range(lat.V):
        rows = order[starts[vv]:ends[vv]]
        if len(rows):
            am[vv] = rows[np.argmax(h3[rows], axis=0)]     # first maximum in row order
    dh = np.zeros((E, w))
    vv, cc = np.nonzero(am >= 0)
    np.add.at(dh, (am[vv, cc], cc), g[vv, cc])
    return pointnet_backward_rows(blocks, seg, dh), am, h3, v, blocks, seg
