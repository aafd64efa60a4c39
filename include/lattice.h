/*
 * lattice.h -- C ABI of the sparse permutohedral-lattice hot path for MI355X (gfx950).
 *
 * The library implements the three lattice operations of LatticeNet
 * (Rosu et al., arXiv 2108.03917) in the order the paper states them:
 * splat a point cloud onto the occupied vertices of a d-dimensional
 * permutohedral lattice, convolve the vertex values over the 1-hop ring,
 * and slice the result back onto the points.
 *
 *   Sec. "Notation": a cloud is P = (G, F) with positions G in R^{m x d} and
 *     features F in R^{m x f_d}; a lattice vertex is (c_v, x_v) with integer
 *     coordinates c_v in Z^{d+1} and values x_v in R^{v_d}; I_p is the set of
 *     d+1 vertices of the simplex containing point p.
 *   Sec. "Permutohedral Lattice": the lattice is (d+1)Z^{d+1} projected along
 *     the all-ones vector onto the hyperplane H_d, so every key sums to zero;
 *     the enclosing simplex comes from a rounding algorithm; the 2(d+1)
 *     neighbours of a vertex sit at +-[-1,..,-1,d,-1,..,-1]; vertices are kept
 *     sparsely in a hash map keyed by c_v.
 *   Sec. "Method": positions are scaled as G / sigma, sigma in R^d.
 *   Sec. "Common Operations on Permutohedral Lattice": splatting (barycentric
 *     weights onto the d+1 simplex vertices, summed per vertex), convolving
 *     over the 2(d+1)+1 vertices of the 1-hop ring (an unallocated neighbour
 *     contributes zero), slicing (the reverse of splatting with the same
 *     barycentric weights); Eq. (splat) and Eq. (slice).
 *
 * Conventions fixed by this library where the paper leaves them open
 * (the CPU test oracle adopts the same ones):
 *   - elevation x = alpha * E * (g / sigma), E the orthonormal basis of H_d
 *     whose j-th column is (1,..,1,-j,0,..,0)/sqrt(j(j+1)) (j ones);
 *     alpha <= 0 selects (d+1) * sqrt(2/3);
 *   - round half to even when rounding to the remainder-0 point; rank ties go
 *     to the lower coordinate index;
 *   - all d+1 vertices of every point's simplex are allocated;
 *   - 1-ring tap order: tap 0 = the vertex, tap 1+j = c + n_j,
 *     tap d+2+j = c - n_j (j = 0..d), n_j = (d+1) e_j - 1;
 *   - convolution weights are laid out [C_out][T][C_in], T = 2(d+1)+1.
 *
 * Memory.  Every pointer marked "dev" is device memory on the device that was
 * current at lattice_create; "host" pointers are host memory.  The caller owns
 * every buffer it passes in; the lattice owns its internal buffers (hash
 * table, packed vertex keys, per-point simplex records, neighbour table,
 * counters).  All work is enqueued on the stream given at creation; no call
 * except lattice_num_vertices, lattice_get_status and lattice_destroy
 * synchronises with the host.  The number of occupied vertices V stays on the
 * device between splat, conv and slice: kernels read it there.
 *
 * Errors.  Functions return a lattice_status.  Argument and call-order errors
 * are detected synchronously and nothing is enqueued.  Failures that only the
 * device can see (hash table full, key coordinate out of range, batch id out
 * of range) set a device status word; lattice_num_vertices and
 * lattice_get_status report it.  It is cleared by the next lattice_splat.
 * lattice_last_error returns a message for the last failure on a lattice.
 *
 * Threading.  A lattice is not thread safe; calls on one lattice must be
 * serialised by the caller.  Distinct lattices are independent.
 */
#ifndef LATTICE_H
#define LATTICE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lattice lattice;

typedef enum {
    LATTICE_OK = 0,
    LATTICE_E_ARG = 1,      /* bad argument (null pointer, d, C, m out of range, ...) */
    LATTICE_E_STATE = 2,    /* call out of order, e.g. conv or slice before splat      */
    LATTICE_E_RANGE = 3,    /* device: a key coordinate or batch id does not fit 16 bits */
    LATTICE_E_CAPACITY = 4, /* device: the hash table is full                          */
    LATTICE_E_NOMEM = 5,    /* device or host allocation failed                        */
    LATTICE_E_HIP = 6       /* a HIP runtime call failed (no device, launch failure)   */
} lattice_status;

typedef enum {
    LATTICE_F32 = 0,  /* fp32 inputs and weights, fp32 accumulation (fp32 MFMA or FMA) */
    LATTICE_BF16 = 1  /* inputs rounded to bf16 (nearest even), bf16 weights, fp32 accumulation on MFMA */
} lattice_dtype;

/* Largest lattice dimension, and the tap count of the 1-ring for dimension d. */
#define LATTICE_MAX_D 4
#define LATTICE_TAPS(d) (2 * ((d) + 1) + 1)

/*
 * lattice_create -- allocate a lattice for clouds of up to max_points points.
 *
 * Sec. "Permutohedral Lattice" and Sec. "Method" (G / sigma).
 *   d              lattice dimension, 1..4 (the paper's clouds use d = 3; the
 *                  space-time lattice uses d = 4).
 *   sigma          host [d] fp32, per-axis lattice scale, each > 0.
 *   alpha          elevation scale; <= 0 selects (d+1) * sqrt(2/3).
 *   max_points     upper bound on m for every later splat, 1 .. 2^28 (the
 *                  pair lists hold a point index in 28 bits).
 *   hash_capacity  number of hash slots; 0 selects the next power of two
 *                  >= 1.5 (d+1) max_points: it can never fill up, and at
 *                  most two thirds of its slots are ever taken, which keeps
 *                  the probe chains of failed lookups short.  A non-zero
 *                  value is rounded up to a power of two; a table that fills
 *                  makes splat report LATTICE_E_CAPACITY.
 *   stream         hipStream_t every call of this lattice is enqueued on
 *                  (NULL = the null stream).
 *   out            host: receives the new lattice.
 * Returns LATTICE_E_ARG, LATTICE_E_NOMEM or LATTICE_E_HIP on failure, in
 * which case *out is NULL.
 */
lattice_status lattice_create(int d, const float *sigma, double alpha, int64_t max_points,
                              int64_t hash_capacity, void *stream, lattice **out);

/* Release every buffer of L (after synchronising its stream).  NULL is a no-op. */
void lattice_destroy(lattice *L);

/*
 * lattice_max_vertices -- the row count callers allocate for per-vertex
 * buffers (values, conv output): min((d+1) * m, hash capacity).  The actual V
 * of a splat is never larger.  Returns -1 for a NULL lattice or m < 0.
 */
int64_t lattice_max_vertices(const lattice *L, int64_t m);

/*
 * lattice_splat -- build the sparse lattice of a cloud and splat its features.
 *
 * Sec. "Permutohedral Lattice" (enclosing simplex, hash map of keys) and
 * Eq. (splat):  x_v = sum_{p in J_v} b_pv f_p.  Also w_v = sum_{p in J_v} b_pv.
 *   pos          dev [m][d] fp32, row-major point positions (unscaled).
 *   batch        dev [m] int32 batch id per point in [0, 65535], or NULL.
 *                Each id is an independent lattice sharing one table;
 *                neighbours never cross ids.  Must be NULL when d = 4.
 *   m            number of points, 0 <= m <= max_points (m = 0 gives V = 0).
 *   feat         dev [m][C] fp32 row-major features, or NULL when C = 0 (then
 *                only the lattice is built).
 *   C            feature channels, 0..4096.
 *   normalize    0: values hold the raw sum x_v;  1: values hold x_v / w_v
 *                (0 where w_v = 0).
 *   values       dev [>= lattice_max_vertices(L, m)][C] output, rows 0..V-1
 *                written (may be NULL when C = 0 or m = 0); sums are fp32.
 *   values_dtype storage of `values`: LATTICE_F32, or LATTICE_BF16 (each sum
 *                rounded to nearest even; for a following bf16 conv this is
 *                the same rounding the conv would apply to fp32 rows).
 *   weight       dev [>= lattice_max_vertices(L, m)] fp32 output w_v, or NULL.
 * Resets the lattice: the previous vertex set, records and neighbour table
 * are discarded.  Vertex order follows, in point order, the pair whose
 * insertion created each vertex (the winner of a concurrent claim): it is not
 * deterministic.  Device-side failures are reported by lattice_num_vertices.
 */
lattice_status lattice_splat(lattice *L, const float *pos, const int32_t *batch, int64_t m,
                             const float *feat, int C, int normalize, void *values,
                             lattice_dtype values_dtype, float *weight);

/*
 * lattice_build_neighbors -- build the 1-hop-ring neighbour table of the
 * last splat's vertices now (otherwise the first lattice_conv builds it).
 *
 * Sec. "Permutohedral Lattice": the 2(d+1) neighbours of vertex c are
 * c +- n_j, n_j = (d+1) e_j - 1; Sec. "Common Operations": the convolution
 * spans the vertex and these neighbours (T = 2(d+1)+1 taps).  One hash
 * lookup per tap; a neighbour that is not allocated gets index -1.
 * Returns LATTICE_E_STATE before the first splat; a no-op when the table of
 * the current lattice exists.
 */
lattice_status lattice_build_neighbors(lattice *L);

/*
 * lattice_conv -- 1-hop-ring lattice convolution over the occupied vertices.
 *
 * Sec. "Common Operations on Permutohedral Lattice" (Convolving) and the
 * caption of its figure (an unallocated neighbour contributes zero):
 *   y_v[o] = bias[o] + sum_{t < T} sum_{i < C_in} x_{nbr(v,t)}[i] * W[o][t][i].
 *   in         dev [V][C_in] vertex values (rows of the last splat's vertices).
 *   in_dtype   storage of `in`: LATTICE_F32 or LATTICE_BF16.
 *   C_in       input channels, 1..1024.
 *   w          dev weights [C_out][T][C_in]: fp32 for compute LATTICE_F32,
 *              bf16 (raw 16-bit patterns) for LATTICE_BF16 (see
 *              lattice_weights_to_bf16).
 *   C_out      output channels, 1..1024.
 *   dt         compute type.  LATTICE_F32: fp32 products and sums.
 *              LATTICE_BF16: inputs rounded to bf16 (nearest even; a no-op
 *              for bf16-stored input), exact products, fp32 sums.
 *   bias       dev [C_out] fp32 or NULL.
 *   out        dev [>= V][C_out] output; must not overlap `in`.
 *   out_dtype  storage of `out`: LATTICE_F32, or LATTICE_BF16 (fp32 result
 *              rounded to nearest even).
 * The first conv after a splat also builds the neighbour table (2(d+1) hash
 * lookups per vertex).  Returns LATTICE_E_STATE before the first splat.
 */
lattice_status lattice_conv(lattice *L, const void *in, lattice_dtype in_dtype, int C_in, const void *w,
                            int C_out, lattice_dtype dt, const float *bias, void *out,
                            lattice_dtype out_dtype);

/*
 * lattice_set_conv_path -- choose the kernel family of later lattice_conv
 * calls (the result is the same to the stated tolerances; this is for
 * testing and benchmarking each kernel).
 *   LATTICE_CONV_AUTO    the fastest kernel built for the shape (default)
 *   LATTICE_CONV_TILED   the LDS-tiled kernel (weights and gathered rows
 *                        staged per K chunk), else the any-shape one
 *   LATTICE_CONV_WS      weight slice resident in LDS, rows gathered straight
 *                        into registers, where built for the shape; else TILED
 *   LATTICE_CONV_RS      weights resident in registers, rows gathered into
 *                        LDS by direct loads, where built for the shape
 *                        (bf16 rows and weights: 64 -> 64, 64 -> 128,
 *                        128 -> 128 with 9 taps, 64 -> 64 and 64 -> 128 with
 *                        11; fp32: 64 -> 64 with 9 taps); else as AUTO
 * Returns LATTICE_E_ARG for another value.
 */
enum { LATTICE_CONV_AUTO = 0, LATTICE_CONV_TILED = 1, LATTICE_CONV_WS = 2, LATTICE_CONV_RS = 3 };
lattice_status lattice_set_conv_path(lattice *L, int path);

/*
 * lattice_slice -- interpolate vertex values back onto the points.
 *
 * Eq. (slice):  f_p = sum_{v in I_p} b_pv x_v, with the barycentric weights
 * of the last splat; fp32 products and sums.
 *   values        dev [V][C] vertex values.
 *   values_dtype  storage of `values`: LATTICE_F32 or LATTICE_BF16.
 *   C             channels, 1..4096.
 *   out           dev [m][C] fp32 (m of the last splat).
 * Returns LATTICE_E_STATE before the first splat.
 */
lattice_status lattice_slice(lattice *L, const void *values, lattice_dtype values_dtype, int C, float *out);

/*
 * lattice_deform_slice -- slice with learned offsets on the barycentric
 * weights (DeformSlice), optionally fused with a linear classifier.
 *
 * Sec. "Proposed Operations" (DeformSlicing), Eq. (deformSlice) and the
 * network figure's DeformSlice block; Sec. "Implementation" fuses the final
 * classifier so that the per-point features are never written.  For point p
 * of the last splat, with simplex vertices v_k and weights b_k (k <= d):
 *   q_k   = b_k x_{v_k}                     (Gather)
 *   mx    = max_k q_k, per channel          (MaxPool over all d+1 vertices)
 *   db_k  = tanh(b_delta + (q_k - mx) . w_delta)
 *   f_p   = sum_k (b_k + db_k) x_{v_k}
 *   out_p = f_p, or f_p W_cls^T + b_cls when w_cls is given.
 * fp32 products and sums; tanh in fp32.
 *   values        dev [V][C] vertex values (the last lattice conv's output).
 *   values_dtype  storage of `values`: LATTICE_F32 or LATTICE_BF16.
 *   C             channels, 1..1024; above 256 C must be a multiple of 4
 *                 and values, w_delta and (w_cls or out) aligned to 16
 *                 bytes (8 for bf16 values) -- true of every device
 *                 allocation and of row offsets that are multiples of 4.
 *   w_delta       dev [C] fp32 weights of the offsets' linear layer.
 *   b_delta       its bias (a host value).
 *   w_cls         dev [n_cls][C] fp32 classifier weights, or NULL for none.
 *   b_cls         dev [n_cls] fp32 classifier bias, or NULL (zero).
 *   n_cls         classes, 1..256 (ignored without w_cls).
 *   out           dev fp32 [m][n_cls] logits with w_cls, else [m][C] f_p;
 *                 must not overlap `values`.
 *   delta         dev fp32 [m][d+1] receives db (the learned offsets), or
 *                 NULL.
 * Caller owns every buffer.  Returns LATTICE_E_STATE before the first splat,
 * LATTICE_E_ARG for a size or pointer outside the above.
 */
lattice_status lattice_deform_slice(lattice *L, const void *values, lattice_dtype values_dtype, int C,
                                    const float *w_delta, float b_delta, const float *w_cls, const float *b_cls,
                                    int n_cls, float *out, float *delta);

/*
 * Backward passes.  Sec. "Implementation": the network is trained end to
 * end, so every lattice operation needs the gradient of a loss L with
 * respect to its inputs.  Each forward is linear in what is differentiated,
 * so each gradient is the transposed map of the forward with the same
 * lattice (the last splat's simplex records and neighbour table).  All
 * sums are fp32; the caller owns every buffer; rows 0..V-1 (or 0..m-1) are
 * written.  Each returns LATTICE_E_STATE before the first splat and
 * LATTICE_E_ARG for a bad size or a missing pointer.
 */

/*
 * lattice_slice_backward -- gradient of Eq. (slice) with respect to the
 * vertex values: dL/dy_v = sum over the points p with v in I_p of
 * b_pv dL/df_p, i.e. Eq. (splat) applied to the point gradients.
 *   grad_out      dev [m][C] fp32 dL/df (m of the last splat).
 *   C             channels, 1..4096.
 *   grad_values   dev [>= lattice_max_vertices][C] output dL/dy, rows 0..V-1
 *                 written; must not overlap grad_out.
 *   grad_dtype    storage of grad_values: LATTICE_F32, or LATTICE_BF16 (each
 *                 fp32 sum rounded to nearest even).
 * The first call with more channels than any splat before it grows the
 * lattice's gather scratch (a device allocation).
 */
lattice_status lattice_slice_backward(lattice *L, const float *grad_out, int C, void *grad_values,
                                      lattice_dtype grad_dtype);

/*
 * lattice_splat_backward -- gradient of Eq. (splat) with respect to the
 * point features: dL/df_p = sum_k b_pk dL/dx_{v_k}, i.e. Eq. (slice)
 * applied to the vertex gradients.  For the normalised splat (values
 * x_v / w_v) each vertex gradient is divided by w_v first, and a vertex with
 * w_v = 0 (whose value is the constant 0) passes no gradient.
 *   grad_values   dev [V][C] dL/dx, stored as gv_dtype (LATTICE_F32 or LATTICE_BF16).
 *   C             channels, 1..4096.
 *   normalize     0: the raw splat;  1: the normalised splat.
 *   weight        dev [V] fp32, the w_v the splat returned; required when
 *                 normalize = 1, ignored otherwise.
 *   grad_feat     dev [m][C] fp32 output dL/df.
 */
lattice_status lattice_splat_backward(lattice *L, const void *grad_values, lattice_dtype gv_dtype, int C,
                                      int normalize, const float *weight, float *grad_feat);

/*
 * lattice_deform_slice_backward -- gradients of lattice_deform_slice (Eq.
 * deformSlice and the fused classifier) given g = dL/dout, through the
 * forward's steps in reverse:
 *   gf_p     = g_p W_cls (with the classifier) or g_p
 *   dW_cls   = sum_p g_p^T f_p,      db_cls = sum_p g_p
 *   darg_pk  = (gf_p . x_k)(1 - db_pk^2),  S_p = sum_k darg_pk
 *   dw_delta = sum_pk darg_pk (q_pk - mx_p),  db_delta = sum_pk darg_pk
 *   dx_pk    = (b_pk + db_pk) gf_p + b_pk w_delta (darg_pk - [k = k*] S_p),
 *   dX_v     = sum of dx_pk over the pairs with v_pk = v,
 * k* per channel the vertex whose product b x wins the max (the first of
 * equal maxima of the fp32 products, as the forward computes them).  fp32
 * throughout; the vertex gradient is pulled over the splat's pair lists (no
 * atomics) and the weight gradients are summed in a fixed order.
 *   values, values_dtype, C, w_delta, b_delta, w_cls, n_cls   as in the
 *                 forward (C 1..1024; b_cls does not enter the gradients).
 *   grad_out      dev fp32 [m][n_cls] with w_cls, else [m][C].  With an
 *                 empty cloud (m = 0) values and grad_out may be NULL, and
 *                 the weight gradients are zero.
 *   grad_values   dev [>= V][C] dX stored as grad_dtype, or NULL; must not
 *                 overlap values or grad_out.
 *   grad_w_delta  dev fp32 [C], or NULL.     grad_b_delta  dev fp32 [1], or NULL.
 *   grad_w_cls    dev fp32 [n_cls][C], or NULL (needs w_cls).
 *   grad_b_cls    dev fp32 [n_cls], or NULL (needs w_cls).
 * At least one output.  Per-point records (5C + 12(d+1) bytes per point,
 * 4C more with the classifier) are kept in the lattice's scratch, grown on
 * demand.
 */
lattice_status lattice_deform_slice_backward(lattice *L, const void *values, lattice_dtype values_dtype, int C,
                                             const float *w_delta, float b_delta, const float *w_cls, int n_cls,
                                             const float *grad_out, void *grad_values, lattice_dtype grad_dtype,
                                             float *grad_w_delta, float *grad_b_delta, float *grad_w_cls,
                                             float *grad_b_cls);

/*
 * lattice_conv_backward -- gradients of lattice_conv (Sec. "Common
 * Operations", Convolving):
 *   dL/dx_u[i]    = sum over (v, t) with nbr(v,t) = u of sum_o g_v[o] W[o][t][i]
 *   dL/dW[o][t][i] = sum_v g_v[o] x_{nbr(v,t)}[i]   (an absent tap reads zero)
 *   dL/dbias[o]   = sum_v g_v[o]
 * with g = dL/dy.  The input gradient is computed as a forward convolution
 * of g with the flipped, transposed weights (the 1-ring is symmetric: tap
 * 1+j of v is u exactly when tap d+2+j of u is v), on the same kernels as
 * lattice_conv; the weight gradient is a product reduced over the vertices
 * in fixed chunks added in a fixed order (run to run identical).
 *   grad_out       dev [V][C_out] g, stored as g_dtype.
 *   C_out, C_in    channels of the forward conv, 1..1024 each.
 *   w              dev [C_out][T][C_in] forward weights (fp32 for dt =
 *                  LATTICE_F32, bf16 for LATTICE_BF16); needed for grad_in.
 *   dt             compute type as in lattice_conv: LATTICE_BF16 rounds g
 *                  and x to bf16 before the products (exact products, fp32 sums).
 *   in             dev [V][C_in] the forward input x, stored as in_dtype;
 *                  needed for grad_w.
 *   grad_in        dev [>= V][C_in] output dL/dx stored as grad_in_dtype, or NULL.
 *   grad_w         dev [C_out][T][C_in] fp32 output dL/dW, or NULL.
 *   grad_bias      dev [C_out] fp32 output dL/dbias, or NULL.
 * The first call with a larger shape grows the lattice's backward scratch
 * (flipped weights; one partial weight gradient per vertex chunk).
 */
lattice_status lattice_conv_backward(lattice *L, const void *grad_out, lattice_dtype g_dtype, int C_out,
                                     const void *w, int C_in, lattice_dtype dt, const void *in,
                                     lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                     float *grad_w, float *grad_bias);

/*
 * lattice_conv_backward_noalloc -- lattice_conv_backward for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * or training loops, and harnesses that forbid hipMalloc.  Same arguments,
 * same kernels and the same results; it calls no hipMalloc, hipFree or other
 * allocating routine (and records no stage timing, whose events would be
 * created on first use).  Its two scratch buffers (the flipped, transposed
 * weights for grad_in, and one partial weight and bias gradient per vertex
 * chunk for grad_w / grad_bias) live in a fixed workspace of
 * LATTICE_NOALLOC_WORKSPACE_BYTES that the library holds on each GPU it runs
 * on until the process ends, instead of the lattice's scratch.
 *   Limit: C_out T C_in (2 or 4 bytes, padded to 256) for grad_in plus
 *   chunks (C_out T C_in + C_out) 4 bytes for grad_w / grad_bias must fit;
 *   every shape up to 128 -> 128 channels with 11 taps does.  A larger one
 *   returns LATTICE_E_ARG before anything is enqueued.
 *   Every call on one GPU shares that GPU's workspace and leaves its
 *   contents behind: calls that overlap on one GPU (other streams, other
 *   threads, other lattices) race and must be serialised by the caller.
 * Returns LATTICE_E_HIP if the workspace of the lattice's device could not be
 * resolved when the lattice was created.
 */
#define LATTICE_NOALLOC_WORKSPACE_BYTES (24 * 1024 * 1024)
lattice_status lattice_conv_backward_noalloc(lattice *L, const void *grad_out, lattice_dtype g_dtype, int C_out,
                                             const void *w, int C_in, lattice_dtype dt, const void *in,
                                             lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                             float *grad_w, float *grad_bias);

/*
 * Downsampling and upsampling between two lattices of one cloud (Sec.
 * "Proposed Operations": Downsampling, Upsampling, and the Coarsen figure).
 * The coarse lattice is the cloud's lattice at twice the scale (the positions
 * divided by 2): create it with sigma doubled and splat the same positions
 * (C = 0 builds only the lattice).  Both lattices must have been splatted,
 * have the same d, the same stream, the same alpha, both or neither be
 * batched, and the coarse sigma must be exactly twice the fine one on every
 * axis (LATTICE_E_ARG otherwise: this also catches the two lattices passed
 * in the wrong order).
 *
 * lattice_downsample -- strided convolution onto the coarse vertices: coarse
 * vertex c' is embedded in the fine lattice as 2c' and convolves over the
 * fine vertices 2c' + offset_t, offset_t the 1-ring offsets in the tap order
 * of lattice_conv (an unallocated vertex contributes zero):
 *   y_c'[o] = bias[o] + sum_t sum_i x_{fine(2c' + offset_t)}[i] W[o][t][i].
 *   fine, coarse  the two lattices; out has the coarse lattice's V rows.
 *   in            dev [V_fine][C_in] fine vertex values, stored as in_dtype.
 *   other arguments as in lattice_conv (weights [C_out][T][C_in], compute
 *   type dt, optional bias, out dev [>= V_coarse][C_out] stored as out_dtype).
 *
 * lattice_upsample -- transposed convolution onto the fine vertices: fine
 * vertex u is embedded in the coarse lattice as u/2 and convolves over the
 * coarse vertices (u + offset_t)/2; a tap whose key has a fractional
 * coordinate (it falls inside a coarse simplex) or is not allocated
 * contributes zero:
 *   z_u[o] = bias[o] + sum_t sum_i x_{coarse((u + offset_t)/2)}[i] W[o][t][i].
 *   coarse, fine  the two lattices; out has the fine lattice's V rows.
 *   in            dev [V_coarse][C_in] coarse vertex values.
 * With W'[i][s][o] = W[o][flip(s)][i] (flip exchanging +n_j and -n_j),
 * upsampling with W' is the adjoint of downsampling with W.
 *
 * Each builds (on its first call after either lattice's splat) a table of
 * T lookups per output vertex, held by the output lattice, then runs the
 * lattice_conv kernels over it.  Returns LATTICE_E_STATE if a lattice has not
 * been splatted, LATTICE_E_ARG for mismatched lattices or bad arguments.
 */
lattice_status lattice_downsample(lattice *fine, lattice *coarse, const void *in, lattice_dtype in_dtype, int C_in,
                                  const void *w, int C_out, lattice_dtype dt, const float *bias, void *out,
                                  lattice_dtype out_dtype);
lattice_status lattice_upsample(lattice *coarse, lattice *fine, const void *in, lattice_dtype in_dtype, int C_in,
                                const void *w, int C_out, lattice_dtype dt, const float *bias, void *out,
                                lattice_dtype out_dtype);

/*
 * lattice_downsample_backward, lattice_upsample_backward -- gradients of the
 * two resamplings above with respect to their input, weights and bias, given
 * grad_out on the output lattice's vertices (the paper trains every lattice
 * operator end to end, Sec. "Implementation"; these are the adjoints of the
 * operations defined in Sec. "Proposed Operations").
 *   grad_in[u][i] = sum over (v, t) with table(v, t) = u of
 *                   sum_o grad_out[v][o] W[o][t][i]
 *   grad_w[o][t][i] = sum_v grad_out[v][o] in[table(v, t)][i]
 *   grad_bias[o]    = sum_v grad_out[v][o]
 * where table is the forward's cross table (v runs over the output lattice's
 * vertices, u over the input lattice's).  The input gradient is computed as
 * the resampling in the other direction with W'[i][s][o] = W[o][flip(s)][i]
 * (the adjoint stated above), the weight gradient by the conv weight-gradient
 * kernels over the forward table, summed in a fixed order.
 *   fine, coarse / coarse, fine   as in the forward call.
 *   grad_out   dev [V_out][C_out], stored as g_dtype.
 *   w          dev forward weights [C_out][T][C_in] (fp32 or bf16 by dt); needed
 *              for grad_in.
 *   in         dev forward input [V_in][C_in] stored as in_dtype; needed for
 *              grad_w and grad_bias.
 *   grad_in    dev [V_in][C_in] stored as grad_in_dtype, or NULL.
 *   grad_w     dev [C_out][T][C_in] fp32, or NULL.
 *   grad_bias  dev [C_out] fp32, or NULL.
 *   dt         as in lattice_conv (LATTICE_BF16 rounds the operands to bf16).
 * At least one of grad_in, grad_w, grad_bias.  The flipped weights are kept
 * by the input lattice and the weight-gradient partials by the output
 * lattice (grown on demand).  Returns as the forward calls, and
 * LATTICE_E_ARG when grad_in overlaps grad_out or in.
 */
lattice_status lattice_downsample_backward(lattice *fine, lattice *coarse, const void *grad_out,
                                           lattice_dtype g_dtype, int C_out, const void *w, int C_in,
                                           lattice_dtype dt, const void *in, lattice_dtype in_dtype, void *grad_in,
                                           lattice_dtype grad_in_dtype, float *grad_w, float *grad_bias);
lattice_status lattice_upsample_backward(lattice *coarse, lattice *fine, const void *grad_out, lattice_dtype g_dtype,
                                         int C_out, const void *w, int C_in, lattice_dtype dt, const void *in,
                                         lattice_dtype in_dtype, void *grad_in, lattice_dtype grad_in_dtype,
                                         float *grad_w, float *grad_bias);

/*
 * lattice_distribute_pointnet -- Distribute + PointNet + per-vertex max, fused
 * into one operation so that the distributed rows are never stored.
 *
 * Sec. "Proposed Operations" (Distribute, Eq. distribute), the PointNet block
 * of the network figure, Sec. "Implementation" (every convolution is
 * pre-activated by a group normalisation and a ReLU; 32 groups by default),
 * and Sec. "Performance" (fusing the two).  Every pair (point p, vertex v of
 * p's simplex) of the last splat is one row
 *   h_0 = [g_p - mu_v ; f_p],  mu_v = mean of g_q over the points q of J_v
 *   (every pair counts, whatever its barycentric weight);
 * three blocks of normalisation, ReLU and a fully connected (1x1) layer
 *   h_l = W_l relu(N_l(h_{l-1})) + b_l,  widths 16, 32, 64;
 * and x_v = max over the rows of v of h_3, per channel.
 *   groups given: N_l is a group normalisation with groups[l-1] groups of
 *                 consecutive channels.  Per cloud (each batch id of a
 *                 batched lattice is its own cloud) and group, the mean and
 *                 the (biased) variance are taken over all the cloud's rows
 *                 and the group's channels; then per channel
 *                 gamma_c (h - mean) / sqrt(var + eps) + beta_c.  Computed on
 *                 the device in three statistics passes (fp64 sums) before
 *                 the final pass.
 *   groups NULL:  N_l is the per-channel affine a_l h + s_l given by the
 *                 caller (a normalisation whose statistics are known).
 * fp32 products and sums; mu_v summed in fp64.
 *   pos       dev [m][d] fp32, the positions the last splat was given.
 *   feat      dev [m][f_d] fp32 point features, or NULL when f_d = 0.
 *   f_d       feature channels, 0 <= f_d <= 16 - d.
 *   params    dev fp32, per block l = 1, 2, 3 in order: the normalisation's
 *             per-channel vectors (gamma [K_l] then beta [K_l] with groups;
 *             a [K_l] then s [K_l] without), W [w_l][K_l] (row-major), b
 *             [w_l]; K_1 = d + f_d, K_2 = 16, K_3 = 32, w = 16, 32, 64.
 *   n_blocks  3;  widths  host [3], must be {16, 32, 64} (the widths the
 *             fused kernel is built for).
 *   groups    host [3] group counts, each >= 1 and dividing its block's K_l,
 *             or NULL (see above).  The paper's default of 32 groups is
 *             min(32, K) groups for these widths: {d + f_d, 16, 32}.
 *   eps       added to each variance (finite, >= 0; 1e-5 is the usual
 *             value); unused without groups.
 *   out       dev [>= V][64] output x_v (rows 0..V-1 written), in out_dtype:
 *             LATTICE_F32, or LATTICE_BF16 (the fp32 max rounded to nearest
 *             even once: the storage a bf16 conv that reads the rows takes).
 *   mean      dev [>= V][d] fp32 output mu_v, or NULL.
 * Per-cloud statistics cover batch ids 0..63: on a batched lattice with a
 * larger batch id the call sets a device status that lattice_num_vertices
 * and lattice_get_status report as LATTICE_E_RANGE (the rows of those
 * clouds are then not normalised correctly).
 * The first call allocates the lattice's scratch for it (an entry-to-vertex
 * map, fp64 position sums, running-max keys, and 1 MiB of statistics).
 * Returns LATTICE_E_STATE before the first splat, LATTICE_E_ARG for anything
 * outside the above.
 */
lattice_status lattice_distribute_pointnet(lattice *L, const float *pos, const float *feat, int f_d,
                                           const float *params, int n_blocks, const int *widths, const int *groups,
                                           float eps, void *out, lattice_dtype out_dtype, float *mean);

/*
 * lattice_distribute_pointnet_backward -- gradients of
 * lattice_distribute_pointnet with respect to every block's parameters, given
 * grad_out = dL/dx (the network trains end to end, Sec. "Implementation").
 * The max sends grad_out[v][c] to the row of v whose last-block output c is
 * largest (the first such row of v's pair list); then, from the last block:
 *   db = sum_rows dh,  dW = dh^T r,  dr = dh W,  dhn = dr [hn > 0],
 *   d(gamma or a) = sum_rows dhn xhat,  d(beta or s) = sum_rows dhn,
 *   with group normalisation (xhat = (h - mean) rstd per cloud and group)
 *   dh_prev = rstd (gn - mean(gn) - xhat mean(gn xhat)),  gn = gamma dhn,
 *   the means over the cloud's rows and the group's channels; with the
 *   fixed affine dh_prev = a dhn.
 * The positions and features are the network's raw inputs and get no
 * gradient.  The call first runs the forward (its statistics and affines),
 * then recomputes each row's activations in fp32.  Sums are fp32 per
 * wavefront, the partial sums added in a fixed order in fp64: two calls on
 * the same inputs give identical bits.
 *   pos, feat, f_d, params, n_blocks, widths, groups, eps   as in the forward.
 *   grad_out     dev fp32 [>= V][64] dL/dx.
 *   grad_params  dev fp32 output in the layout of params (per block:
 *                d(gamma or a) [K], d(beta or s) [K], dW [w][K], db [w]);
 *                must not overlap params.
 * The first call grows the lattice's scratch for it (a record of 512 bytes
 * per pair and the partial sums).  Returns as the forward, and
 * LATTICE_E_ARG for a missing grad_out or grad_params.
 */
lattice_status lattice_distribute_pointnet_backward(lattice *L, const float *pos, const float *feat, int f_d,
                                                    const float *params, int n_blocks, const int *widths,
                                                    const int *groups, float eps, const float *grad_out,
                                                    float *grad_params);

/*
 * lattice_weights_to_bf16 -- round n fp32 values to bf16 (nearest, ties to
 * even) on the lattice's stream: the weight format LATTICE_BF16 convs take.
 *   src  dev [n] fp32;  dst  dev [n] uint16 (bf16 bit patterns).
 */
lattice_status lattice_weights_to_bf16(lattice *L, const float *src, int64_t n, uint16_t *dst);

/*
 * lattice_num_vertices -- synchronise the stream and return V of the last
 * splat in *V.  Returns the device status (LATTICE_E_CAPACITY,
 * LATTICE_E_RANGE) if the splat (or a distribute with group normalisation
 * on more clouds than it keeps statistics for) failed on the device,
 * LATTICE_E_STATE before the first splat.
 */
lattice_status lattice_num_vertices(lattice *L, int64_t *V);

/* lattice_get_status -- synchronise and return the device status of the last splat. */
lattice_status lattice_get_status(lattice *L);

/*
 * Introspection of the sparse lattice (for tests and downstream operators).
 * Outputs are dev buffers with at least V rows; vertex order is the order in
 * which the hash table created the vertices and is not deterministic.
 *   lattice_get_keys      keys dev [V][d+1] int32 (sum to zero per row);
 *                         batch dev [V] int32 or NULL.
 *   lattice_get_neighbors nbr dev [V][T] int32, -1 where a neighbour is not
 *                         allocated (builds the table if needed).
 *   lattice_get_point_simplex  idx dev [m][d+1] int32 vertex index of the
 *                         simplex vertex with remainder k (column k); bary dev
 *                         [m][d+1] fp32 its barycentric weight.  Either may be NULL.
 */
lattice_status lattice_get_keys(lattice *L, int32_t *keys, int32_t *batch);
lattice_status lattice_get_neighbors(lattice *L, int32_t *nbr);
lattice_status lattice_get_point_simplex(lattice *L, int32_t *idx, float *bary);

/*
 * Stage timing.  With lattice_set_timing(L, 1) the library records a pair of
 * hipEvents on its stream around every stage it launches (splat, neighbours,
 * conv, slice, deform slice); the slice and the deform slice, one kernel
 * each, have their kernel's launch record the pair at the kernel's start and
 * end (the kernel's own duration, without the gap before it).  It
 * accumulates their elapsed times; lattice_get_timing
 * synchronises and returns, per stage, the summed milliseconds and the number
 * of launches since the last reset (arrays of LATTICE_NUM_STAGES).
 * lattice_set_timing(L, 0) stops recording; (L, 2) resets the sums.
 */
#define LATTICE_NUM_STAGES 15
enum {
    LATTICE_STAGE_SPLAT = 0,
    LATTICE_STAGE_NEIGHBORS = 1,
    LATTICE_STAGE_CONV = 2,
    LATTICE_STAGE_SLICE = 3,
    LATTICE_STAGE_DEFORM = 4,
    LATTICE_STAGE_SLICE_BACKWARD = 5,
    LATTICE_STAGE_CONV_BACKWARD = 6,
    LATTICE_STAGE_SPLAT_BACKWARD = 7,
    LATTICE_STAGE_DOWNSAMPLE = 8,  /* recorded on the output (coarse) lattice */
    LATTICE_STAGE_UPSAMPLE = 9,    /* recorded on the output (fine) lattice   */
    LATTICE_STAGE_DISTRIBUTE = 10,
    LATTICE_STAGE_DOWNSAMPLE_BACKWARD = 11,  /* recorded on the coarse lattice */
    LATTICE_STAGE_UPSAMPLE_BACKWARD = 12,    /* recorded on the fine lattice   */
    LATTICE_STAGE_DEFORM_BACKWARD = 13,
    LATTICE_STAGE_DISTRIBUTE_BACKWARD = 14
};
lattice_status lattice_set_timing(lattice *L, int mode);
lattice_status lattice_get_timing(lattice *L, double *ms, int64_t *count);

/* Query the hash capacity and dimension of L. */
int64_t lattice_hash_capacity(const lattice *L);
int lattice_dim(const lattice *L);

const char *lattice_status_string(lattice_status s);
const char *lattice_last_error(const lattice *L);

#ifdef __cplusplus
}
#endif

#endif /* LATTICE_H */
