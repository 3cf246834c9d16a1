/*
 * liblattice: the permutohedral-lattice hot path of LatticeNet
 * (Rosu, Schuett, Quenzel, Behnke, arXiv:1912.05905) on AMD MI355X (gfx950).
 *
 * Lattice notation (paper, Notation section): a lattice V = (C, X) has n
 * vertices with integer coordinates c_v in Z^{d+1} (summing to zero) and
 * values x_v; a point cloud P = (G, F) has m points with positions g_p in R^d
 * and features f_p.  I_p is the set of d+1 vertices of the simplex enclosing
 * p, b_pv the barycentric weight of p at v, J_v the points splatting onto v.
 * Only d = 3 is supported.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Pointers named *_dev are device pointers owned by the caller; they must
 *    stay valid until the work enqueued on the given stream has finished.
 *    Pointers named *_host are read before the call returns.
 *  - All calls enqueue work on `stream` and return without waiting, except
 *    the first call that needs the vertex count n of a lattice
 *    (lattice_num_vertices, or an operator or export on it): it waits once
 *    for the event that follows the lattice's insert kernel.
 *    lattice_create, lattice_coarsen, lattice_num_points and lattice_level
 *    never wait.
 *  - Work space comes from a caching pool of device blocks.  A block goes
 *    back first to the stream that released it, else to another stream once
 *    the releasing stream is idle, else a new block is allocated; only when
 *    a size class already holds four idle blocks of busy streams does a
 *    call wait for one of those streams (with no error).
 *  - Matrices are row-major.  ld_* arguments are row strides in elements
 *    (0 = dense, i.e. the number of channels); they let several ops write
 *    disjoint column ranges of one buffer (channel concatenation).
 *  - Channel counts: multiples of 4 for LAT_F32 and of 8 for LAT_BF16, and
 *    ld_* likewise; device pointers 16-byte aligned.
 *  - Outputs are overwritten, never accumulated into.
 *  - Vertex numbering is the order in which the device hash claimed vertices
 *    (not deterministic); compare lattices by sorting their keys.
 *  - Return value: LAT_OK (0) or a negative LAT_E* status.  Host-detectable
 *    errors return immediately with nothing enqueued.  Errors found on the
 *    device (hash full, coordinate range, non-finite positions) are reported
 *    by the call that waits for that lattice's count (a coarse lattice also
 *    reports its parent's); the handle is then poisoned and every later call
 *    on it returns the same status.  lattice_last_error() gives the text of
 *    the last non-OK status of the calling thread.
 *  - Handles are not thread-safe; distinct handles are independent.
 */
#ifndef LATTICE_H_
#define LATTICE_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lattice_s* lattice_t;

typedef enum { LAT_F32 = 0, LAT_BF16 = 1 } lat_dtype;

enum {
  LAT_OK = 0,
  LAT_EINVAL = -1,        /* bad argument (null pointer, size, alignment, aliasing) */
  LAT_EUNSUPPORTED = -2,  /* d != 3 or an unsupported dtype / channel count */
  LAT_ENOMEM = -3,        /* device allocation failed */
  LAT_EHASHFULL = -4,     /* more distinct vertices than the hash table holds */
  LAT_EKEYRANGE = -5,     /* a vertex coordinate reaches +-2^20 */
  LAT_ENONFINITE = -6,    /* a position is NaN or infinite */
  LAT_EDEVICE = -7,       /* a HIP runtime call failed */
  LAT_ELEVEL = -8         /* lattices not related as the call requires */
};

#define LAT_RELU 1         /* flags bit: apply max(0, .) after bias */
#define LAT_ON_STREAM 1    /* lattice_coarsen_ex flags bit: build on the given stream */
#define LAT_TAPS 9         /* 2(d+1)+1 vertices of the 1-hop neighbourhood */

/* Text of the calling thread's last non-OK status ("" if none). */
const char* lattice_last_error(void);

/* Static name of a status code ("LAT_EHASHFULL", ...). */
const char* lattice_status_string(int status);

/*
 * Build the lattice of a point cloud (Permutohedral Lattice section and
 * Method: positions scaled as G/sigma, each point embedded in H_d, its
 * enclosing simplex found by rounding, the d+1 vertices inserted into a
 * device hash map keyed by their coordinates).
 *   pos_dev        m x d float32 positions.
 *   m              number of points, >= 0 (m = 0 gives an empty lattice).
 *   d              must be 3 (else LAT_EUNSUPPORTED).
 *   sigma_host     d float32 scale factors, each > 0 and finite.
 *   capacity_hint  upper bound on the number of vertices used to size the
 *                  hash table (0: d+1 per point); too small -> LAT_EHASHFULL.
 *   out            receives the new handle (owned by the caller; release it
 *                  with lattice_destroy).
 * The handle keeps the elevated positions (m x 4 float32), every point's
 * simplex (vertex indices and weights), the vertex keys, the neighbour
 * table and the per-vertex point lists J_v.
 */
int lattice_create(const float* pos_dev, int64_t m, int d, const float* sigma_host,
                   int64_t capacity_hint, hipStream_t stream, lattice_t* out);

/*
 * Coarser lattice for Downsample (Proposed Operations: positions divided by
 * 2 create the coarse lattice).  The coarse lattice holds the same points
 * with elevated positions halved, and a table mapping each coarse vertex c
 * and tap t to the fine vertex at 2c + o_t.  The coarse handle refers to
 * `fine`, which must outlive it (destroying a parent with live children
 * returns LAT_ELEVEL).  The coarse level builds its point lists J_v and
 * per-point simplices on the stream of the first operator that reads them
 * (splat, slice, their backward passes, DeformSlice, Distribute, the
 * simplex export); the convolutions need only its tables.  Work on other
 * streams that uses the handle must be ordered after that call.
 */
int lattice_coarsen(lattice_t fine, int64_t capacity_hint, hipStream_t stream, lattice_t* coarse);

/*
 * lattice_coarsen with flags.  LAT_ON_STREAM builds the coarse level on
 * `stream` itself, after the work enqueued there so far, instead of on the
 * library's side stream: for callers that already build their lattices on a
 * stream of their own (overlapping the construction with other work there).
 * Unknown flag bits return LAT_EINVAL.
 */
int lattice_coarsen_ex(lattice_t fine, int64_t capacity_hint, int flags, hipStream_t stream, lattice_t* coarse);

/*
 * A hierarchy of `levels` lattices (1 to 8) in one call, all built on
 * `stream`: out[0] as lattice_create with capacity_hint h[0], out[l] as
 * lattice_coarsen_ex(out[l - 1], h[l], LAT_ON_STREAM, stream, ...) for
 * l >= 1 (Proposed Operations: each coarser level is the same points with
 * positions divided by 2), where h = capacity_hints (`levels` values in
 * host memory, or all 0 when capacity_hints is null; negative values count
 * as 0).  A hint sizes its level's hash table as lattice_create's
 * capacity_hint does (0 = automatic), except that a table that overflows is
 * rebuilt at the worst-case size (as with hint 0) instead of failing.  A
 * caller that builds clouds of similar sizes in turn can pass the last
 * cloud's vertex counts (smaller tables to clear and probe).  The lattices
 * are those of that sequence of calls (the vertex sets and simplices do not
 * depend on the table sizes); the device work is issued in fewer launches
 * and in an order that
 * gives the host every level's vertex count sooner: the levels' tables are
 * cleared in one launch, the inserts of all levels run in one launch (each
 * level elevates the positions and halves them l times, which gives the
 * same floats as halving the finer level's), then the finest level's lists,
 * the convolution tables of all levels in one launch and the row orders of
 * all tables in one launch.
 * out must hold `levels` handles; on an error none is created.  Handles
 * are destroyed coarsest first, as for lattice_coarsen.
 */
int lattice_create_hierarchy(const float* pos_dev, int64_t m, int d, const float* sigma_host, int levels,
                             const int64_t* capacity_hints, hipStream_t stream, lattice_t* out);

/* Release a handle and its device memory (LAT_ELEVEL while it has children). */
int lattice_destroy(lattice_t L);

/* Number of vertices n / of points m.  Reports deferred device errors. */
int lattice_num_vertices(lattice_t L, int64_t* n);
int lattice_num_points(lattice_t L, int64_t* m);

/* Coarsening level of a handle (0 for lattice_create). */
int lattice_level(lattice_t L, int* level);

/* Vertex coordinates c_v, n x (d+1) int32. */
int lattice_export_keys(lattice_t L, int32_t* keys_dev, hipStream_t stream);

/* Per point: the d+1 vertex indices of I_p (m x (d+1) int32, vertex k has
 * every coordinate congruent to k mod d+1) and weights b_pv (m x (d+1)). */
int lattice_export_simplices(lattice_t L, int32_t* idx_dev, float* w_dev, hipStream_t stream);

/* 1-hop neighbour table, n x 9 int32: column 0 the vertex itself, 1..d+1 the
 * vertex at c + n_j, d+2..2d+2 at c - n_j, n_j = (d+1)e_j - 1; -1 where the
 * neighbour is not allocated (Permutohedral Lattice section). */
int lattice_export_neighbors(lattice_t L, int32_t* nbr_dev, hipStream_t stream);

/*
 * Occupied taps of a convolution (Fig. (convolve): a missing neighbour
 * contributes nothing): the number of (output vertex, tap) pairs whose
 * neighbour exists, for the 1-hop (dst == src), strided (dst =
 * lattice_coarsen(src)) or Upsample (src = lattice_coarsen(dst)) form.
 * The work the convolution must do is 2 Cin Cout per pair.  Written to
 * *pairs_host; waits for the stream (for measurement, not for hot loops).
 */
int lattice_conv_taps(lattice_t dst, lattice_t src, int64_t* pairs_host, hipStream_t stream);

/*
 * Splat, Eq. (splat): x_v = sum_{p in J_v} b_pv f_p.
 *   feat_dev   m x C features (dtype dt), row stride ld_feat.
 *   normalize  nonzero: divide by sum_{p in J_v} b_pv (the weighted average
 *              the paper describes), 0 where that sum is 0.
 *   vals_dev   n x C output (dtype dt, float32 accumulation), row stride ld_vals.
 *   wsum_dev   optional n float32 sums of weights (may be NULL).
 */
int lattice_splat(lattice_t L, const void* feat_dev, int64_t ld_feat, int C, lat_dtype dt,
                  int normalize, void* vals_dev, int64_t ld_vals, float* wsum_dev,
                  hipStream_t stream);

/*
 * lattice_splat without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, arithmetic and
 * results as lattice_splat; its partial sums live in a fixed 16 MiB scratch
 * array in device memory, one per GPU, held until the process ends and
 * shared by every call on that GPU:
 * calls that overlap on one GPU (concurrent streams or threads) race.
 * Requires the lattice's vertex count to have been read
 * (lattice_num_vertices; else LAT_EINVAL).  A splat whose partials need
 * more than the scratch (about (2C + 2) floats per 256 list entries) returns
 * LAT_EUNSUPPORTED with nothing enqueued.  Never calls hipMalloc or hipFree.
 */
int lattice_splat_noalloc(lattice_t L, const void* feat_dev, int64_t ld_feat, int C, lat_dtype dt, int normalize,
                          void* vals_dev, int64_t ld_vals, float* wsum_dev, hipStream_t stream);

/*
 * Lattice convolution (Method, Convolving; Downsample):
 *   out[v] = bias + sum_{t<9} in[nb(v,t)] W[t]^T   (missing neighbours add 0)
 *   dst == src: 1-hop convolution, nb(v,t) = vertex at c_v + o_t.
 *   dst = lattice_coarsen(src): strided convolution, nb(v,t) = fine vertex
 *   at 2 c_v + o_t (the values of the coarse lattice).
 *   in_dev    n_src x Cin (dtype dt), row stride ld_in.
 *   W_dev     9 x Cout x Cin (dtype dt): W[t][o][i] multiplies input channel
 *             i of tap t into output channel o.  Taps: 0 self, 1+j +n_j,
 *             5+j -n_j.
 *   bias_dev  optional Cout float32.
 *   flags     LAT_RELU or 0.
 *   out_dev   n_dst x Cout (dtype dt, float32 accumulation), row stride
 *             ld_out; must not overlap in_dev.
 */
int lattice_conv(lattice_t dst, lattice_t src, const void* in_dev, int64_t ld_in, int Cin,
                 const void* W_dev, const float* bias_dev, int Cout, lat_dtype dt, int flags,
                 void* out_dev, int64_t ld_out, hipStream_t stream);

/*
 * Upsample (Proposed Operations): transposed convolution from `coarse`
 * (= lattice_coarsen(fine)) to `fine`.  Fine vertex f reads, for tap t, the
 * coarse vertex at (c_f + o_t)/2 when that is a lattice point; taps landing
 * between coarse vertices contribute nothing.  With W[t] = W_down[mirror t]^T
 * this is exactly the adjoint of the strided convolution.  Arguments as for
 * lattice_conv with in_dev n_coarse x Cin and out_dev n_fine x Cout.
 */
int lattice_refine(lattice_t fine, lattice_t coarse, const void* in_dev, int64_t ld_in, int Cin,
                   const void* W_dev, const float* bias_dev, int Cout, lat_dtype dt, int flags,
                   void* out_dev, int64_t ld_out, hipStream_t stream);

/*
 * Pre-activated convolutions (Implementation: every convolution is
 * pre-activated by Group Normalization with 32 groups and a ReLU):
 *   out = conv(relu(GN(in))) for lattice_conv_preact (1-hop or strided, as
 *   lattice_conv) and lattice_refine_preact (Upsample, as lattice_refine).
 * GN: channel c of in belongs to group c / (Cin / groups); mean and biased
 * variance of a group over all rows of the input lattice and its channels
 * (summed in float64 in a fixed order); each value becomes
 * (x - mean) / sqrt(var + eps) * gamma_c + beta_c, then max(., 0).  The
 * normalisation is applied inside the convolution to the gathered values of
 * neighbours that exist (a missing neighbour still contributes 0); the
 * normalised input is never stored.
 *   groups     divides Cin (the paper uses 32); gamma_dev / beta_dev
 *              optional Cin float32 (NULL = 1 / 0); eps > 0.
 *   res_dev    lattice_conv_preact only: optional n_dst x Cout residual
 *              (dtype dt, row stride ld_res, 0 = Cout) added to the output
 *              after its activation -- the identity branch of a ResNet
 *              block (architecture figure).  It may be out_dev itself (same
 *              row stride), any other overlap with out_dev is rejected.
 *   Other arguments as for lattice_conv / lattice_refine.  Cin <= 1024.
 */
int lattice_conv_preact(lattice_t dst, lattice_t src, const void* in_dev, int64_t ld_in, int Cin, int groups,
                        const float* gamma_dev, const float* beta_dev, float eps, const void* W_dev,
                        const float* bias_dev, int Cout, lat_dtype dt, int flags, const void* res_dev,
                        int64_t ld_res, void* out_dev, int64_t ld_out, hipStream_t stream);
int lattice_refine_preact(lattice_t fine, lattice_t coarse, const void* in_dev, int64_t ld_in, int Cin, int groups,
                          const float* gamma_dev, const float* beta_dev, float eps, const void* W_dev,
                          const float* bias_dev, int Cout, lat_dtype dt, int flags, void* out_dev, int64_t ld_out,
                          hipStream_t stream);

/*
 * Distribute + PointNet (Proposed Operations, Eq. (distribute); the scaled
 * positions G_s = G / sigma of the Method section; PointNet block of the
 * architecture figure).  For every vertex v each point p of J_v gives a row
 *   r = [g_p / sigma - mu_v ; f_p],  mu_v = mean of g_p / sigma over J_v,
 * with sigma the lattice's scale (doubled per coarsening level).  The rows
 * pass three blocks [GroupNorm, ReLU, 1x1]:
 *   h_i = W_i relu(GN_i(h_{i-1})) + b_i   (h_0 = r, i = 1, 2, 3),
 * and x_v is the per-channel maximum of h_3 over J_v (MaxPool).
 * GN_i: mean and biased variance over all distributed rows (every (v, p)
 * pair, (d+1) m rows) and the channels of a group; a layer input of at most
 * 32 channels has one channel per group, a wider one 32 groups; then
 * (x - mean) / sqrt(var + eps) * gamma_c + beta_c.  Statistics are summed
 * in float64 in a fixed order.  float32 only.
 *   pos_dev    m x d float32, the positions the lattice was built from.
 *   feat_dev   m x Cf float32, row stride ld_feat (0 = Cf); may be NULL when
 *              Cf = 0.  0 <= Cf <= 29 (d + Cf <= 32).
 *   gn_gamma_dev, gn_beta_dev  optional per-channel parameters of the
 *              three normalisations, concatenated: (d + Cf) for the raw
 *              rows (coordinates first), then C1, then C2 (NULL = 1 / 0).
 *   eps        >= 0, finite (the paper's default is 1e-5).
 *   W1_dev     C1 x (d + Cf) float32, [out][in]: inputs 0..d-1 are the
 *              coordinates, d.. the features.  W2_dev C2 x C1, W3_dev C3 x C2.
 *   b*_dev     optional C1 / C2 / C3 float32 biases (NULL = 0).
 *   C1, C2, C3  16, 32 or 64 (C3 also 48; the paper uses 16, 32, 64).
 *   out_dt     LAT_F32, or LAT_BF16 (the float32 maxima rounded to nearest
 *              even, for a bfloat16 network).
 *   out_dev    n x C3 of out_dt, row stride ld_out (0 = C3).
 * A non-finite feature makes every output value NaN (the statistics it
 * reaches are not finite).  Uses a work space of O(n + 4m) bytes from the
 * library's pool.
 */
int lattice_distribute_pointnet(lattice_t L, const float* pos_dev, const float* feat_dev, int64_t ld_feat,
                                int Cf, const float* gn_gamma_dev, const float* gn_beta_dev, float eps,
                                const float* W1_dev, const float* b1_dev, int C1, const float* W2_dev,
                                const float* b2_dev, int C2, const float* W3_dev, const float* b3_dev, int C3,
                                lat_dtype out_dt, void* out_dev, int64_t ld_out, hipStream_t stream);

/*
 * Slice, Eq. (slice): out_p = sum_{v in I_p} b_pv x_v.
 *   vals_dev  n x C (dtype dt), row stride ld_vals.
 *   out_dev   m x C float32 (dense).
 */
int lattice_slice(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                  float* out_dev, hipStream_t stream);

/*
 * DeformSlice, Eq. (deformSlice) with the permutation-equivariant offsets:
 *   q_k = b_k x_k (k over I_p),  M = max_k q_k per channel,
 *   db_k = tanh(beta + (q_k - M) . wv),  out_p = sum_k (b_k + db_k) x_k.
 *   wv_dev     C float32 weight vector, beta the scalar bias.
 *   out_dev    m x C float32; delta_dev optional m x (d+1) float32 offsets.
 */
int lattice_deform_slice(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                         const float* wv_dev, float beta, float* out_dev, float* delta_dev,
                         hipStream_t stream);

/*
 * Slice (Eq. slice) and DeformSlice (Eq. deformSlice) of the same values in
 * one pass over the gathered vertex rows: slice_dev receives what
 * lattice_slice writes, deform_dev what lattice_deform_slice writes (same
 * arithmetic, same results).  Both m x C float32, dense, not overlapping;
 * the rest as lattice_deform_slice (no offsets output).
 */
int lattice_slice_and_deform(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                             const float* wv_dev, float beta, float* slice_dev, float* deform_dev,
                             hipStream_t stream);

/*
 * DeformSlice fused with the last linear classification layer
 * (Implementation: fused to avoid storing the high-dimensional per-point
 * features): logits_p = Wc f_p + bc, f_p the DeformSlice output of point p
 * (as lattice_deform_slice, which this does not store).
 *   Wc_dev     K x C float32 [class][channel], 16-byte aligned;
 *   bc_dev     optional K float32;  1 <= K <= 64, K x C <= 16384.
 *   logits_dev m x K float32, row stride K.
 * Other arguments as for lattice_deform_slice.
 */
int lattice_deform_slice_classify(lattice_t L, const void* vals_dev, int64_t ld_vals, int C, lat_dtype dt,
                                  const float* wv_dev, float beta, const float* Wc_dev, const float* bc_dev, int K,
                                  float* logits_dev, hipStream_t stream);

/*
 * Backward passes (Implementation: the lattice operators have forward and
 * backward passes on the GPU).  Each returns the gradient of a scalar loss
 * with respect to the forward's inputs, given its gradient with respect to
 * the forward's output.  float32 only.  Output buffers are overwritten (not
 * accumulated into).
 */

/*
 * Splat backward: dF_p = sum_{v in I_p} b_pv dX_v (Eq. (splat) transposed);
 * with normalize != 0 each term is divided by wsum_v = sum_{q in J_v} b_qv
 * (0 where wsum_v = 0), the gradient of the normalised splat.
 *   dX_dev    n x C float32, row stride ld_dX (0 = C).  C a multiple of 4.
 *   wsum_dev  optional n float32: the weight sums the forward lattice_splat
 *             returned; NULL = summed again over the lists.  Only read when
 *             normalize != 0.
 *   dF_dev    m x C float32, row stride C.
 */
int lattice_splat_backward(lattice_t L, const float* dX_dev, int64_t ld_dX, int C, int normalize,
                           const float* wsum_dev, float* dF_dev, hipStream_t stream);

/*
 * Slice backward: dX_v = sum_{p in J_v} b_pv dOut_p (Eq. (slice)
 * transposed), computed as a splat over the vertex lists.
 *   dOut_dev  m x C float32, row stride ld_dOut (0 = C).
 *   dX_dev    n x C float32, row stride ld_dX (0 = C).  C <= 256.
 */
int lattice_slice_backward(lattice_t L, const float* dOut_dev, int64_t ld_dOut, int C, float* dX_dev, int64_t ld_dX,
                           hipStream_t stream);

/*
 * Convolution backward for Y = act(conv(X, W) + bias) as computed by
 * lattice_conv(dst, src) (1-hop or strided) or lattice_refine(dst, src)
 * (Upsample: src = lattice_coarsen(dst)); the form follows from dst and src.
 *   X_dev     n_src x Cin forward input (needed for dW), row stride ld_X.
 *   W_dev     9 x Cout x Cin forward weights (needed for dX).
 *   flags     LAT_RELU if the forward applied the ReLU; then Y_dev (n_dst x
 *             Cout, row stride ld_Y) is the forward output and dY is masked
 *             by Y > 0 (the derivative is taken as 0 at 0).
 *   dY_dev    n_dst x Cout gradient of the output, row stride ld_dY.
 *   dX_dev    n_src x Cin, row stride ld_dX, or NULL: the convolution of the
 *             masked dY with W'[t] = W[mirror t]^T over the adjoint table;
 *             must not overlap dY.
 *   dW_dev    9 x Cout x Cin, or NULL: dW[t] = sum_v dY_v^T X[nb(v,t)].
 *   dbias_dev Cout (16-byte aligned), or NULL: sum_v dY_v.
 * Row strides of 0 mean dense.  Cin, Cout multiples of 4.  Uses work space
 * from the library's pool; the sums over vertices run in a fixed order.
 */
int lattice_conv_backward(lattice_t dst, lattice_t src, const float* X_dev, int64_t ld_X, int Cin, const float* W_dev,
                          int Cout, int flags, const float* Y_dev, int64_t ld_Y, const float* dY_dev, int64_t ld_dY,
                          float* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev, hipStream_t stream);

/*
 * lattice_conv_backward for a bfloat16 (or float32) network: X, W, Y, dY and
 * dX are of dtype dt (LAT_BF16: channels and row strides multiples of 8).
 * dX is the adjoint convolution on the matrix cores with bfloat16 operands
 * and float32 accumulation, rounded to dt once; dW and dbias stay float32
 * (the bfloat16 values are widened exactly and summed in float32).  Other
 * arguments and rules as for lattice_conv_backward.
 */
int lattice_conv_backward_ex(lattice_t dst, lattice_t src, const void* X_dev, int64_t ld_X, int Cin, const void* W_dev,
                             int Cout, lat_dtype dt, int flags, const void* Y_dev, int64_t ld_Y, const void* dY_dev,
                             int64_t ld_dY, void* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev,
                             hipStream_t stream);

/*
 * Backward of the pre-activated convolution (Implementation: Group
 * Normalization with a ReLU before every convolution) for
 *   Y = act(conv(relu(GN(X)), W) + bias)
 * as lattice_conv_preact / lattice_refine_preact compute it (1-hop,
 * strided or Upsample: the form follows from dst and src as for
 * lattice_conv_backward), given dY = dL/dY:
 *   A = relu(GN(X)) is recomputed exactly as the forward applied it, the
 *   convolution's backward on A gives dW, dbias and dA, and the GroupNorm +
 *   ReLU backward of dA gives
 *     dbeta_c = sum_v g,  dgamma_c = sum_v g xhat,  g = dA [GN(X) > 0],
 *     dX = inv_g (gamma_c g - mean_g(gamma g) - xhat mean_g(gamma g xhat))
 *   with xhat = (X - mean_g) inv_g, inv_g = 1 / sqrt(var_g + eps), the
 *   group means over all rows of src and the group's channels (sums in
 *   float64, fixed order).
 *   X_dev      n_src x Cin float32, row stride ld_X (0 = Cin): the input the
 *              forward normalised; Cin <= 1024, a multiple of 4.
 *   groups, gamma_dev, beta_dev, eps   as for lattice_conv_preact.
 *   W_dev, Cout, flags, Y_dev, dY_dev  as for lattice_conv_backward (Y is
 *              the output before any residual was added; a residual's own
 *              gradient is dY itself).
 *   dX_dev     n_src x Cin, row stride ld_dX, or NULL; must not overlap X.
 *   dW_dev, dbias_dev  as for lattice_conv_backward, or NULL.
 *   dgamma_dev, dbeta_dev  Cin float32 each, or NULL.
 * float32 only.  Uses work space of O(n_src Cin) bytes from the pool.
 */
int lattice_conv_preact_backward(lattice_t dst, lattice_t src, const float* X_dev, int64_t ld_X, int Cin, int groups,
                                 const float* gamma_dev, const float* beta_dev, float eps, const float* W_dev,
                                 int Cout, int flags, const float* Y_dev, int64_t ld_Y, const float* dY_dev,
                                 int64_t ld_dY, float* dX_dev, int64_t ld_dX, float* dW_dev, float* dbias_dev,
                                 float* dgamma_dev, float* dbeta_dev, hipStream_t stream);

/*
 * DeformSlice backward (Eq. (deformSlice) with the equivariant offset
 * regressor) for out_p = sum_k (b_pk + db_pk) x_k, db_pk = tanh(beta +
 * (b_pk x_k - max_j b_pj x_j) . wv), given dOut = dL/dout:
 *   dvals  n x C (row stride ld_dvals): dL/dx for every vertex, gathered
 *          over the vertex lists (deterministic order);
 *   dwv    C floats: dL/dwv;  dbeta  1 float: dL/dbeta.
 * The maximum passes its gradient to the first vertex slot whose float32
 * product b_pk x_k is maximal.  vals, wv, beta are the forward's inputs (n x
 * C float32, row stride ld_vals); dOut is m x C (row stride ld_dOut).  Row
 * strides of 0 mean dense; C a multiple of 4, at most 512; dvals must not
 * overlap vals.  Uses work space of O(m (64 + C)) bytes from the pool.
 */
int lattice_deform_slice_backward(lattice_t L, const float* vals_dev, int64_t ld_vals, int C, const float* wv_dev,
                                  float beta, const float* dOut_dev, int64_t ld_dOut, float* dvals_dev,
                                  int64_t ld_dvals, float* dwv_dev, float* dbeta_dev, hipStream_t stream);

/*
 * Backward of DeformSlice fused with the linear classifier (Implementation:
 * the last linear layer fused with DeformSlice) for logits_p = Wc f_p + bc
 * as lattice_deform_slice_classify computes it, given dlogits = dL/dlogits
 * (m x K float32, row stride ld_dlogits, 0 = K):
 *   dWc = sum_p dlogits_p f_p^T (K x C), dbc = sum_p dlogits_p (K), each
 *   summed over chunks of points added in a fixed order; df_p = Wc^T
 *   dlogits_p, and the DeformSlice backward of df (as
 *   lattice_deform_slice_backward) gives dvals, dwv and dbeta.
 * f is recomputed from vals (float32, as lattice_deform_slice) and not
 * stored by the caller.  dWc_dev / dbc_dev may be NULL; the other outputs
 * are required.  Limits as lattice_deform_slice_classify (K <= 64, K x C <=
 * 16384, C <= 512); dvals must not overlap vals.  Uses work space of
 * O(m C) bytes from the pool.
 */
int lattice_deform_slice_classify_backward(lattice_t L, const float* vals_dev, int64_t ld_vals, int C,
                                           const float* wv_dev, float beta, const float* Wc_dev, int K,
                                           const float* dlogits_dev, int64_t ld_dlogits, float* dvals_dev,
                                           int64_t ld_dvals, float* dwv_dev, float* dbeta_dev, float* dWc_dev,
                                           float* dbc_dev, hipStream_t stream);

/*
 * Distribute + PointNet backward (Proposed Operations, Eq. (distribute);
 * PointNet block of the architecture figure) for x = the
 * lattice_distribute_pointnet output, given dX = dL/dx (n x C3 float32, row
 * stride ld_dX, 0 = C3):
 *   the maximum over J_v passes dX[v][c] to the row of J_v holding channel
 *   c's maximum (the first such row in the lattice's list order);
 *   each block h_i = W_i relu(GN_i(h_{i-1})) + b_i goes backward as
 *     dW_i = sum_rows dh_i a_{i-1}^T,  db_i = sum_rows dh_i,  da_{i-1} = W_i^T dh_i,
 *   then the GroupNorm + ReLU backward of da_{i-1} (as described for
 *   lattice_conv_preact_backward, statistics over all rows) gives dh_{i-1}
 *   and the normalisation's dgamma / dbeta;
 *   dfeat_p = sum over the d+1 rows of point p of the feature part of dh_0.
 * The forward is recomputed in float32 (every block's input kept in the
 * work space); positions are inputs and get no gradient.
 *   Arguments pos_dev .. C3 as for lattice_distribute_pointnet (W2_dev and
 *   W3_dev 16-byte aligned).
 *   dfeat_dev  m x Cf float32, row stride ld_dfeat (0 = Cf), or NULL.
 *   dW*_dev    C1 x (d + Cf), C2 x C1, C3 x C2 ([out][in]) or NULL;
 *   db*_dev    C1 / C2 / C3 or NULL.
 *   dgamma_dev, dbeta_dev  (d + Cf) + C1 + C2 floats each (the layout of
 *              gn_gamma_dev), or NULL.
 * Sums over rows run in a fixed order.  Uses work space of about
 * 4 m ((d + Cf) + C1 + C2 + 4 max width) floats from the pool.
 */
int lattice_distribute_pointnet_backward(lattice_t L, const float* pos_dev, const float* feat_dev, int64_t ld_feat,
                                         int Cf, const float* gn_gamma_dev, const float* gn_beta_dev, float eps,
                                         const float* W1_dev, const float* b1_dev, int C1, const float* W2_dev,
                                         const float* b2_dev, int C2, const float* W3_dev, const float* b3_dev, int C3,
                                         const float* dX_dev, int64_t ld_dX, float* dfeat_dev, int64_t ld_dfeat,
                                         float* dW1_dev, float* db1_dev, float* dW2_dev, float* db2_dev,
                                         float* dW3_dev, float* db3_dev, float* dgamma_dev, float* dbeta_dev,
                                         hipStream_t stream);

/*
 * Timing of the library's kernels with HIP events on the launch stream, for
 * measurement.  enable != 0 records a start/stop event pair around every
 * launch of the kernel family `name` ("conv", "splat", "slice", "insert",
 * ...); lattice_timing_read waits for the recorded events and returns the
 * number of launches and their summed duration in milliseconds, then clears
 * the record.
 */
int lattice_timing_enable(const char* name, int enable);
int lattice_timing_read(const char* name, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* LATTICE_H_ */
