/*
 * e3mi -- channelwise Clebsch-Gordan tensor product and message-passing
 * convolution on AMD Instinct MI355X (gfx950).  C ABI.
 *
 * The operation (App. E.1 of "E3J: An Efficient and Open-Source Backend for
 * Euclidean Equivariant Operations on GPU and TPU"):
 *
 *   tensor product, eq. (tensor_product_formula) and eq. (edge_scalar_weighting):
 *     z[r, i0, q] = w[r, i3(i0), q] * sum_{i1,i2} C[i0, i1, i2] x[r, i1, q] y[r, i2]
 *   convolution, eq. (message_passing_convolution):
 *     m[b, i0, q] = sum_{e : receiver(e) = b} s[e, i3(i0), q] *
 *                   sum_{i1,i2} C[i0, i1, i2] x[sender(e), i1, q] Y(vec[e]/|vec[e]|)[i2]
 *   backward, eq. (conv-bwd): dx, ds and dvec from dm (dvec through the
 *     harmonics' Jacobian).
 *
 * Index spaces.  An irreps string "Cx l p + ..." (every block with the same
 * multiplicity C, the channel count) defines the x feature axis D_in: block
 * by block, rows m = -l..l.  The harmonics axis D_sh holds l2 = 0..lmax_sh,
 * rows m = -l2..l2 (D_sh = (lmax_sh+1)^2).  Paths are enumerated x block by
 * x block, then l2 ascending, then l3 ascending from |l1-l2| to
 * min(l1+l2, lmax_out); each path owns 2*l3+1 consecutive rows of the output
 * axis D_out and one scalar block (i3) of the weights.
 *
 * Conventions (the paper leaves them open): unitary real Clebsch-Gordan
 * coefficients in the basis of the real harmonics below, canonical sign =
 * first non-zero entry of each path block (row-major over (M, m1, m2))
 * positive; harmonics Y_l(u) = S_l(u_z, u_x, u_y) with S_l the textbook real
 * solid harmonics, sum_m Y_lm(u)^2 = 2l+1, so Y_0 = 1 and Y_1(u) = sqrt(3) u.
 *
 * Layouts: every tensor is float32, contiguous, row-major, channels last
 * ("trailing channels", App. E.1):
 *   x, dx  [N, D_in, C]      m, dm  [N, D_out, C]
 *   s, ds  [E, P, C]         vec, dvec [E, 3]
 *   y      [rows, D_sh]      (tensor product: x [R, D_in, C], w [R, P, C],
 *                              z [R, D_out, C])
 *
 * Ownership: all data pointers are device buffers owned by the caller.  Plan
 * and graph handles are owned by the library (create/destroy).  Calls that
 * take a stream are asynchronous on it; the *_fwd / *_bwd / e3_sh* entry
 * points never allocate, never synchronise, and fully overwrite their
 * outputs.  Results are bitwise reproducible for identical inputs on one
 * device and build: every floating-point sum runs in a fixed order
 * (receiver-sorted or sender-sorted CSR order and a fixed reduction tree) and
 * no floating-point atomics are used (the graph build counts keys with
 * integer atomics, whose result does not depend on their order).
 *
 * Errors: every call returns an e3_status; nothing is thrown across the ABI.
 * Arguments are validated before any device work is enqueued.
 */
#ifndef E3MI_H
#define E3MI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  E3_OK = 0,
  E3_ERR_INVALID_ARG = 1,          /* null/misaligned pointer, negative size, bad irreps string */
  E3_ERR_UNSUPPORTED = 2,          /* no kernels for these irreps (see e3_plan_create), or C unsupported */
  E3_ERR_INDEX_OUT_OF_RANGE = 3,   /* an edge index outside [0, n_nodes) */
  E3_ERR_WORKSPACE_TOO_SMALL = 4,  /* ws_bytes below e3_conv_workspace_size */
  E3_ERR_HIP = 5,                  /* a HIP runtime call failed; see e3_last_error() */
  E3_ERR_ALLOC = 6                 /* a library-owned allocation failed (create calls only) */
} e3_status;

/* Opaque handles. */
typedef struct e3_plan e3_plan;    /* paths, i3, offsets, coupling tables, kernels */
typedef struct e3_graph e3_graph;  /* receiver- and sender-sorted CSR of an edge list, on device */

/* hipStream_t without the HIP headers; pass 0 for the null stream. */
typedef void* e3_stream;

#define E3_PARITY_ALL 0u      /* keep every triangle-allowed path (default) */
#define E3_PARITY_NATURAL 1u  /* keep only paths whose output parity is (-1)^l3 */
#define E3_PLAN_RECORDS 2u    /* run on the record path even where a compiled variant exists */
#define E3_PLAN_COMPOSED 4u   /* run on the composed path even where a compiled variant exists */

typedef struct {
  int C;            /* channels (the common multiplicity) */
  int P;            /* number of paths == number of scalar blocks per edge */
  int D_in, D_sh, D_out;
  int nnz;          /* non-zero coupling records */
  int lmax_sh, lmax_out;
  int supported;    /* 1: a compiled kernel variant; 2: the record path; 3: the composed path; 0: none */
} e3_plan_info;

/* Builds the path list and the coupling tables on the host (float64).
 * irreps_x: e.g. "128x0e+128x1o+128x2e+128x3o".  lmax_sh in [0, 3],
 * lmax_out >= 0.  flags: E3_PARITY_ALL or E3_PARITY_NATURAL, optionally or-ed
 * with one of E3_PLAN_RECORDS and E3_PLAN_COMPOSED.  INVALID_ARG for a
 * malformed string, out-of-range degree or unknown flag (or both path
 * flags); UNSUPPORTED when the blocks have different multiplicities.
 *
 * Kernels.  A layout whose path list was compiled into the library runs its
 * generated kernels (info.supported == 1).  Any other layout with x blocks
 * and outputs of degree <= 3 and C a multiple of 4 up to 1024 runs on the
 * composed path (info.supported == 3): the library also holds generated
 * kernels for every single x block (degree, all or natural-parity paths,
 * harmonics and output degrees), and runs them block by block with the
 * layout's strides and offsets; each block writes its own output rows, ds
 * rows, x-cotangent partial rows and harmonic partial sums, which the shared
 * sender-order segment sum and the harmonic sum then complete.  Nothing is
 * uploaded.  E3_PLAN_RECORDS selects instead the record path
 * (info.supported == 2): the generic sparse kernel of App. E ("CUDA
 * kernels"), which walks the plan's unfolded records (i0, i1, i2, C) at run
 * time, lanes on the channels, each receiver's messages summed on chip; its
 * tables are uploaded at creation to the device current then (the call
 * allocates and waits for the copy), and its compute calls return
 * E3_ERR_INVALID_ARG when another device is current.  E3_PLAN_COMPOSED
 * selects the composed path even for a compiled layout.  Both paths serve
 * e3_tp_fwd / e3_tp_bwd / e3_tp_workspace_size, e3_conv_fwd / e3_conv_bwd /
 * e3_conv_workspace_size / e3_conv_bwd_noalloc, e3_conv_fwd_y /
 * e3_conv_bwd_y and e3_conv_bwd2, with the same semantics (deterministic,
 * atomics-free); the composed path also serves the float64 builds and the
 * fused radial weights (the record path has neither).  Otherwise (a larger degree; the record path without a device
 * at creation) the plan is still created (info.supported == 0): its tables
 * can be queried, and the compute entry points return E3_ERR_UNSUPPORTED. */
e3_status e3_plan_create(const char* irreps_x, int lmax_sh, int lmax_out, unsigned flags,
                         e3_plan** out);
e3_status e3_plan_query(const e3_plan* plan, e3_plan_info* info);
e3_status e3_plan_destroy(e3_plan* plan);

/* Host copies of the plan's tables (for inspection and tests).
 * e3_plan_paths: per path (l1, l2, l3, p3, x_off, y_off, out_off), 7 ints each,
 * into paths[7*P].  e3_plan_records: the non-zero records (App. E.2's unfolded
 * COO form) sorted by (i0, i1, i2); writes at most cap records and sets *n to
 * the total count. */
e3_status e3_plan_paths(const e3_plan* plan, int32_t* paths);
e3_status e3_plan_records(const e3_plan* plan, int64_t cap, int32_t* i0, int32_t* i1,
                          int32_t* i2, double* val, int64_t* n);

/* Host evaluation of the builder's harmonic polynomials (float64), rows
 * [n, (lmax+1)^2], for unit vectors u[n, 3].  lmax in [0, 3]. */
e3_status e3_sh_host(int lmax, const double* u, double* y, int64_t n);

/* Builds the receiver- and sender-sorted CSR on the device (App. E.2.2 /
 * App. E.3 receiver order; App. E.4 sender order for the backward).
 * sender, receiver: device int32 [n_edges].  Edges with the same key keep
 * their edge-id order (stable).  Edges with sender or receiver equal to
 * pad_node (pad_node >= 0) are padding: they are skipped by every kernel and
 * get zero cotangents; pad_node = -1 means no padding node.
 * Validates every index (E3_ERR_INDEX_OUT_OF_RANGE); it synchronises the
 * stream to read the validation result and again before it frees its
 * temporaries (the sort's key and count buffers).  n_edges may be 0.  The
 * graph allocates its own device memory. */
e3_status e3_graph_create(const int32_t* sender, const int32_t* receiver, int64_t n_nodes,
                          int64_t n_edges, int32_t pad_node, e3_stream stream, e3_graph** out);
/* Number of non-padding edges. */
e3_status e3_graph_live_edges(const e3_graph* g, int64_t* n_live);
/* Copies the CSR to device buffers: perm_r[n_live] (edge ids by receiver),
 * rowptr_r[n_nodes+1], perm_s[n_live] (edge ids by sender), rowptr_s[n_nodes+1].
 * Any pointer may be null.  Synchronous on the null stream. */
e3_status e3_graph_export(const e3_graph* g, int32_t* perm_r, int32_t* rowptr_r, int32_t* perm_s,
                          int32_t* rowptr_s);
e3_status e3_graph_destroy(e3_graph* g);

/* Real harmonics of edge vectors (App. A.3 "Harmonics"): y[n, (lmax+1)^2] =
 * Y(vec/|vec|).  lmax in [0, 3].  A zero vector gives Y_0 = 1 and zeros. */
e3_status e3_sh(int lmax, const float* vec, float* y, int64_t n, e3_stream stream);
/* dvec[n, 3] = (dY/dvec)^T dy[n, (lmax+1)^2]; zero for a zero vector. */
e3_status e3_sh_bwd(int lmax, const float* vec, const float* dy, float* dvec, int64_t n,
                    e3_stream stream);

/* Weighted tensor product (App. E.1, eq. tensor_product_formula with
 * eq. edge_scalar_weighting): x [rows, D_in, C], y [rows, D_sh] (broadcast over
 * channels), w [rows, P, C] -> z [rows, D_out, C]. */
e3_status e3_tp_fwd(const e3_plan* plan, const float* x, const float* y, const float* w, float* z,
                    int64_t rows, e3_stream stream);

/* Backward of the weighted tensor product (App. E.1, eq. tp-bwd with the path
 * weight of eq. edge_scalar_weighting): from dz [rows, D_out, C] computes
 * dx [rows, D_in, C], dy [rows, D_sh] (summed over channels) and dw [rows, P, C],
 * streaming x, y, w and dz once.  ws: at least e3_tp_workspace_size bytes (the
 * per-wave partial sums of dy, added in a fixed order). */
e3_status e3_tp_workspace_size(const e3_plan* plan, int64_t rows, size_t* bwd_bytes);
e3_status e3_tp_bwd(const e3_plan* plan, const float* x, const float* y, const float* w, const float* dz,
                    float* dx, float* dy, float* dw, void* ws, size_t ws_bytes, int64_t rows, e3_stream stream);

/* Device workspace the convolution needs (bytes, 256-byte aligned start).
 * Forward: 0.  Backward: the per-edge x-cotangent partials [n_live, D_in, C]
 * summed later in sender order, plus the per-edge harmonic cotangents. */
e3_status e3_conv_workspace_size(const e3_plan* plan, const e3_graph* graph, size_t* fwd_bytes,
                                 size_t* bwd_bytes);

/* Forward convolution (eq. message_passing_convolution): m [n_nodes, D_out, C].
 * Receivers with no live in-edge (and the padding node) get m = 0. */
e3_status e3_conv_fwd(const e3_plan* plan, const e3_graph* graph, const float* x, const float* vec,
                      const float* s, float* m, void* ws, size_t ws_bytes, e3_stream stream);

/* Backward convolution (eq. conv-bwd): from dm [n_nodes, D_out, C] computes
 * dx [n_nodes, D_in, C], dvec [E, 3] and ds [E, P, C].  Deterministic and
 * atomics-free: edge-local cotangents in a receiver-ordered sweep, dx by a
 * sender-ordered segment sum of per-edge partials kept in ws. */
e3_status e3_conv_bwd(const e3_plan* plan, const e3_graph* graph, const float* x, const float* vec,
                      const float* s, const float* dm, float* dx, float* dvec, float* ds, void* ws,
                      size_t ws_bytes, e3_stream stream);

/* float64 builds of the tensor product and the convolution: the operations,
 * layouts, index spaces and semantics of e3_tp_fwd / e3_tp_bwd / e3_conv_fwd /
 * e3_conv_bwd with every floating-point array (x, y, w, z, dz, dx, dy, dw, vec,
 * s, m, dm, ds, dvec) in float64 -- the precision App. D measures the float32
 * kernels against ("Precision").  The same generated per-edge code runs in
 * simpler kernels (one channel per lane); deterministic, atomics-free.
 * Workspaces: e3_tp_workspace_size_f64 / e3_conv_workspace_size_f64 bytes
 * (the x-cotangent and harmonic-cotangent partials, in float64).  Arrays with
 * a channel axis and ws must be 16-byte aligned. */
e3_status e3_tp_fwd_f64(const e3_plan* plan, const double* x, const double* y, const double* w, double* z,
                        int64_t rows, e3_stream stream);
e3_status e3_tp_workspace_size_f64(const e3_plan* plan, int64_t rows, size_t* bwd_bytes);
e3_status e3_tp_bwd_f64(const e3_plan* plan, const double* x, const double* y, const double* w, const double* dz,
                        double* dx, double* dy, double* dw, void* ws, size_t ws_bytes, int64_t rows,
                        e3_stream stream);
e3_status e3_conv_workspace_size_f64(const e3_plan* plan, const e3_graph* graph, size_t* bwd_bytes);
e3_status e3_conv_fwd_f64(const e3_plan* plan, const e3_graph* graph, const double* x, const double* vec,
                          const double* s, double* m, e3_stream stream);
e3_status e3_conv_bwd_f64(const e3_plan* plan, const e3_graph* graph, const double* x, const double* vec,
                          const double* s, const double* dm, double* dx, double* dvec, double* ds, void* ws,
                          size_t ws_bytes, e3_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): e3_conv_bwd
 * with its scratch -- the per-edge x-cotangent partials and the harmonic-
 * cotangent partials -- in a fixed array of the library instead of a caller
 * workspace.  Same arguments, outputs and results as e3_conv_bwd, bit for
 * bit.  The array holds E3_NOALLOC_SCRATCH_BYTES (64 MiB) on each device the
 * library runs on, kept until the process ends; a graph whose scratch
 * (e3_conv_workspace_size's bwd_bytes) exceeds it is refused with
 * E3_ERR_WORKSPACE_TOO_SMALL -- about 7,800 live edges with 16 feature rows
 * of 128 channels.  The call allocates nothing (its first call on a device
 * looks up that device's copy of the array once).  Every call on one device
 * shares that device's array, which keeps the last call's contents: calls that
 * overlap on one device (other streams, other threads) race, and the caller
 * must order them. */
#define E3_NOALLOC_SCRATCH_BYTES (64u << 20)
e3_status e3_conv_bwd_noalloc(const e3_plan* plan, const e3_graph* graph, const float* x, const float* vec,
                              const float* s, const float* dm, float* dx, float* dvec, float* ds, e3_stream stream);

/* The convolution with the harmonics y [E, D_sh] given by the caller instead of
 * computed from edge vectors: eq. message_passing_convolution and eq. conv-bwd
 * exactly as stated (y is an input of both, dy an output of the backward).
 * e3_conv_fwd_y:  m = conv(x, y, s).
 * e3_conv_bwd_y:  dx [n_nodes, D_in, C], dy [E, D_sh], ds [E, P, C]; any of the
 *   three may be NULL (not stored; dx == NULL also skips its segment sum).
 * accumulate != 0: results are added to the outputs' contents (padding edges'
 *   rows are then left unchanged) instead of overwriting them.
 * ws as for e3_conv_bwd. */
e3_status e3_conv_fwd_y(const e3_plan* plan, const e3_graph* graph, const float* x, const float* y,
                        const float* s, float* m, int accumulate, e3_stream stream);
e3_status e3_conv_bwd_y(const e3_plan* plan, const e3_graph* graph, const float* x, const float* y,
                        const float* s, const float* dm, float* dx, float* dy, float* ds, int accumulate,
                        void* ws, size_t ws_bytes, e3_stream stream);

/* Double backward of the convolution (eq. conv-bwd-bwd-ddm and eq.
 * conv-bwd2-xys): given the primals (x, y, s, dm) of a backward call and
 * variations (ddx [n_nodes, D_in, C], ddy [E, D_sh], dds [E, P, C]) of its
 * outputs, computes the variations of its inputs:
 *   gdm = conv(ddx, y, s) + conv(x, ddy, s) + conv(x, y, dds)      [n_nodes, D_out, C]
 *   gx  = dx of conv_bwd(x, ddy, s, dm) + dx of conv_bwd(x, y, dds, dm)
 *   gy  = dy of conv_bwd(ddx, y, s, dm) + dy of conv_bwd(x, y, dds, dm)
 *   gs  = ds of conv_bwd(ddx, y, s, dm) + ds of conv_bwd(x, ddy, s, dm)
 * gdm by one sweep that forms the three forward terms together, and gx, gy,
 * gs by one sweep that forms the three backward terms together (one channel
 * per lane; a build with more runs three backward sweeps that store only the
 * cotangents used and add in place).  The composed path runs both sweeps per
 * x block, the record path three forward and three backward calls.
 * Deterministic.  ws as for e3_conv_bwd. */
e3_status e3_conv_bwd2(const e3_plan* plan, const e3_graph* graph, const float* x, const float* y,
                       const float* s, const float* dm, const float* ddx, const float* ddy, const float* dds,
                       float* gx, float* gy, float* gs, float* gdm, void* ws, size_t ws_bytes, e3_stream stream);

/* Convolution with fused radial weights (eq. message-passing-linear, where the
 * edge scalars come from a radial embedding followed by an MLP; App. A.3).
 * The MLP's last linear layer is fused: with h [E, K] the per-edge features
 * entering it (the radial basis itself for a one-layer model) and W [K, P, C]
 * its weight, the kernels use s_e[k, q] = sum_j h[e, j] W[j, k, q], formed on
 * the matrix cores and never written to memory.  1 <= K <= 16.
 *
 * e3_conv_fwd_radial: m [n_nodes, D_out, C] as e3_conv_fwd with these s.
 * e3_conv_bwd_radial: from dm computes dx [n_nodes, D_in, C], dvec [E, 3]
 *   (through the harmonics only: the dependence of h on the edge length is the
 *   caller's), dh [E, K] = sum_{k,q} ds W and dW [K, P, C] = sum_e h_e ds_e,
 *   with ds of eq. conv-bwd.  Deterministic: dW is a fixed-order sum of
 *   fixed row-chunk partials.  Padding edges get dh = 0 and dvec = 0.
 *   ws: at least e3_conv_radial_workspace_size bytes (ds of the live edges,
 *   the partials of dW and dh, and the plain backward's scratch).
 * x, W, m, dx, dm and ws must be 16-byte aligned; h, dh, dW need 4. */
e3_status e3_conv_radial_workspace_size(const e3_plan* plan, const e3_graph* graph, int K, size_t* bwd_bytes);
e3_status e3_conv_fwd_radial(const e3_plan* plan, const e3_graph* graph, const float* x, const float* vec,
                             const float* h, const float* W, int K, float* m, e3_stream stream);
e3_status e3_conv_bwd_radial(const e3_plan* plan, const e3_graph* graph, const float* x, const float* vec,
                             const float* h, const float* W, int K, const float* dm, float* dx, float* dvec,
                             float* dh, float* dW, void* ws, size_t ws_bytes, e3_stream stream);

/* Equivariant linear mixing (App. A.3, linear mixing between features of the
 * same degree, with the weight shared over the 2l+1 components so that it
 * commutes with rotations).  An output block of type (l, p) receives every
 * input block of the same (l, p), in input order, multiplicities concatenated:
 *   out[n, o + m, j] = sum_t sum_k x[n, in_t + m, k] W_o[t * C_in + k, j].
 * An output type with no input is zero.  W is the concatenation over output
 * blocks, in order, of W_o [n_in(o) * C_in, C_out] row-major; e3_linear_query
 * gives its length.  irreps_in / irreps_out: irreps strings with one
 * multiplicity each (C_in, C_out multiples of 16; at most 64 blocks a side).
 * Layouts: x [n, D_in, C_in], out [n, D_out, C_out], both 16-byte aligned.
 * fp32 on the matrix cores.  e3_linear_create uploads the descriptor's small
 * block tables to the device current at creation (it allocates and waits for
 * the copy; E3_ERR_HIP if that fails); the compute calls then only launch
 * kernels, and return E3_ERR_INVALID_ARG when another device is current.
 * e3_linear_bwd: dx [n, D_in, C_in] and dW (same layout as W) from dout; dW is
 *   a fixed-order sum of fixed row-chunk partials kept in ws (at least
 *   e3_linear_workspace_size bytes), so it is deterministic. */
typedef struct e3_linear e3_linear;
e3_status e3_linear_create(const char* irreps_in, const char* irreps_out, e3_linear** out);
e3_status e3_linear_query(const e3_linear* lin, int64_t* n_weights, int* d_in, int* d_out, int* c_in, int* c_out);
e3_status e3_linear_destroy(e3_linear* lin);
e3_status e3_linear_fwd(e3_linear* lin, const float* x, const float* W, float* out, int64_t n, e3_stream stream);
e3_status e3_linear_workspace_size(const e3_linear* lin, size_t* bwd_bytes);
e3_status e3_linear_bwd(e3_linear* lin, const float* x, const float* W, const float* dout, float* dx, float* dW,
                        void* ws, size_t ws_bytes, int64_t n, e3_stream stream);

/* Tensor product with caller-supplied coefficient records (App. E.2's
 * unfolded COO form): z[r, i0, q] = sum over records (i0, i1, i2, v) of
 * v x[r, i1, q] y[r, i2, q] (y_per_channel != 0) or v x[r, i1, q] y[r, i2]
 * (y shared by the channels).  Any record set is allowed, e.g. several paths
 * sent to one output block (collapsed output multiplicities).  Layouts:
 * x [rows, d_x, C], y [rows, d_y, C] or [rows, d_y], z [rows, d_z, C]; any
 * C >= 1.  Records are copied at create (index errors: E3_ERR_INDEX_OUT_OF_RANGE);
 * operand rows must fit 64 KiB of staging per 64 channels (else
 * E3_ERR_UNSUPPORTED).  A wave stages up to four rows (as many as fit the
 * limit); an operand block of those rows, d C element bytes per row, must stay
 * under 2 GiB (else E3_ERR_INVALID_ARG).  e3_tpg_create uploads the tables
 * to the device current at creation (it allocates and waits for the copy);
 * the compute calls then only launch kernels, and return E3_ERR_INVALID_ARG
 * when another device is current.
 * e3_tpg_bwd (eq. tp-bwd): dx = tensor_product(C^{i1}_{i2 i0}, y, dz) and
 *   dy = tensor_product(C^{i2}_{i1 i0}, x, dz), summed over the channels when y
 *   is shared (then ws holds per-slab partials, e3_tpg_workspace_size bytes,
 *   enough for either precision).
 * Record values are given in float64; the _f64 entry points compute in float64
 * throughout (operand rows then fit half the staging limit), the others in
 * float32 with the values rounded once. */
typedef struct e3_tpg e3_tpg;
e3_status e3_tpg_create(int d_x, int d_y, int d_z, int64_t nnz, const int32_t* i0, const int32_t* i1,
                        const int32_t* i2, const double* val, int y_per_channel, e3_tpg** out);
e3_status e3_tpg_destroy(e3_tpg* tpg);
e3_status e3_tpg_fwd(e3_tpg* tpg, const float* x, const float* y, float* z, int64_t rows, int C, e3_stream stream);
e3_status e3_tpg_workspace_size(const e3_tpg* tpg, int64_t rows, int C, size_t* bwd_bytes);
e3_status e3_tpg_bwd(e3_tpg* tpg, const float* x, const float* y, const float* dz, float* dx, float* dy, void* ws,
                     size_t ws_bytes, int64_t rows, int C, e3_stream stream);
e3_status e3_tpg_fwd_f64(e3_tpg* tpg, const double* x, const double* y, double* z, int64_t rows, int C,
                         e3_stream stream);
e3_status e3_tpg_bwd_f64(e3_tpg* tpg, const double* x, const double* y, const double* dz, double* dx, double* dy,
                         void* ws, size_t ws_bytes, int64_t rows, int C, e3_stream stream);

/* Per-kernel timing (instrumentation).  While enabled, every kernel the
 * library launches is bracketed by two HIP events on the caller's stream.
 * e3_timing_read waits for the recorded events and returns, per kernel name
 * (32-byte NUL-padded slots in names[cap*32]), the summed duration in ms and
 * the number of launches since the last reset; *n is the number of names
 * (which may exceed cap).  Not thread-safe with respect to concurrent streams
 * of one process beyond the ordering of the calls. */
e3_status e3_timing_enable(int on);
e3_status e3_timing_reset(void);
e3_status e3_timing_read(int cap, char* names, double* ms, int64_t* count, int* n);

/* Streaming probe (instrumentation): measures what HBM sustains for a given
 * read:write mix, with the sweeps' own memory instructions -- buffer loads and
 * stores of `width` bytes per lane (4, 8 or 16) at a per-lane offset, with the
 * non-temporal bit on the loads (flags & E3_PROBE_NT_LOAD) and on the stores
 * (flags & E3_PROBE_NT_STORE).  Throughput is defined as in App. D (bytes
 * moved over run time).  Each step reads read_units and writes write_units
 * contiguous units of 64 x width bytes (0..16 each, not both 0), so the mix
 * is read_units:write_units; steps run until either buffer is exhausted.
 * src (read) and dst (written, contents undefined afterwards) are device
 * buffers of the caller, 16-byte aligned where used; *bytes_read and
 * *bytes_written receive the bytes one call moves.  Asynchronous on stream;
 * its launch is timed as "probe_stream" by e3_timing_*. */
#define E3_PROBE_NT_LOAD 1u
#define E3_PROBE_NT_STORE 2u
e3_status e3_probe_stream(const void* src, size_t src_bytes, void* dst, size_t dst_bytes, int read_units,
                          int write_units, int width, unsigned flags, size_t* bytes_read, size_t* bytes_written,
                          e3_stream stream);

const char* e3_status_str(e3_status s);
/* Text of the last HIP error seen by this thread (empty if none). */
const char* e3_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* E3MI_H */
