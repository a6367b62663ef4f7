/*
 * ggnn.h -- C ABI of the banded gated-GNN propagation library for AMD MI355X
 * (gfx950).
 *
 * The library implements one step of gated graph neural network propagation
 * (Balog et al., "Fast Training of Sparse Graph Neural Networks on Dense
 * Hardware", arXiv 1906.11786; Eq. 1 and its typed form) on a graph whose
 * nodes were reordered to low bandwidth (Compilation section, reverse
 * Cuthill-McKee) and whose per-edge-type adjacency A_e is stored as three
 * block diagonals of B x B blocks (Eq. 3, Algorithm 1).  A_e M is then three
 * batched dense block products, cost O(N B H) instead of O(N^2 H).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - An edge is (src j, dst i, type e): node i receives from node j, i.e.
 *    a_ij = 1 in the transposed adjacency matrix A_e (Background, Eq. 1).
 *  - All tensors are dense, contiguous, row-major, with no strides, and
 *    16-byte aligned.  Shapes are written outermost first.
 *  - Node-major tensors are [n_pad][F]; feature-major tensors are [F][n_pad]
 *    (feature f of node i at f * n_pad + i).
 *  - "dt" tensors hold the compute dtype: IEEE float32 (GGNN_F32) or bfloat16
 *    (GGNN_BF16, round-to-nearest-even on every store).  Accumulation is
 *    always float32.  Tensors documented as "float" are float32 for both.
 *  - Ownership: the caller allocates and frees everything.  The library never
 *    allocates or frees device memory, never synchronises a stream, and never
 *    keeps a pointer after a call returns.
 *  - Device entry points are asynchronous: every argument is validated on
 *    the host before anything is enqueued, then kernels are launched on
 *    `stream` (a hipStream_t; NULL is the null stream).  They issue no
 *    hipMemsetAsync and no allocation, so they can be captured into a HIP
 *    graph.  A launch error reported by hipGetLastError is GGNN_ERR_DEVICE.
 *  - Errors: a non-OK status leaves a message retrievable with
 *    ggnn_last_error() on the calling thread.  Nothing throws across the ABI.
 *  - Supported sizes for device work: B in {32, 64, 128, 256, 512},
 *    H in {32, 64, 128, 256}, 1 <= E <= 64, n_pad a positive multiple of B
 *    (and of 32 for the node-wise calls, which take no B).
 *  - Results are deterministic: no float atomics; cross-block reductions use a
 *    fixed partition and a fixed summation order.
 */
#ifndef GGNN_H
#define GGNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GGNN_ABI_VERSION 12

typedef enum {
  GGNN_OK = 0,
  GGNN_ERR_INVALID_ARG = 1,  /* bad size, NULL pointer, id out of range       */
  GGNN_ERR_UNSUPPORTED = 2,  /* valid arguments with no kernel for them       */
  GGNN_ERR_OUT_OF_BAND = 3,  /* strict packing met an edge outside the band   */
  GGNN_ERR_DEVICE = 4,       /* HIP launch or runtime error                   */
  GGNN_ERR_HOST_ALLOC = 5,   /* host-side temporary allocation failed         */
  GGNN_ERR_WORKSPACE = 6     /* workspace missing or smaller than required    */
} ggnn_status;

typedef enum { GGNN_F32 = 0, GGNN_BF16 = 1 } ggnn_dtype;

/* Storage of the block band: dense elements of the compute dtype, or one bit
 * per entry (lossless, since A_e has entries in {0,1}). */
typedef enum { GGNN_BAND_DENSE = 0, GGNN_BAND_BITS = 1 } ggnn_band_format;

/* Version of this ABI (GGNN_ABI_VERSION of the built library). */
int ggnn_abi_version(void);

/* Text of the last non-OK status raised on the calling thread ("" if none).
 * The pointer stays valid until the next library call on that thread. */
const char* ggnn_last_error(void);

/* Short fixed name of a status code. */
const char* ggnn_status_string(ggnn_status s);

/* ======================================================================
 * Host-side graph compilation (synchronous, host memory only)
 * ====================================================================== */

/* Reverse Cuthill-McKee node order (Compilation section: permute the nodes
 * to expose low bandwidth; the bandwidth is defined in the Background
 * section).  The graph is the union of all edge types, symmetrised, with
 * self-loops and repeated pairs ignored.  Components are taken in order of
 * their smallest label; each starts at a pseudo-peripheral node found by the
 * George-Liu iteration from its node of smallest (degree, label); the
 * breadth-first search appends unvisited neighbours by increasing
 * (degree, label); the whole sequence is reversed.
 *   n          number of nodes (>= 0); m number of edges (>= 0)
 *   src, dst   [m] node ids in [0, n)
 *   order      [n] out: order[p] = old label placed at new position p
 *   rank       [n] out: rank[v] = new position of old label v
 *   bandwidth  nullable out: max |rank[src] - rank[dst]| over the edges
 * Errors: INVALID_ARG for negative sizes, NULL arrays (when n or m > 0) or
 * ids out of range; HOST_ALLOC if temporaries cannot be allocated. */
ggnn_status ggnn_rcm_order(int32_t n, int64_t m, const int32_t* src, const int32_t* dst,
                           int32_t* order, int32_t* rank, int32_t* bandwidth);

/* Bandwidth of an edge list (Background: the smallest b with a_ij = 0 for
 * |i - j| > b) under an optional relabelling rank[v] (nullable: identity).
 *   n          number of nodes; src, dst [m] ids in [0, n); rank [n] with values in [0, n), or NULL
 *   bandwidth  out (0 for m == 0)
 * Errors: ids or rank values out of range, NULL pointers -> INVALID_ARG. */
ggnn_status ggnn_bandwidth(int32_t n, int64_t m, const int32_t* src, const int32_t* dst,
                           const int32_t* rank, int32_t* bandwidth);

/* Sparse batching (Background section: a batch of graphs is one graph whose
 * connected components are the batch's graphs): the graphs' nodes are placed
 * one after another, graph i at supergraph ids offsets[i] .. offsets[i+1]-1,
 * each graph's nodes first reordered with reverse Cuthill-McKee (exactly as
 * ggnn_rcm_order does for that graph alone) when reorder is 1, or kept in
 * their order when 0.  Edges keep their order (so per-edge arrays such as
 * the edge types carry over unchanged).
 *   n_graphs     number of graphs (>= 0)
 *   node_counts  [n_graphs] nodes of each graph (>= 0; at most 2^31 - 1 in all)
 *   edge_counts  [n_graphs] edges of each graph (>= 0)
 *   src, dst     [sum edge_counts] the graphs' edges one graph after another, ids local to their graph
 *   out_src, out_dst [sum edge_counts] out: the same edges in supergraph ids (may not alias src, dst)
 *   offsets      [n_graphs + 1] out: first supergraph id of each graph; offsets[n_graphs] = all nodes
 *   bandwidth    out: the largest bandwidth of a graph after the reordering (the supergraph's, as
 *                no edge joins two graphs)
 * Host memory only.  Errors: INVALID_ARG for negative counts, NULL arrays, too many nodes or ids out of
 * range (the message names the graph); HOST_ALLOC if temporaries cannot be allocated. */
ggnn_status ggnn_batch_graphs(int32_t n_graphs, const int32_t* node_counts, const int64_t* edge_counts,
                              const int32_t* src, const int32_t* dst, int32_t reorder, int32_t* out_src,
                              int32_t* out_dst, int64_t* offsets, int32_t* bandwidth);

/* The same batching with supernodes (Discussion section): the listed hub
 * nodes of every graph take the first labels, 0 .. (all hubs - 1) < s, graph
 * after graph in list order; each graph's other nodes are reordered with
 * reverse Cuthill-McKee on the edges between them (the band's share; as
 * ggnn_rcm_order on those nodes in their label order) and placed from
 * label s on, graph after graph.
 *   hub_counts   [n_graphs] hubs of each graph (0 .. node count)
 *   hubs         [sum hub_counts] each graph's hubs, ids local to the graph, distinct within it
 *   s            supernode slots (>= all hubs)
 *   n_nodes      out: s + the non-hub nodes of all graphs (the labels used)
 *   bandwidth    out: the largest bandwidth of a graph's non-hub part after the reordering
 *   the other arguments as ggnn_batch_graphs (no offsets: hubs and graphs interleave)
 * Host memory only.  Errors: INVALID_ARG for negative counts, NULL arrays, more hubs than s, repeated or
 * out-of-range hubs or ids (the message names the graph); HOST_ALLOC if temporaries cannot be allocated. */
ggnn_status ggnn_batch_graphs_super(int32_t n_graphs, const int32_t* node_counts, const int64_t* edge_counts,
                                    const int32_t* src, const int32_t* dst, const int32_t* hub_counts,
                                    const int32_t* hubs, int32_t s, int32_t* out_src, int32_t* out_dst,
                                    int32_t* n_nodes, int32_t* bandwidth);

/* Bytes of a block band: E * (n_pad / B) * 3 * B * B elements of dtype dt.
 * Returns 0 for invalid arguments. */
size_t ggnn_band_bytes(int32_t n_pad, int32_t E, int32_t B, ggnn_dtype dt);

/* Pack typed edges into the three block diagonals of Eq. 3 (Algorithm 1's
 * Cks, Uks, Lks), one band per edge type:
 *   band[e][k][s][r][c] = 1 for an edge j -> i of type e with
 *   i = rank(dst) = k*B + r and j = rank(src) = (k - 1 + s)*B + c,
 * so s = 0 is the sub-diagonal block L_k (block column k-1), s = 1 the
 * diagonal block C_k and s = 2 the super-diagonal block U_k (block column
 * k+1).  Slot (k = 0, s = 0) and slot (k = nb-1, s = 2) are always zero.
 * Edges whose block row and block column differ by more than one are not
 * covered (the lossy regime described after Eq. 3): they are dropped and
 * counted, or, with strict != 0, make the call fail with OUT_OF_BAND after
 * the whole list has been scanned.  A repeated (src, dst, type) is one edge
 * (A_e has entries in {0,1}) and is counted as a duplicate.
 *   n_pad      positive multiple of B (B >= 1 here; the device entry points
 *              need B in {32..512})
 *   src, dst   [m] ids in [0, n_pad); etype [m] in [0, E)
 *   rank       [n_pad] relabelling applied to src and dst, or NULL (identity)
 *   band       host buffer of ggnn_band_bytes(n_pad, E, B, dt) bytes; fully
 *              overwritten (zeros, then ones at the edges)
 *   n_packed, n_dropped, n_duplicate   nullable counters (out) */
ggnn_status ggnn_banded_pack(int32_t n_pad, int32_t E, int32_t B, int64_t m,
                             const int32_t* src, const int32_t* dst, const int32_t* etype,
                             const int32_t* rank, ggnn_dtype dt, int strict, void* band,
                             int64_t* n_packed, int64_t* n_dropped, int64_t* n_duplicate);

/* Bytes of a 1-bit block band: E * (n_pad / B) * 3 * B * (B / 8).
 * Returns 0 for invalid arguments (B must be a multiple of 8). */
size_t ggnn_band_bits_bytes(int32_t n_pad, int32_t E, int32_t B);

/* Pack typed edges into the three block diagonals of Eq. 3 at one bit per
 * entry, plus (optionally) the transposed blocks used by the reverse pass.
 *   bits[e][k][s][r][B/8]: row r of block (e, k, s) as in ggnn_banded_pack;
 *     byte c/8 of the row holds columns c..c+7, bit c%8 is column c.
 *   bits_t[e][j][s][c][B/8]: the transposed blocks with the sub- and
 *     super-diagonal roles swapped, bits_t[e][j][s] = band[e][j-1+s][2-s]^T:
 *     row c of block (e, j, s) holds bit r for every edge from node
 *     j*B + c to node (j-1+s)*B + r.  Nullable.
 * Coverage, duplicates, counters, strict and errors are as for
 * ggnn_banded_pack.  B must be a multiple of 8; both buffers hold
 * ggnn_band_bits_bytes(...) bytes and are fully overwritten. */
ggnn_status ggnn_banded_pack_bits(int32_t n_pad, int32_t E, int32_t B, int64_t m,
                                  const int32_t* src, const int32_t* dst, const int32_t* etype,
                                  const int32_t* rank, int strict, void* bits, void* bits_t,
                                  int64_t* n_packed, int64_t* n_dropped, int64_t* n_duplicate);

/* ======================================================================
 * Device entry points: one propagation step and its reverse.
 * All pointers are device memory owned by the caller.
 * ====================================================================== */

/* Message transform (typed form of Eq. 1; per-type bias of the Appendix's
 * "Model" paragraph): M_e = X W_e (+ 1 bias_e^T) for every edge type e.
 *   X     [n_pad][H] dt, node-major node states
 *   W     [E][H][H] dt, W[e][h_in][h_out]
 *   bias  [E][H] float, or NULL for no bias
 *   M     [E][H][n_pad] float, feature-major: M[e][h][i] (written).  The
 *         messages stay float in both modes: they are summed over many edges
 *         next, and a bf16 copy would add a rounding as large as that of
 *         the bf16 state itself. */
ggnn_status ggnn_msg_transform(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E,
                               const void* X, const void* W, const float* bias, float* M,
                               void* stream);

/* Banded propagation (Eq. 3; Algorithm 1's three batched products):
 *   a[k] = sum_e  band[e][k][0] M_e[k-1] + band[e][k][1] M_e[k] + band[e][k][2] M_e[k+1]
 * for every block row k (out-of-range blocks are zero), i.e. a = sum_e A_e M_e
 * on the covered edges, messages summed.  In bf16 mode each message enters
 * the matrix cores as a bf16 pair (hi + lo), so the products keep about 16
 * bits of the float message.
 *   band  [E][n_pad/B][3][B][B] dt (as ggnn_banded_pack writes it)
 *   M     [E][H][n_pad] float feature-major
 *   a     [n_pad][H] float node-major (written) */
ggnn_status ggnn_banded_propagate(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                  const void* band, const float* M, float* a, void* stream);

/* GRU node update (Eq. 1's GRU, Cho et al. 2014 form; gates (r, z, n)):
 *   r = sigmoid(a Wi_r + h U_r + b_r),  z = sigmoid(a Wi_z + h U_z + b_z)
 *   n = tanh(a Wi_n + (r*h) U_n + b_n), h_out = z*h + (1-z)*n
 * In bf16 mode a enters the matrix cores as a bf16 pair (hi + lo) and r*h
 * is rounded to bf16.
 *   a      [n_pad][H] float;  h [n_pad][H] dt
 *   Wi, U  [H][3H] dt (columns r | z | n);  b [3H] float
 *   h_out  [n_pad][H] dt (written; must not alias h)
 *   saved  [n_pad][3H] dt (written: r | z | n per node), or NULL */
ggnn_status ggnn_gru_update(ggnn_dtype dt, int32_t n_pad, int32_t H, const float* a, const void* h,
                            const void* Wi, const void* U, const float* b, void* h_out, void* saved,
                            void* stream);

/* Aggregate-first propagation step on a 1-bit band (Algorithm 1's operand
 * order; Eq. 3's three block products):
 *   a = sum_e (A_e X) W_e  (+ sum_e (A_e 1) bias_e^T when bias != NULL)
 * The aggregation A_e X and the transform by W_e run in one kernel; the
 * per-type aggregates never leave the chip (in bf16 mode they enter the
 * transform as bf16 hi + lo pairs).  Same result as ggnn_msg_transform
 * followed by ggnn_banded_propagate, without the messages in memory.
 *   bits  as written by ggnn_banded_pack_bits (16-byte aligned)
 *   X     [n_pad][H] dt node-major;  W [E][H][H] dt;  bias [E][H] float or NULL
 *   a     [n_pad][H] float (written) */
ggnn_status ggnn_banded_step_bits(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                  const void* bits, const void* X, const void* W, const float* bias,
                                  float* a, void* stream);

/* Reverse of the banded product on a 1-bit band: dM_e = A_e^T da, read
 * through the transposed blocks (bits_t of ggnn_banded_pack_bits).
 *   da [H][n_pad] dt feature-major;  dM [E][H][n_pad] dt feature-major (written) */
ggnn_status ggnn_banded_propagate_bits_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                           const void* bits_t, const void* da, void* dM, void* stream);

/* Reverse of ggnn_banded_step_bits in the same fused form (Algorithm 1's
 * operand order run backwards), per edge type e:
 *   dM_e = A_e^T da                      (through bits_t; stored, rounded to dt)
 *   dX_out = dX_in + sum_e dM_e W_e^T    (dM_e enters as the stored value)
 *   bits_t  transposed bit band of ggnn_banded_pack_bits (16-byte aligned)
 *   da      [H][n_pad] dt feature-major;  W [E][H][H] dt
 *   dX_in   [n_pad][H] float or NULL (zero); dX_out [n_pad][H] float (written;
 *           may be the same buffer as dX_in)
 *   dM      node-major, dt: row r (< n_pad) of type e at dM + (e * ldm + r) * H;
 *           ldm >= n_pad rows per type (written) */
ggnn_status ggnn_banded_step_bits_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                      const void* bits_t, const void* da, const void* W, const float* dX_in,
                                      float* dX_out, void* dM, int64_t ldm, void* stream);

/* One forward step of Eq. 1 on a 1-bit band: ggnn_banded_step_bits followed
 * by ggnn_gru_update on its result, run as one kernel where the shape allows
 * (small grids, H <= 64), as two otherwise.  Same arguments and layouts as
 * those two calls:
 *   a      [n_pad][H] float (written: the aggregate, kept for the reverse pass)
 *   h_out  [n_pad][H] dt (written: the next state);  saved [n_pad][3H] dt (r | z | n)
 * Wi, U [H][3H] dt; b [3H] float.  X and h_out must not share a byte (INVALID_ARG otherwise: workgroups
 * read the neighbour rows of X that others' rows of h_out would overwrite).  Wt: W_e^T
 * (ggnn_transpose_weights) or NULL; the result does not depend on it. */
ggnn_status ggnn_step_bits_gru(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                               const void* bits, const void* X, const void* W, const void* Wt,
                               const float* bias, const void* Wi, const void* U, const float* b, float* a,
                               void* h_out, void* saved, void* stream);

/* W_e^T for every edge type: Wt[e][o][h] = W[e][h][o] (both [E][H][H] dt, 16-byte aligned, not
 * overlapping).  The transposed weights are an optional operand of the forward steps (Wt of
 * ggnn_step_bits_gru and of ggnn_model). */
ggnn_status ggnn_transpose_weights(ggnn_dtype dt, int32_t H, int32_t E, const void* W, void* Wt, void* stream);

/* GRU weights repacked for the large-width GRU kernels (bf16, H = 128 or 256):
 * those kernels stream Wi and U through on-chip memory in stages, and the
 * packed copy holds every stage's 16-byte pieces in the order they are
 * staged, so staging becomes contiguous loads.  The packing is a pure
 * reordering of the elements of Wi and U (the GRU of Eq. 1 is unchanged):
 * results with and without it are bitwise identical.  An optional operand of
 * ggnn_model (gru_packed).
 * ggnn_gru_pack_bytes: bytes of the packed copy, 12 H^2 elements of dt; 0 where
 *   no kernel reads it (float32, or H < 128), and then ggnn_gru_pack_weights
 *   does nothing and `packed` may be NULL.
 * ggnn_gru_pack_weights: Wi, U [H][3H] dt (device); packed: device memory of
 *   ggnn_gru_pack_bytes bytes, 16-byte aligned, overlapping neither. */
size_t ggnn_gru_pack_bytes(ggnn_dtype dt, int32_t H);
ggnn_status ggnn_gru_pack_weights(ggnn_dtype dt, int32_t H, const void* Wi, const void* U, void* packed,
                                  void* stream);

/* One reverse step on a 1-bit band, the form ggnn_backward runs for t > 0:
 * the reverse of step t's propagation (ggnn_banded_step_bits_bwd: dM_e =
 * A_e^T da and g = dX_in + sum_e dM_e W_e^T), then the reverse of step t-1's
 * GRU update with g as the gradient of its output (ggnn_gru_update_bwd's
 * node part), one kernel where the shape allows.  g itself is not stored.
 *   da, W, dX_in, dM, ldm    as for ggnn_banded_step_bits_bwd
 *   h_prev [n_pad][H] dt (X_{t-1});  saved_prev [n_pad][3H] dt (gates of step t-1)
 *   da_prev [H][n_pad] dt feature-major (written; must not alias da)
 *   dh_prev [n_pad][H] float (written);  ghat_prev [n_pad][3H] dt (written: the
 *           gate pre-activation gradients r^ | z^ | n^ of step t-1, the factor of the
 *           GRU weight gradients) */
ggnn_status ggnn_step_bits_gru_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                   const void* bits_t, const void* da, const void* W, const float* dX_in,
                                   void* dM, int64_t ldm, const void* Wi, const void* U, const void* h_prev,
                                   const void* saved_prev, void* da_prev, float* dh_prev, void* ghat_prev,
                                   void* stream);

/* Workspace bytes needed by ggnn_gru_update_bwd for these sizes. */
size_t ggnn_gru_update_bwd_workspace_bytes(ggnn_dtype dt, int32_t n_pad, int32_t H);

/* Reverse of ggnn_gru_update for the upstream gradient dh_out of h_out:
 *   da   [H][n_pad] dt, feature-major (written)     = dL/da
 *   dh   [n_pad][H] float (written)                   = dL/dh through the GRU
 *   dWi, dU [H][3H] float, db [3H] float: += (the caller zeroes them once;
 *         weights are shared across steps)
 *   workspace  device buffer of at least the queried size; its contents
 *         on entry do not matter
 *   a, h, saved as passed to / written by the forward call. */
ggnn_status ggnn_gru_update_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, const float* dh_out,
                                const float* a, const void* h, const void* saved,
                                const void* Wi, const void* U,
                                void* da, float* dh, float* dWi, float* dU, float* db,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Reverse of ggnn_banded_propagate: dM_e = A_e^T da on the covered edges,
 * evaluated with transposed blocks and the sub/super-diagonal roles swapped:
 *   dM_e[c] = band[e][c-1][2]^T da[c-1] + band[e][c][1]^T da[c] + band[e][c+1][0]^T da[c+1]
 *   band  as for the forward; da [H][n_pad] dt feature-major
 *   dM    [E][H][n_pad] dt feature-major (written) */
ggnn_status ggnn_banded_propagate_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                      const void* band, const void* da, void* dM, void* stream);

/* Workspace bytes needed by ggnn_msg_transform_bwd for these sizes. */
size_t ggnn_msg_transform_bwd_workspace_bytes(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E);

/* Reverse of ggnn_msg_transform:
 *   dX_out = dX_in + sum_e dM_e W_e^T   ([n_pad][H] float; dX_in may be NULL
 *            for zero, and may equal dX_out for an in-place update)
 *   dW    [E][H][H] float  += X^T dM_e
 *   dbias [E][H] float     += column sums of dM_e, or NULL to skip
 *   X     [n_pad][H] dt;  W [E][H][H] dt;  dM [E][H][n_pad] dt */
ggnn_status ggnn_msg_transform_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E,
                                   const void* X, const void* W, const void* dM,
                                   const float* dX_in, float* dX_out, float* dW, float* dbias,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* ======================================================================
 * T-step orchestration (Eq. 1 for t = 0..T-1, with stored activations, and
 * the reverse pass).  Each call enqueues 3*T (forward) or 3*T plus a few
 * reduction launches (backward) kernels on `stream`.
 * ====================================================================== */

typedef struct ggnn_model {
  int32_t dtype;        /* ggnn_dtype */
  int32_t n_pad, B, H, E, T;
  const void* band;     /* dense: [E][n_pad/B][3][B][B] dt; bits: bits of ggnn_banded_pack_bits */
  const void* W;        /* [E][H][H] dt */
  const float* bias;    /* [E][H] or NULL */
  const void* Wi;       /* [H][3H] dt */
  const void* U;        /* [H][3H] dt */
  const float* b;       /* [3H] */
  int32_t band_format;  /* ggnn_band_format */
  const void* band_t;   /* bits: the transposed bit band (bits_t); dense: unused */
  const void* Wt;       /* [E][H][H] dt, W_e^T (Wt[e][o][h] = W[e][h][o], ggnn_transpose_weights), or NULL.
                           Optional: lets the bit-band forward read its weight fragments as rows; the
                           caller refreshes it whenever W changes. */
  const void* gru_packed; /* Wi, U as ggnn_gru_pack_weights lays them out, or NULL (optional, used where
                             ggnn_gru_pack_bytes > 0; the caller refreshes it whenever Wi or U change). */
  /* Supernodes next to the band (Discussion section; optional, bit band only): n_super = 0 for none.
   * Otherwise nodes 0 .. n_super-1 are supernode slots and the four slices of ggnn_super_pack hold every
   * edge that touches one (the band holds the others).  n_super_active: 0 when the slices hold no edge,
   * else a multiple of 16, at most n_super, with no slice edge at a supernode index at or above it
   * (ggnn_super_active computes it from the packed slices); the slices' rows and columns at or beyond it
   * are never read.  super_ws: device scratch of ggnn_super_model_workspace_bytes(model) bytes, 16-byte
   * aligned, used by ggnn_forward and ggnn_backward (neither keeps anything in it between calls). */
  int32_t n_super, n_super_active;
  const void* super_rows;    /* [E][n_super][n_pad/8] */
  const void* super_cols;    /* [E][n_pad][n_super/8] */
  const void* super_rows_t;  /* [E][n_pad][n_super/8] */
  const void* super_cols_t;  /* [E][n_super][n_pad/8] */
  void* super_ws;
  size_t super_ws_bytes;
} ggnn_model;

typedef struct ggnn_activations {
  void* X;              /* [T+1][n_pad][H] dt: X[0] is the input, X[1..T] written */
  float* a;             /* [T][n_pad][H] float, written by the forward */
  void* saved;          /* [T][n_pad][3H] dt, written by the forward */
  float* M;             /* [E][H][n_pad] float scratch for the dense band (NULL allowed with bits) */
} ggnn_activations;

typedef struct ggnn_grads {
  float* dX;            /* [n_pad][H]: on entry dL/dX_T, on return dL/dX_0 */
  float* dW;            /* [E][H][H]  += */
  float* dbias;         /* [E][H]     += (ignored when the model has no bias) */
  float* dWi;           /* [H][3H]    += */
  float* dU;            /* [H][3H]    += */
  float* db;            /* [3H]       += */
  void* da;             /* [H][n_pad] dt scratch */
  void* dM;             /* E*H*T*n_pad dt scratch: every step's message gradient.  Dense band:
                         * feature-major [E][H][T*n_pad], step t in columns [t*n_pad, (t+1)*n_pad)
                         * of every (e, h) row.  Bit band: node-major [E][T*n_pad][H], step t in
                         * rows [t*n_pad, (t+1)*n_pad) of every type. */
  float* dh;            /* [n_pad][H] float scratch */
  void* workspace;      /* device scratch of ggnn_backward_workspace_bytes() */
  size_t workspace_bytes;
} ggnn_grads;

/* Workspace bytes needed by ggnn_backward for this model. */
size_t ggnn_backward_workspace_bytes(const ggnn_model* model);

/* Workspace bytes of the supernode slices for this model (model->super_ws); 0 without supernodes. */
size_t ggnn_super_model_workspace_bytes(const ggnn_model* model);

/* Forward over T steps: for t = 0..T-1,
 *   dense band: M = msg_transform(X[t]); a[t] = banded_propagate(M);
 *   bit band:   a[t] = banded_step_bits(X[t]);
 *   with supernodes (bit band): a[t] += the slices' share (ggnn_super_propagate);
 *   then X[t+1], saved[t] = gru_update(a[t], X[t]).
 * With supernodes, in bf16 at H <= 64 with n_super_active <= 32 and a grid small enough for the
 * two-group fused steps (ggnn_super_fusable), the slices run inside the fused step kernels: the
 * column slice as a fourth block next to the three of Eq. 3 (the 32 supernodes' states staged once per
 * workgroup), and the supernode rows' aggregate R_e X from one launch per step before it (a gather of
 * the node states each slice row lists); otherwise the slice kernels of ggnn_super_propagate run between
 * the band step and the GRU. */
ggnn_status ggnn_forward(const ggnn_model* model, const ggnn_activations* act, void* stream);

/* Reverse pass for L with dL/dX_T given in grads->dX: for t = T-1..0,
 *   da, dh, G^_t = gru_update_bwd node pass(dX);
 *   with supernodes: the slices' reverse (fused as in ggnn_forward: the transposed row slice as a fourth
 *   block, the supernode rows' message gradients C_e^T da from one launch per step before it (the
 *   listed rows of the step's gate gradients G^ summed, then times Wi^T: da = G^ Wi^T row by row), all
 *   of it in dM; otherwise ggnn_super_propagate_bwd adds its share to dh, dW and dbias first);
 *   dense band: dM_t = banded_propagate_bwd(da); dX = dh + sum_e dM_t,e W_e^T;
 *   bit band:   dM_t, dX = banded_step_bits_bwd(da, dX_in = dh) (one kernel);
 * then the weight gradients as single contractions over all T * n_pad rows:
 *   dWi, dU, db += sums over t of the GRU products of (a[t], X[t], saved[t], G^_t),
 *   dW_e += sum_t X[t]^T dM_t,e, dbias_e += row sums of dM_t,e (accumulate, +=).
 * G^_t is kept in the workspace, dM_t in grads->dM.
 * Needs the activations of a preceding ggnn_forward. */
ggnn_status ggnn_backward(const ggnn_model* model, const ggnn_activations* act,
                          const ggnn_grads* grads, void* stream);

/* ---- Launch profiler (device time of every kernel of a real pass) --------
 *
 * While enabled, ggnn_forward and ggnn_backward bracket each kernel launch
 * they enqueue with two HIP events on the launch's stream and tag the pair
 * with the launch kind (ggnn_profile_name: "step_fwd", "step_fwd_gru",
 * "gru_fwd", "transform_fwd", "banded_fwd", "gru_rev", "step_rev",
 * "step_rev_gru", "banded_rev", "transform_rev_dx", "wgrad_gru",
 * "wgrad_transform", "reduce", "super_record" (the supernode rows' record of a fused supernode
 * step: their per-type sums over all nodes), "super" (the stand-alone slice kernels of one step's share);
 * the "_gru" forms are band steps with the GRU
 * or GRU reverse fused into the same kernel).  Launches made while the stream
 * is being captured into a HIP graph, and launches beyond `capacity`, are not
 * recorded.  The state is process-wide and meant for one driving host thread;
 * the events are host-side objects (no device memory is allocated).
 *
 * ggnn_profile_start(capacity): releases earlier records, creates `capacity`
 *   event pairs and enables recording (capacity 0: release and disable).
 *   Errors: capacity outside [0, 2^20] -> INVALID_ARG; event creation
 *   failure -> DEVICE.
 * ggnn_profile_stop(): disables recording; the records stay readable.
 * ggnn_profile_count(): records taken since the last start.
 * ggnn_profile_read(i, &id, &ms): waits for record i's stop event and returns
 *   its launch kind and elapsed device time in milliseconds.  Errors: i out
 *   of range or NULL outputs -> INVALID_ARG; HIP error -> DEVICE.
 * ggnn_profile_name(id): name of a launch kind ("" when out of range). */
ggnn_status ggnn_profile_start(int32_t capacity);
ggnn_status ggnn_profile_stop(void);
int32_t ggnn_profile_count(void);
ggnn_status ggnn_profile_read(int32_t i, int32_t* id, float* ms);
const char* ggnn_profile_name(int32_t id);

/* ---- Closing one training step: readout, loss, parameter update ----------
 *
 * Readout and loss (Background, "Variable misuse"): a learned linear map
 * R^H -> R applied to the final embedding of each candidate node gives its
 * logit; a softmax over each graph's candidates gives the probability of
 * each filling the hole, and the loss is the cross-entropy of the correct
 * candidate, averaged over the graphs of the supergraph:
 *   logits[c] = X[cand_node[c]] . w_out + b_out
 *   loss[g]   = log sum_{c in g} exp(logits[c]) - logits[cand_ptr[g] + target[g]]
 *   dlogit[c] = (softmax_g(logits)[c] - [c is the target of g]) / n_graphs
 * Candidate lists: graph g owns candidates cand_ptr[g] .. cand_ptr[g+1]-1
 * (cand_ptr [n_graphs + 1] int32, non-decreasing, cand_ptr[n_graphs] =
 * n_cand), candidate c is node cand_node[c] ([n_cand] int32, < n_pad),
 * target[g] ([n_graphs] int32) indexes the graph's own list.  A graph without
 * candidates gets loss 0; a target outside the graph's list gives loss NaN.
 * All of these arrays are device memory.
 *   X [n_pad][H] dt (the final states X_T);  w_out [H] float;  b_out [1] float
 *   logits, dlogit [n_cand] float (written);  loss [n_graphs] float (written) */
ggnn_status ggnn_readout_loss(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t n_graphs, int32_t n_cand,
                              const void* X, const float* w_out, const float* b_out, const int32_t* cand_node,
                              const int32_t* cand_ptr, const int32_t* target, float* logits, float* loss,
                              float* dlogit, void* stream);

/* Workspace bytes of ggnn_readout_loss_bwd (0 for unsupported sizes). */
size_t ggnn_readout_loss_bwd_workspace_bytes(int32_t H, int32_t n_cand);

/* Reverse of the readout for the upstream gradients dlogit (of
 * ggnn_readout_loss):
 *   dX [n_pad][H] float (written whole: dlogit[c] * w_out on the row of each
 *      candidate, zero elsewhere) -- the dL/dX_T that ggnn_backward takes
 *   dw_out [H] float += sum_c dlogit[c] X[cand_node[c]];  db_out [1] float += sum_c dlogit[c]
 * A node may be the candidate of at most one graph, once (otherwise its dX
 * row holds one of the contributions).  workspace: 16-byte aligned, at least
 * ggnn_readout_loss_bwd_workspace_bytes(H, n_cand) bytes (per-block partial
 * sums, reduced in a fixed order). */
ggnn_status ggnn_readout_loss_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t n_cand, const void* X,
                                  const float* w_out, const int32_t* cand_node, const float* dlogit, float* dX,
                                  float* dw_out, float* db_out, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Bytes of the device array ggnn_readout_loss_bwd_noalloc keeps its partial
 * sums in (one per device, held until the process ends). */
#define GGNN_NOALLOC_SCRATCH_BYTES (4u << 20)

/* ggnn_readout_loss_bwd without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight
 * training or serving loops, harnesses that forbid hipMalloc): the per-block
 * partial sums go to a scratch array of GGNN_NOALLOC_SCRATCH_BYTES that the
 * library holds on each device.  Same arguments, results and determinism as
 * ggnn_readout_loss_bwd (bitwise equal outputs); the call allocates nothing.
 * Every partial is written before it is read, so no state carries over
 * between calls, but all calls on one device share the array: calls that
 * overlap on a device (concurrent streams or threads) race and must be
 * serialised by the caller.  The first call on a device looks up the array's
 * address there (host side; the stream's device is used).
 * Errors: as ggnn_readout_loss_bwd; partial sums larger than the scratch
 * (ggnn_readout_loss_bwd_workspace_bytes(H, n_cand) >
 * GGNN_NOALLOC_SCRATCH_BYTES: above 261,120 candidates at H = 256, 1,032,384
 * at H = 64) -> GGNN_ERR_UNSUPPORTED, checked before anything is enqueued. */
ggnn_status ggnn_readout_loss_bwd_noalloc(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t n_cand, const void* X,
                                          const float* w_out, const int32_t* cand_node, const float* dlogit,
                                          float* dX, float* dw_out, float* db_out, void* stream);

/* One Momentum-optimizer step (Appendix, "Optimization": Momentum, with
 * Nesterov momentum and L2 weight decay as options) on count float32 master
 * parameters, element-wise:
 *   g = grad + weight_decay * param;  velocity = momentum * velocity + g;
 *   param -= lr * (nesterov ? g + momentum * velocity : velocity)
 * param, velocity [count] float (updated in place); grad [count] float.
 * param_copy: NULL, or a [count] tensor of copy_dtype rewritten from the new
 * param (round to nearest even for bf16) -- the compute copy that the
 * propagation reads.  The four buffers must not overlap.  momentum and
 * weight_decay must be >= 0; all three scalars finite. */
ggnn_status ggnn_sgd_momentum(int64_t count, float* param, float* velocity, const float* grad, float lr,
                              float momentum, float weight_decay, int32_t nesterov, ggnn_dtype copy_dtype,
                              void* param_copy, void* stream);

/* ---- Evaluation on every edge (the lossy regime) --------------------------
 *
 * A model trained on the block band with B smaller than some graphs'
 * bandwidth drops their out-of-band edges (the coverage remark after Eq. 3);
 * its parameters are those of the sparse model, which evaluates with
 * messages passed along all edges (Experiments, "Training time to validation
 * accuracy").  These two calls are that sparse evaluation path.
 *
 * Host, synchronous: receiver-major lists of all edges, deduplicated (A_e has
 * entries in {0, 1}).  Row r = i * E + e lists the senders j of edges
 * j -> i of type e, ascending: col[row_ptr[r] .. row_ptr[r+1]-1].
 *   src, dst, etype [m] int32 (nodes < n_pad, types < E);
 *   row_ptr [n_pad * E + 1] int32 (written);  col [m] int32 (first *nnz written)
 *   *nnz = distinct edges; *n_duplicate = m - *nnz (either may be NULL). */
ggnn_status ggnn_sparse_csr(int32_t n_pad, int32_t E, int64_t m, const int32_t* src, const int32_t* dst,
                            const int32_t* etype, int32_t* row_ptr, int32_t* col, int64_t* nnz,
                            int64_t* n_duplicate);

/* Device: one propagation step's aggregate over every listed edge, in the
 * operand order of Algorithm 1:
 *   a[i] = sum_e ( sum_{j in col[row i*E+e]} X[j] ) W_e  (+ deg_e(i) bias_e)
 * row_ptr, col: ggnn_sparse_csr output copied to the device (nnz entries of
 * col; every col value < n_pad -- device data is not checked);
 * X [n_pad][H] dt; Wt [E][H][H] dt = W_e^T (ggnn_transpose_weights);
 * bias [E][H] float or NULL; a [n_pad][H] float (written).  The GRU update
 * of ggnn_gru_update then completes the step. */
ggnn_status ggnn_sparse_step(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, const int32_t* row_ptr,
                             const int32_t* col, int64_t nnz, const void* X, const void* Wt, const float* bias,
                             float* a, void* stream);

/* ---- Supernodes: dense slices of the first rows and columns ---------------
 *
 * A second runtime primitive next to the band (Discussion section: nodes that
 * communicate with all nodes, through dense slices of the first rows and
 * columns of the adjacency matrix).  The supernodes are nodes 0 .. s-1
 * (s in {32, 64, 96, 128}; n_pad a multiple of 64).  Per edge type e, 1 bit
 * per entry:
 *   rows   [E][s][n_pad/8]:  edges j -> i with i < s   (row i, byte j/8, bit j%8)
 *   cols   [E][n_pad][s/8]:  edges j -> i with i >= s, j < s
 *   rows_t [E][n_pad][s/8]:  rows transposed (row j, bit i);  cols_t [E][s][n_pad/8]: cols transposed
 * Every other edge (both ends >= s) belongs to the block band.
 *
 * Host, synchronous: sizes in bytes of one slice (0 for unsupported sizes),
 * and the packing of an edge list (rows_t, cols_t may be NULL).  n_rows /
 * n_cols count the distinct edges packed into each slice, n_rest the edges
 * left to the band, n_duplicate the repeats (any count pointer may be NULL). */
size_t ggnn_super_bytes(int32_t n_pad, int32_t E, int32_t s);
ggnn_status ggnn_super_pack(int32_t n_pad, int32_t E, int32_t s, int64_t m, const int32_t* src, const int32_t* dst,
                            const int32_t* etype, void* rows, void* cols, void* rows_t, void* cols_t,
                            int64_t* n_rows, int64_t* n_cols, int64_t* n_rest, int64_t* n_duplicate);

/* Workspace bytes of the two device calls below (0 for unsupported sizes). */
size_t ggnn_super_workspace_bytes(int32_t n_pad, int32_t H, int32_t E, int32_t s);

/* Host: the smallest multiple of 16 above every supernode index that has an edge in the slices (0 when
 * they hold none): rows i of rows [E][s][n_pad/8] with a bit set, columns j of cols [E][n_pad][s/8] with
 * a bit set.  Returns -1 (message via ggnn_last_error) for a NULL slice or unsupported sizes. */
int32_t ggnn_super_active(int32_t n_pad, int32_t E, int32_t s, const void* rows, const void* cols);

/* Whether ggnn_forward / ggnn_backward run the slices inside the fused step kernels for this shape
 * (bf16, H <= 64, two-group fused forms at this n_pad, B; and n_super_active = 16 or 32). */
int32_t ggnn_super_fusable(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E, int32_t n_super_active);

/* Device: the slices' share of one propagation step, added onto a (the
 * band's aggregate, e.g. from ggnn_banded_step_bits), with M_e = X W_e + b_e:
 *   a[i] += sum_e sum_j R_e[i][j] M_e[j]      (i < s; computed as (R_e X) W_e + deg b_e)
 *   a[i] += sum_e sum_{j<s} C_e[i][j] M_e[j]  (all i; M_e of the s supernodes)
 * X [n_pad][H] dt;  W [E][H][H] dt;  bias [E][H] float or NULL;  a [n_pad][H] float (+=).
 * ggnn_gru_update then completes the step. */
ggnn_status ggnn_super_propagate(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, int32_t s, const void* rows,
                                 const void* cols, const void* X, const void* W, const float* bias, float* a,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Device: reverse of ggnn_super_propagate for the upstream gradient da of a:
 * with dM_e = S_e^T da (S_e = the two slices),
 *   dX += sum_e dM_e W_e^T;  dW_e += X^T dM_e;  dbias_e += column sums of dM_e (dbias may be NULL)
 * da [H][n_pad] dt feature-major (as ggnn_gru_update_bwd writes it);
 * dX [n_pad][H] float, dW [E][H][H] float, dbias [E][H] float: accumulated. */
ggnn_status ggnn_super_propagate_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, int32_t s,
                                     const void* rows, const void* rows_t, const void* cols_t, const void* X,
                                     const void* W, const void* da, float* dX, float* dW, float* dbias,
                                     void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GGNN_H */
