// Launchers of the gfx950 kernels, one per device operation.  Arguments are
// validated by the C-ABI layer before these are called; each returns the
// hipGetLastError() of its launches.
//
// Every kernel source is built twice, once per storage dtype (bf16 kernels
// with matrix-core results kept in VGPRs, fp32 kernels with the compiler's
// default register assignment); the launchers of each build live in
// ggnn::impl_bf16 / ggnn::impl_f32, and the functions below pick one by dt.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

#include "../../include/ggnn.h"

namespace ggnn {

// Partial-sum reductions that a caller can collect and launch together
// (launch_reduce_multi): out[i] += sum_{s < nsplit} part[s * stride + i].
struct ReduceSeg {
  const float* part;
  float* out;
  int nsplit, count;
  long stride;
};
struct ReduceList {
  static constexpr int kMax = 8;
  ReduceSeg seg[kMax];
  int n = 0;
};
hipError_t launch_reduce_multi(const ReduceList& l, hipStream_t st);
// Appends to *defer (when non-NULL and not full), else launches the reduction.
// Message-transform weight gradient at H = 256 in bf16 with node-major dM
// (csrc/wgrad_wide.hip): per-split partials P [nsplit][E][256][256] and, when
// Pb is not NULL, Pb [nsplit][E][256]; splits of rows_per_split rows.
hipError_t launch_transform_wgrad_nm256(int nsplit, int rows_per_split, long K, int E, const void* X, const void* dM,
                                        long ldk, float* P, float* Pb, hipStream_t st);
// GRU weight gradients at H = 256 in bf16 (csrc/wgrad_wide.hip): partials
// P [nsplit][2][256][768] (dWi, dU) and Pb [nsplit][768]; splits of
// rows_per_split rows (a multiple of 32, as K); prog: nsplit x 8 ints of
// pacing counters (any contents; NULL turns pacing off).
hipError_t launch_gru_wgrad256(int nsplit, int rows_per_split, long K, const float* a, const void* h,
                               const void* saved, const void* ghat, float* P, float* Pb, int* prog, hipStream_t st);
hipError_t reduce_or_defer(const float* part, float* out, int nsplit, int count, long stride, ReduceList* defer,
                           hipStream_t st);

// Supernode share of a fused bit-band step (the first 32 nodes are
// supernodes): the slice bits of the step's direction, [E][n_pad][s/8] (the
// column slice forward, the transposed row slice reverse), and the record
// [P_e (sr x H) | deg_e (sr)], the sums over all nodes that give the first sr
// supernode rows their per-type aggregate (launch_super_long_fused forward,
// launch_super_gather_rev or launch_super_long_fused reverse).
struct SnStep {
  const void* bits;
  const float* rec;
  int s;
  int sr;   // record rows: the supernodes with edges are among the first sr (16 or 32)
};

#define GGNN_DT_LAUNCHERS                                                                                         \
  hipError_t launch_banded_fwd(int n_pad, int B, int H, int E, const void* band, const float* M, float* a,        \
                               hipStream_t st);                                                                   \
  hipError_t launch_banded_bwd(int n_pad, int B, int H, int E, const void* band, const void* da, void* dM,        \
                               long ldm, hipStream_t st);                                                         \
  hipError_t launch_step_fwd_bits(int n_pad, int B, int H, int E, const void* bits, const void* X, const void* W, \
                                  const float* bias, float* a, hipStream_t st);                                   \
  hipError_t launch_banded_bwd_bits(int n_pad, int B, int H, int E, const void* bits_t, const void* da, void* dM, \
                                    long ldm, hipStream_t st);                                                    \
  hipError_t launch_step_fwd_bits_gru(int n_pad, int B, int H, int E, const void* bits, const void* X,           \
                                      const void* W, const void* Wt, const float* bias, float* a, const void* Wi, \
                                      const void* U, const float* bg, void* h_out, void* saved, bool* fused,      \
                                      hipStream_t st);                                                            \
  hipError_t launch_transpose_weights(int H, int E, const void* W, void* Wt, hipStream_t st);                    \
  hipError_t launch_step_bwd_bits_gru(int n_pad, int B, int H, int E, const void* bits_t, const void* da,         \
                                      const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,       \
                                      const void* Wi, const void* U, const void* h_prev, const void* saved_prev,  \
                                      void* da_prev, float* dh_prev, void* ghat_prev, bool* fused,                \
                                      hipStream_t st);                                                            \
  hipError_t launch_step_bwd_bits(int n_pad, int B, int H, int E, const void* bits_t, const void* da,             \
                                  const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,           \
                                  hipStream_t st);                                                                \
  hipError_t launch_transform_fwd(int n_pad, int H, int E, const void* X, const void* W, const float* bias,       \
                                  float* M, hipStream_t st);                                                      \
  hipError_t launch_transform_bwd_dx(int n_pad, int H, int E, const void* W, const void* dM, long ld,             \
                                     const float* dX_in, float* dX_out, hipStream_t st);                          \
  hipError_t launch_transform_wgrad(long K, int H, int E, const void* X, const void* dM, long ld, float* dW,      \
                                    float* dbias, void* ws, hipStream_t st);                                      \
  hipError_t launch_transform_wgrad_nm(long K, int H, int E, const void* X, const void* dM, long ldk, float* dW,  \
                                       float* dbias, void* ws, ReduceList* defer, hipStream_t st);                \
  hipError_t launch_gru_fwd(int n_pad, int H, const float* a, const void* h, const void* Wi, const void* U,       \
                            const float* b, void* h_out, void* saved, const void* packed, hipStream_t st);        \
  hipError_t launch_gru_bwd_nodes(int n_pad, int H, const float* dh_out, const void* h, const void* saved,        \
                                  const void* Wi, const void* U, void* da, float* dh, void* ghat,                 \
                                  const void* packed, hipStream_t st);                                            \
  hipError_t launch_gru_pack(int H, const void* Wi, const void* U, void* packed, hipStream_t st);               \
  hipError_t launch_gru_wgrad(long K, int H, const float* a, const void* h, const void* saved, const void* ghat,  \
                              float* dWi, float* dU, float* db, void* ws, ReduceList* defer, hipStream_t st);    \
  hipError_t launch_readout_loss(int H, int n_graphs, const void* X, const float* w_out, const float* b_out,      \
                                 const int32_t* cand_node, const int32_t* cand_ptr, const int32_t* target,       \
                                 float* logits, float* loss, float* dlogit, hipStream_t st);                     \
  hipError_t launch_readout_bwd(int n_pad, int H, int n_cand, const void* X, const float* w_out,                 \
                                const int32_t* cand_node, const float* dlogit, float* dX, float* dw_out,         \
                                float* db_out, void* ws, hipStream_t st);                                        \
  hipError_t launch_sparse_step(int n_pad, int H, int E, const int32_t* row_ptr, const int32_t* col,            \
                                const void* X, const void* Wt, const float* bias, float* a, hipStream_t st);   \
  hipError_t launch_super_fwd(int n_pad, int H, int E, int s, const void* rows, const void* cols, const void* X,  \
                              const void* W, const float* bias, float* a, void* ws, hipStream_t st);            \
  hipError_t launch_super_bwd(int n_pad, int H, int E, int s, const void* rows, const void* rows_t,              \
                              const void* cols_t, const void* X, const void* W, const void* da, float* dX,       \
                              float* dW, float* dbias, void* ws, hipStream_t st);                                \
  bool step_wide_applies(int B, int H);                                                                           \
  hipError_t launch_step_wide(bool rev, int n_pad, int B, int H, int E, const void* bits, const void* V,          \
                              const void* Wsrc, const float* bias, float* out, const float* dX_in, void* dM,      \
                              long ldm, hipStream_t st);

namespace impl_bf16 {
GGNN_DT_LAUNCHERS
// Fused supernode steps (bf16, H <= 64, grids small enough for the
// two-group forms): whether both fused steps take the supernode share at
// this size, and the forward step (with its GRU) and reverse step (with the
// previous step's GRU reverse when da_prev is not NULL) carrying it.
bool step_sn_fusable(int n_pad, int B, int H, int E);
// The record of the fused supernode steps: rec = [P_e (sr x H) | deg_e (sr)],
// P_e = bits_e Z over all nodes for the first sr slice rows (zfm: Z
// feature-major), as a gather where Z is node-major (n_pad a multiple of 64),
// else as the long contraction with its per-chunk partials in ws.
hipError_t launch_super_long_fused(int n_pad, int H, int E, int s, int sr, const void* bits, const void* Z, bool zfm,
                                   float* ws, float* rec, hipStream_t st);
// The fused reverse step's supernode record from the step's gate gradients G^ (node-major [n_pad][3H])
// and Wi: (sum over the listed out-edges of G^ rows) Wi^T (bf16, H = 32 or 64).
bool super_gather_rev_applies(int n_pad, int H);
hipError_t launch_super_gather_rev(int n_pad, int H, int E, int s, int sr, const void* bits, const void* ghat,
                                   const void* Wi, float* rec, hipStream_t st);
hipError_t launch_step_fwd_bits_gru_sn(int n_pad, int B, int H, int E, const void* bits, const void* X, const void* W,
                                       const void* Wt, const float* bias, float* a, const void* Wi, const void* U,
                                       const float* bg, void* h_out, void* saved, const SnStep& sn, hipStream_t st);
hipError_t launch_step_bwd_bits_sn(int n_pad, int B, int H, int E, const void* bits_t, const void* da,
                                   const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,
                                   const void* Wi, const void* U, const void* h_prev, const void* saved_prev,
                                   void* da_prev, float* dh_prev, void* ghat_prev, const SnStep& sn, hipStream_t st);
}
namespace impl_f32 {
GGNN_DT_LAUNCHERS
}
#undef GGNN_DT_LAUNCHERS

#define GGNN_DT_PICK(fn, ...) (dt == GGNN_BF16 ? impl_bf16::fn(__VA_ARGS__) : impl_f32::fn(__VA_ARGS__))

// Dense band: transform-first propagation and its reverse.  dM rows have
// length ldm >= n_pad (ldm = T * n_pad when the reverse pass keeps every
// step's message gradient for the weight-gradient products).
inline hipError_t launch_banded_fwd(int dt, int n_pad, int B, int H, int E, const void* band, const float* M,
                                    float* a, hipStream_t st) {
  return GGNN_DT_PICK(launch_banded_fwd, n_pad, B, H, E, band, M, a, st);
}
inline hipError_t launch_banded_bwd(int dt, int n_pad, int B, int H, int E, const void* band, const void* da,
                                    void* dM, long ldm, hipStream_t st) {
  return GGNN_DT_PICK(launch_banded_bwd, n_pad, B, H, E, band, da, dM, ldm, st);
}

// out[i] += sum_s part[s * stride + i], i < count, fixed summation order.
hipError_t launch_reduce_partials(const float* part, float* out, int nsplit, int count, long stride,
                                  hipStream_t st);
hipError_t launch_fill_zero(float* p, size_t count, hipStream_t st);

// 1-bit band: fused aggregate-first forward and transposed-band reverse.
inline hipError_t launch_step_fwd_bits(int dt, int n_pad, int B, int H, int E, const void* bits, const void* X,
                                       const void* W, const float* bias, float* a, hipStream_t st) {
  return GGNN_DT_PICK(launch_step_fwd_bits, n_pad, B, H, E, bits, X, W, bias, a, st);
}
inline hipError_t launch_banded_bwd_bits(int dt, int n_pad, int B, int H, int E, const void* bits_t, const void* da,
                                         void* dM, long ldm, hipStream_t st) {
  return GGNN_DT_PICK(launch_banded_bwd_bits, n_pad, B, H, E, bits_t, da, dM, ldm, st);
}
// Forward step with the GRU update fused in where the shape allows (sets
// *fused; otherwise only `a` is written and the caller runs the GRU).
// Wt (W_e^T, optional) lets the direct-weight forms read their weight
// fragments as 16-byte rows instead of 2-byte column gathers.
//
// Wide shapes (bf16, H = 128 or 256, B = 128..512) run the sliced wide step
// kernel instead (forward: only when Wt is given); the GRU then runs in its
// own kernel.
inline bool step_wide(int dt, int B, int H) { return dt == GGNN_BF16 && impl_bf16::step_wide_applies(B, H); }
inline hipError_t launch_step_fwd_bits_gru(int dt, int n_pad, int B, int H, int E, const void* bits, const void* X,
                                           const void* W, const void* Wt, const float* bias, float* a,
                                           const void* Wi, const void* U, const float* bg, void* h_out, void* saved,
                                           bool* fused, hipStream_t st) {
  if (Wt != nullptr && step_wide(dt, B, H)) {
    if (fused) *fused = false;
    return impl_bf16::launch_step_wide(false, n_pad, B, H, E, bits, X, Wt, bias, a, nullptr, nullptr, 0, st);
  }
  return GGNN_DT_PICK(launch_step_fwd_bits_gru, n_pad, B, H, E, bits, X, W, Wt, bias, a, Wi, U, bg, h_out, saved,
                      fused, st);
}
// Wt[e][o][h] = W[e][h][o].
inline hipError_t launch_transpose_weights(int dt, int H, int E, const void* W, void* Wt, hipStream_t st) {
  return GGNN_DT_PICK(launch_transpose_weights, H, E, W, Wt, st);
}
// Reverse step that continues, where the shape allows (sets *fused), with
// the previous step's GRU reverse on the completed dX: writes da_prev
// (feature-major), dh_prev and ghat_prev; dX_out may then be NULL.  When
// not fused, dX_out is written and the caller runs the GRU reverse.
inline hipError_t launch_step_bwd_bits_gru(int dt, int n_pad, int B, int H, int E, const void* bits_t, const void* da,
                                           const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,
                                           const void* Wi, const void* U, const void* h_prev, const void* saved_prev,
                                           void* da_prev, float* dh_prev, void* ghat_prev, bool* fused,
                                           hipStream_t st) {
  if (dX_out != nullptr && step_wide(dt, B, H)) {
    if (fused) *fused = false;
    return impl_bf16::launch_step_wide(true, n_pad, B, H, E, bits_t, da, W, nullptr, dX_out, dX_in, dM, ldm, st);
  }
  return GGNN_DT_PICK(launch_step_bwd_bits_gru, n_pad, B, H, E, bits_t, da, W, dX_in, dX_out, dM, ldm, Wi, U, h_prev,
                      saved_prev, da_prev, dh_prev, ghat_prev, fused, st);
}
// Fused reverse step: dM_e = A_e^T da stored node-major (rows of type e start
// at row e * ldm of dM), dX_out = dX_in (or 0) + sum_e dM_e W_e^T.
inline hipError_t launch_step_bwd_bits(int dt, int n_pad, int B, int H, int E, const void* bits_t, const void* da,
                                       const void* W, const float* dX_in, float* dX_out, void* dM, long ldm,
                                       hipStream_t st) {
  if (step_wide(dt, B, H))
    return impl_bf16::launch_step_wide(true, n_pad, B, H, E, bits_t, da, W, nullptr, dX_out, dX_in, dM, ldm, st);
  return GGNN_DT_PICK(launch_step_bwd_bits, n_pad, B, H, E, bits_t, da, W, dX_in, dX_out, dM, ldm, st);
}

inline hipError_t launch_transform_fwd(int dt, int n_pad, int H, int E, const void* X, const void* W,
                                       const float* bias, float* M, hipStream_t st) {
  return GGNN_DT_PICK(launch_transform_fwd, n_pad, H, E, X, W, bias, M, st);
}
// Input gradient dX_out = dX_in + sum_e dM_e W_e^T (dM rows of length ld).
inline hipError_t launch_transform_bwd_dx(int dt, int n_pad, int H, int E, const void* W, const void* dM, long ld,
                                          const float* dX_in, float* dX_out, hipStream_t st) {
  return GGNN_DT_PICK(launch_transform_bwd_dx, n_pad, H, E, W, dM, ld, dX_in, dX_out, st);
}
// Weight gradients over K rows: dW += X^T dM, dbias += row sums of dM (NULL
// to skip), X = K rows [K][H], dM rows of length ld >= K.  The workspace
// (transform_wgrad_workspace bytes) holds per-split partials, reduced in a
// fixed order.
size_t transform_wgrad_workspace(long K, int H, int E);
inline hipError_t launch_transform_wgrad(int dt, long K, int H, int E, const void* X, const void* dM, long ld,
                                         float* dW, float* dbias, void* ws, hipStream_t st) {
  return GGNN_DT_PICK(launch_transform_wgrad, K, H, E, X, dM, ld, dW, dbias, ws, st);
}
// The same with node-major dM: row k of type e at dM + (e * ldk + k) * H.
// With defer non-NULL the partial-sum reductions are appended to it instead
// of launched (launch_reduce_multi runs them together).
inline hipError_t launch_transform_wgrad_nm(int dt, long K, int H, int E, const void* X, const void* dM, long ldk,
                                            float* dW, float* dbias, void* ws, hipStream_t st,
                                            ReduceList* defer = nullptr) {
  return GGNN_DT_PICK(launch_transform_wgrad_nm, K, H, E, X, dM, ldk, dW, dbias, ws, defer, st);
}

// GRU weights packed in the staging order of the large-H kernels (bf16,
// H >= 128): gru_pack_bytes is 0 where no kernel reads the packed form, and
// `packed` (NULL allowed) is then ignored by the launchers below.
size_t gru_pack_bytes(int dt, int H);
inline hipError_t launch_gru_pack(int dt, int H, const void* Wi, const void* U, void* packed, hipStream_t st) {
  return GGNN_DT_PICK(launch_gru_pack, H, Wi, U, packed, st);
}
inline hipError_t launch_gru_fwd(int dt, int n_pad, int H, const float* a, const void* h, const void* Wi,
                                 const void* U, const float* b, void* h_out, void* saved, hipStream_t st,
                                 const void* packed = nullptr) {
  return GGNN_DT_PICK(launch_gru_fwd, n_pad, H, a, h, Wi, U, b, h_out, saved, packed, st);
}
// Node pass of the GRU reverse: da, dh and the gate gradients G^ [n_pad][3H].
inline hipError_t launch_gru_bwd_nodes(int dt, int n_pad, int H, const float* dh_out, const void* h,
                                       const void* saved, const void* Wi, const void* U, void* da, float* dh,
                                       void* ghat, hipStream_t st, const void* packed = nullptr) {
  return GGNN_DT_PICK(launch_gru_bwd_nodes, n_pad, H, dh_out, h, saved, Wi, U, da, dh, ghat, packed, st);
}
size_t ghat_bytes(int dt, long rows, int H);
// GRU weight gradients over K rows of (a, h, saved, G^) stacked node-major:
// dWi, dU, db += (partials in ws of gru_wgrad_workspace bytes, fixed order).
size_t gru_wgrad_workspace(long K, int H);
inline hipError_t launch_gru_wgrad(int dt, long K, int H, const float* a, const void* h, const void* saved,
                                   const void* ghat, float* dWi, float* dU, float* db, void* ws, hipStream_t st,
                                   ReduceList* defer = nullptr) {
  return GGNN_DT_PICK(launch_gru_wgrad, K, H, a, h, saved, ghat, dWi, dU, db, ws, defer, st);
}
// One step: node pass with G^ in ws, then the weight gradients over n_pad rows.
size_t gru_bwd_workspace(int dt, int n_pad, int H);
hipError_t launch_gru_bwd(int dt, int n_pad, int H, const float* dh_out, const float* a, const void* h,
                          const void* saved, const void* Wi, const void* U, void* da, float* dh, float* dWi,
                          float* dU, float* db, void* ws, hipStream_t st);

// Readout and loss (candidate logits, per-graph softmax cross-entropy, mean
// over graphs) and their reverse: dX (written whole), dw_out and db_out
// (accumulated; partials in readout_bwd_workspace bytes, fixed order).
inline hipError_t launch_readout_loss(int dt, int H, int n_graphs, const void* X, const float* w_out,
                                      const float* b_out, const int32_t* cand_node, const int32_t* cand_ptr,
                                      const int32_t* target, float* logits, float* loss, float* dlogit,
                                      hipStream_t st) {
  return GGNN_DT_PICK(launch_readout_loss, H, n_graphs, X, w_out, b_out, cand_node, cand_ptr, target, logits, loss,
                      dlogit, st);
}
size_t readout_bwd_workspace(int H, int n_cand);
inline hipError_t launch_readout_bwd(int dt, int n_pad, int H, int n_cand, const void* X, const float* w_out,
                                     const int32_t* cand_node, const float* dlogit, float* dX, float* dw_out,
                                     float* db_out, void* ws, hipStream_t st) {
  return GGNN_DT_PICK(launch_readout_bwd, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out, ws, st);
}
// Sparse aggregate-first step over receiver-major edge lists (every edge):
// a = sum_e (A_e X) W_e (+ deg_e b_e), W_e given transposed.
inline hipError_t launch_sparse_step(int dt, int n_pad, int H, int E, const int32_t* row_ptr, const int32_t* col,
                                     const void* X, const void* Wt, const float* bias, float* a, hipStream_t st) {
  return GGNN_DT_PICK(launch_sparse_step, n_pad, H, E, row_ptr, col, X, Wt, bias, a, st);
}
// Supernode slices (first s rows and columns), forward (a +=) and reverse
// (dX, dW, dbias +=); workspace of super_workspace bytes.
size_t super_workspace(int n_pad, int H, int E, int s);
// Workspace of the fused supernode steps (bf16, H = 32 or 64): the record
// (super_fused_record_floats floats, room for [P_e (32 x H) | deg_e (32)]),
// then the scratch of launch_super_long_fused (the per-chunk partials).
size_t super_fused_workspace(int n_pad, int H, int E);
size_t super_fused_record_floats(int H, int E);
inline hipError_t launch_super_fwd(int dt, int n_pad, int H, int E, int s, const void* rows, const void* cols,
                                   const void* X, const void* W, const float* bias, float* a, void* ws,
                                   hipStream_t st) {
  return GGNN_DT_PICK(launch_super_fwd, n_pad, H, E, s, rows, cols, X, W, bias, a, ws, st);
}
inline hipError_t launch_super_bwd(int dt, int n_pad, int H, int E, int s, const void* rows, const void* rows_t,
                                   const void* cols_t, const void* X, const void* W, const void* da, float* dX,
                                   float* dW, float* dbias, void* ws, hipStream_t st) {
  return GGNN_DT_PICK(launch_super_bwd, n_pad, H, E, s, rows, rows_t, cols_t, X, W, da, dX, dW, dbias, ws, st);
}
// Momentum update of float32 master parameters (and their compute copy).
hipError_t launch_sgd_momentum(long count, float* theta, float* vel, const float* grad, float lr, float mu, float wd,
                               int nesterov, int copy_dt, void* copy, hipStream_t st);

#undef GGNN_DT_PICK

}  // namespace ggnn
