// C-ABI device entry points: argument validation on the host, then the
// kernel launches on the caller's stream; and the T-step orchestration of
// Eq. 1 (forward with stored activations, then the reverse pass).
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>

#include "common.h"
#include "kernels.h"
#include "profile.h"

using namespace ggnn;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

ggnn_status device_status(hipError_t err, const char* what) {
  if (err == hipSuccess) return GGNN_OK;
  return fail(GGNN_ERR_DEVICE, "%s: %s", what, hipGetErrorString(err));
}

#define CHECK_PTR(p, name)                                                  \
  do {                                                                      \
    GGNN_CHECK_ARG((p) != nullptr, "%s is NULL", name);                     \
    GGNN_CHECK_ARG(aligned16(p), "%s is not 16-byte aligned", name);        \
  } while (0)
#define CHECK_OPT_PTR(p, name)                                              \
  do {                                                                      \
    if ((p) != nullptr) GGNN_CHECK_ARG(aligned16(p), "%s is not 16-byte aligned", name); \
  } while (0)

ggnn_status check_common(int32_t dt, int32_t n_pad, int32_t H) {
  GGNN_CHECK_ARG(supported_dtype(dt), "unknown dtype %d", dt);
  GGNN_CHECK_ARG(n_pad > 0 && n_pad % 32 == 0, "n_pad=%d must be a positive multiple of 32", n_pad);
  GGNN_CHECK_ARG(supported_H(H), "H=%d must be one of 32, 64, 128, 256", H);
  GGNN_CHECK_ARG((int64_t)n_pad * 3 * H < (int64_t)1 << 31, "n_pad*3H exceeds 2^31 elements");
  return GGNN_OK;
}

ggnn_status check_banded(int32_t dt, int32_t n_pad, int32_t B, int32_t H, int32_t E) {
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(supported_B(B), "B=%d must be one of 32, 64, 128, 256, 512", B);
  GGNN_CHECK_ARG(n_pad % B == 0, "n_pad=%d must be a multiple of B=%d", n_pad, B);
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  return GGNN_OK;
}

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// Whether the byte ranges [p, p + pb) and [q, q + qb) share no byte.
bool disjoint(const void* p, size_t pb, const void* q, size_t qb) {
  const char *a = static_cast<const char*>(p), *c = static_cast<const char*>(q);
  return a + pb <= c || c + qb <= a;
}

}  // namespace

// Reverse-pass workspace: the gate gradients G^ of every step ([T][n_pad][3H],
// kept for the GRU weight gradients), then the GRU and message-transform
// weight-gradient partials over K = T * n_pad rows, each at a 256-byte
// aligned offset.
namespace {
struct BwdLayout {
  size_t ghat, gru_part, tr_part, da2, dh2, total;
};
BwdLayout bwd_layout(const ggnn_model* m) {
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  const long K = (long)m->T * m->n_pad;
  const size_t es = m->dtype == GGNN_BF16 ? 2 : 4;
  BwdLayout l;
  l.ghat = 0;
  l.gru_part = up(ghat_bytes(m->dtype, K, m->H));
  l.tr_part = l.gru_part + up(gru_wgrad_workspace(K, m->H));
  // second da / dh buffers: the fused bit-band reverse step reads one step's
  // and writes the previous step's
  l.da2 = l.tr_part + up(transform_wgrad_workspace(K, m->H, m->E));
  l.dh2 = l.da2 + up((size_t)m->H * m->n_pad * es);
  l.total = l.dh2 + (size_t)m->n_pad * m->H * sizeof(float);
  return l;
}
}  // namespace

extern "C" {

ggnn_status ggnn_msg_transform(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, const void* X, const void* W,
                               const float* bias, float* M, void* stream) {
  clear_error();
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  CHECK_PTR(X, "X");
  CHECK_PTR(W, "W");
  CHECK_OPT_PTR(bias, "bias");
  CHECK_PTR(M, "M");
  return device_status(launch_transform_fwd(dt, n_pad, H, E, X, W, bias, M, as_stream(stream)), "msg_transform");
}

ggnn_status ggnn_banded_propagate(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E, const void* band,
                                  const float* M, float* a, void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(band, "band");
  CHECK_PTR(M, "M");
  CHECK_PTR(a, "a");
  return device_status(launch_banded_fwd(dt, n_pad, B, H, E, band, M, a, as_stream(stream)), "banded_propagate");
}

ggnn_status ggnn_gru_update(ggnn_dtype dt, int32_t n_pad, int32_t H, const float* a, const void* h, const void* Wi,
                            const void* U, const float* b, void* h_out, void* saved, void* stream) {
  clear_error();
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  CHECK_PTR(a, "a");
  CHECK_PTR(h, "h");
  CHECK_PTR(Wi, "Wi");
  CHECK_PTR(U, "U");
  CHECK_PTR(b, "b");
  CHECK_PTR(h_out, "h_out");
  CHECK_OPT_PTR(saved, "saved");
  GGNN_CHECK_ARG(h_out != h, "h_out must not alias h");
  return device_status(launch_gru_fwd(dt, n_pad, H, a, h, Wi, U, b, h_out, saved, as_stream(stream)), "gru_update");
}

size_t ggnn_gru_update_bwd_workspace_bytes(ggnn_dtype dt, int32_t n_pad, int32_t H) {
  if (!supported_dtype(dt) || n_pad <= 0 || n_pad % 32 != 0 || !supported_H(H)) return 0;
  return gru_bwd_workspace(dt, n_pad, H);
}

ggnn_status ggnn_gru_update_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, const float* dh_out, const float* a,
                                const void* h, const void* saved, const void* Wi, const void* U, void* da, float* dh,
                                float* dWi, float* dU, float* db, void* workspace, size_t workspace_bytes,
                                void* stream) {
  clear_error();
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  CHECK_PTR(dh_out, "dh_out");
  CHECK_PTR(a, "a");
  CHECK_PTR(h, "h");
  CHECK_PTR(saved, "saved");
  CHECK_PTR(Wi, "Wi");
  CHECK_PTR(U, "U");
  CHECK_PTR(da, "da");
  CHECK_PTR(dh, "dh");
  CHECK_PTR(dWi, "dWi");
  CHECK_PTR(dU, "dU");
  CHECK_PTR(db, "db");
  GGNN_CHECK_ARG(dh != dh_out, "dh must not alias dh_out");
  const size_t need = gru_bwd_workspace(dt, n_pad, H);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))
    return fail(GGNN_ERR_WORKSPACE, "gru_update_bwd needs a 16-byte aligned workspace of %zu bytes (got %zu)", need,
                workspace ? workspace_bytes : (size_t)0);
  return device_status(
      launch_gru_bwd(dt, n_pad, H, dh_out, a, h, saved, Wi, U, da, dh, dWi, dU, db, workspace, as_stream(stream)),
      "gru_update_bwd");
}

ggnn_status ggnn_banded_propagate_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                      const void* band, const void* da, void* dM, void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(band, "band");
  CHECK_PTR(da, "da");
  CHECK_PTR(dM, "dM");
  return device_status(launch_banded_bwd(dt, n_pad, B, H, E, band, da, dM, n_pad, as_stream(stream)),
                       "banded_propagate_bwd");
}

ggnn_status ggnn_banded_step_bits(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E, const void* bits,
                                  const void* X, const void* W, const float* bias, float* a, void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(bits, "bits");
  CHECK_PTR(X, "X");
  CHECK_PTR(W, "W");
  CHECK_OPT_PTR(bias, "bias");
  CHECK_PTR(a, "a");
  return device_status(launch_step_fwd_bits(dt, n_pad, B, H, E, bits, X, W, bias, a, as_stream(stream)),
                       "banded_step_bits");
}

ggnn_status ggnn_banded_propagate_bits_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                           const void* bits_t, const void* da, void* dM, void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(bits_t, "bits_t");
  CHECK_PTR(da, "da");
  CHECK_PTR(dM, "dM");
  return device_status(launch_banded_bwd_bits(dt, n_pad, B, H, E, bits_t, da, dM, n_pad, as_stream(stream)),
                       "banded_propagate_bits_bwd");
}

ggnn_status ggnn_banded_step_bits_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                      const void* bits_t, const void* da, const void* W, const float* dX_in,
                                      float* dX_out, void* dM, int64_t ldm, void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(bits_t, "bits_t");
  CHECK_PTR(da, "da");
  CHECK_PTR(W, "W");
  CHECK_OPT_PTR(dX_in, "dX_in");
  CHECK_PTR(dX_out, "dX_out");
  CHECK_PTR(dM, "dM");
  GGNN_CHECK_ARG(ldm >= n_pad, "ldm=%lld must be at least n_pad=%d", (long long)ldm, n_pad);
  return device_status(
      launch_step_bwd_bits(dt, n_pad, B, H, E, bits_t, da, W, dX_in, dX_out, dM, (long)ldm, as_stream(stream)),
      "banded_step_bits_bwd");
}

ggnn_status ggnn_transpose_weights(ggnn_dtype dt, int32_t H, int32_t E, const void* W, void* Wt, void* stream) {
  clear_error();
  GGNN_CHECK_ARG(supported_dtype(dt), "unknown dtype %d", dt);
  GGNN_CHECK_ARG(supported_H(H), "H=%d must be one of 32, 64, 128, 256", H);
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  CHECK_PTR(W, "W");
  CHECK_PTR(Wt, "Wt");
  GGNN_CHECK_ARG(W != Wt, "Wt must not overlap W");
  return device_status(launch_transpose_weights(dt, H, E, W, Wt, as_stream(stream)), "transpose_weights");
}

size_t ggnn_gru_pack_bytes(ggnn_dtype dt, int32_t H) {
  if (!supported_dtype(dt) || !supported_H(H)) return 0;
  return gru_pack_bytes(dt, H);
}

ggnn_status ggnn_gru_pack_weights(ggnn_dtype dt, int32_t H, const void* Wi, const void* U, void* packed,
                                  void* stream) {
  clear_error();
  GGNN_CHECK_ARG(supported_dtype(dt), "unknown dtype %d", dt);
  GGNN_CHECK_ARG(supported_H(H), "H=%d must be one of 32, 64, 128, 256", H);
  const size_t bytes = gru_pack_bytes(dt, H);
  if (bytes == 0) return GGNN_OK;   // no kernel reads the packed form
  CHECK_PTR(Wi, "Wi");
  CHECK_PTR(U, "U");
  CHECK_PTR(packed, "packed");
  const size_t wb = (size_t)H * 3 * H * dtype_bytes(dt);
  GGNN_CHECK_ARG(disjoint(packed, bytes, Wi, wb) && disjoint(packed, bytes, U, wb),
                 "packed must not overlap Wi or U");
  return device_status(launch_gru_pack(dt, H, Wi, U, packed, as_stream(stream)), "gru_pack_weights");
}

ggnn_status ggnn_step_bits_gru(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E, const void* bits,
                               const void* X, const void* W, const void* Wt, const float* bias, const void* Wi,
                               const void* U, const float* b, float* a, void* h_out, void* saved, void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(bits, "bits");
  CHECK_PTR(X, "X");
  CHECK_PTR(W, "W");
  CHECK_OPT_PTR(bias, "bias");
  CHECK_PTR(Wi, "Wi");
  CHECK_PTR(U, "U");
  CHECK_PTR(b, "b");
  CHECK_PTR(a, "a");
  CHECK_PTR(h_out, "h_out");
  CHECK_PTR(saved, "saved");
  // Workgroups read neighbour-block rows of X that other workgroups' rows of
  // h_out would overwrite: the two must not share bytes.
  const size_t xb = (size_t)n_pad * H * dtype_bytes(dt);
  GGNN_CHECK_ARG(disjoint(X, xb, h_out, xb), "X and h_out must not overlap");
  hipStream_t s = as_stream(stream);
  bool fused = false;
  CHECK_OPT_PTR(Wt, "Wt");
  hipError_t err =
      launch_step_fwd_bits_gru(dt, n_pad, B, H, E, bits, X, W, Wt, bias, a, Wi, U, b, h_out, saved, &fused, s);
  if (err == hipSuccess && !fused) err = launch_gru_fwd(dt, n_pad, H, a, X, Wi, U, b, h_out, saved, s);
  return device_status(err, "step_bits_gru");
}

ggnn_status ggnn_step_bits_gru_bwd(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E,
                                   const void* bits_t, const void* da, const void* W, const float* dX_in, void* dM,
                                   int64_t ldm, const void* Wi, const void* U, const void* h_prev,
                                   const void* saved_prev, void* da_prev, float* dh_prev, void* ghat_prev,
                                   void* stream) {
  clear_error();
  ggnn_status st = check_banded(dt, n_pad, B, H, E);
  if (st != GGNN_OK) return st;
  CHECK_PTR(bits_t, "bits_t");
  CHECK_PTR(da, "da");
  CHECK_PTR(W, "W");
  CHECK_OPT_PTR(dX_in, "dX_in");
  CHECK_PTR(dM, "dM");
  GGNN_CHECK_ARG(ldm >= n_pad, "ldm=%lld must be at least n_pad=%d", (long long)ldm, n_pad);
  CHECK_PTR(Wi, "Wi");
  CHECK_PTR(U, "U");
  CHECK_PTR(h_prev, "h_prev");
  CHECK_PTR(saved_prev, "saved_prev");
  CHECK_PTR(da_prev, "da_prev");
  CHECK_PTR(dh_prev, "dh_prev");
  CHECK_PTR(ghat_prev, "ghat_prev");
  GGNN_CHECK_ARG(da_prev != da, "da_prev must not alias da (da is read by every workgroup)");
  hipStream_t s = as_stream(stream);
  bool fused = false;
  hipError_t err = launch_step_bwd_bits_gru(dt, n_pad, B, H, E, bits_t, da, W, dX_in, dh_prev, dM, (long)ldm, Wi, U,
                                            h_prev, saved_prev, da_prev, dh_prev, ghat_prev, &fused, s);
  // Unfused shapes: the summed dX went to dh_prev; the GRU reverse reads it
  // there and overwrites it node by node with dh (each node's row is read
  // before it is written, by the same wave).
  if (err == hipSuccess && !fused)
    err = launch_gru_bwd_nodes(dt, n_pad, H, dh_prev, h_prev, saved_prev, Wi, U, da_prev, dh_prev, ghat_prev, s);
  return device_status(err, "step_bits_gru_bwd");
}

size_t ggnn_msg_transform_bwd_workspace_bytes(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E) {
  if (!supported_dtype(dt) || n_pad <= 0 || n_pad % 32 != 0 || !supported_H(H) || E < 1 || E > 64) return 0;
  return transform_wgrad_workspace(n_pad, H, E);
}

ggnn_status ggnn_msg_transform_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, const void* X, const void* W,
                                   const void* dM, const float* dX_in, float* dX_out, float* dW, float* dbias,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  CHECK_PTR(X, "X");
  CHECK_PTR(W, "W");
  CHECK_PTR(dM, "dM");
  CHECK_OPT_PTR(dX_in, "dX_in");
  CHECK_PTR(dX_out, "dX_out");
  CHECK_PTR(dW, "dW");
  CHECK_OPT_PTR(dbias, "dbias");
  const size_t need = transform_wgrad_workspace(n_pad, H, E);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))
    return fail(GGNN_ERR_WORKSPACE, "msg_transform_bwd needs a 16-byte aligned workspace of %zu bytes (got %zu)",
                need, workspace ? workspace_bytes : (size_t)0);
  hipStream_t hs = as_stream(stream);
  hipError_t err = launch_transform_bwd_dx(dt, n_pad, H, E, W, dM, n_pad, dX_in, dX_out, hs);
  if (err == hipSuccess) err = launch_transform_wgrad(dt, n_pad, H, E, X, dM, n_pad, dW, dbias, workspace, hs);
  return device_status(err, "msg_transform_bwd");
}

// ---------------------------------------------------------------------------
// T-step orchestration
// ---------------------------------------------------------------------------

static ggnn_status check_model(const ggnn_model* m) {
  GGNN_CHECK_ARG(m != nullptr, "model is NULL");
  ggnn_status st = check_banded(m->dtype, m->n_pad, m->B, m->H, m->E);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(m->T >= 1 && m->T <= 1024, "T=%d must be in [1, 1024]", m->T);
  CHECK_PTR(m->band, "model.band");
  CHECK_PTR(m->W, "model.W");
  CHECK_OPT_PTR(m->bias, "model.bias");
  CHECK_PTR(m->Wi, "model.Wi");
  CHECK_PTR(m->U, "model.U");
  CHECK_PTR(m->b, "model.b");
  GGNN_CHECK_ARG(m->band_format == GGNN_BAND_DENSE || m->band_format == GGNN_BAND_BITS,
                 "unknown band_format %d", m->band_format);
  if (m->band_format == GGNN_BAND_BITS) CHECK_PTR(m->band_t, "model.band_t");
  CHECK_OPT_PTR(m->Wt, "model.Wt");
  CHECK_OPT_PTR(m->gru_packed, "model.gru_packed");
  GGNN_CHECK_ARG(m->n_super >= 0, "n_super=%d must not be negative", m->n_super);
  if (m->n_super > 0) {
    GGNN_CHECK_ARG(m->band_format == GGNN_BAND_BITS, "supernodes need the bit band");
    GGNN_CHECK_ARG(ggnn_super_bytes(m->n_pad, m->E, m->n_super) > 0,
                   "n_super=%d (32, 64, 96 or 128, at most n_pad; n_pad=%d a multiple of 64)", m->n_super, m->n_pad);
    GGNN_CHECK_ARG(m->n_super_active >= 0 && m->n_super_active <= m->n_super && m->n_super_active % 16 == 0,
                   "n_super_active=%d must be a multiple of 16 in [0, n_super=%d]", m->n_super_active, m->n_super);
    if (m->n_super_active > 0) {
      CHECK_PTR(m->super_rows, "model.super_rows");
      CHECK_PTR(m->super_cols, "model.super_cols");
      CHECK_PTR(m->super_rows_t, "model.super_rows_t");
      CHECK_PTR(m->super_cols_t, "model.super_cols_t");
    }
  }
  return GGNN_OK;
}

// Supernode slices run inside the fused step kernels (see ggnn_forward).
static bool super_fused(const ggnn_model* m) {
  return m->n_super > 0 && (m->n_super_active == 16 || m->n_super_active == 32) && m->dtype == GGNN_BF16 &&
         m->H <= 64 && impl_bf16::step_sn_fusable(m->n_pad, m->B, m->H, m->E);
}
static size_t super_model_ws(const ggnn_model* m) {
  if (m->n_super <= 0 || m->n_super_active <= 0) return 0;
  const size_t a = super_workspace(m->n_pad, m->H, m->E, m->n_super);
  const size_t b = super_fused(m) ? super_fused_workspace(m->n_pad, m->H, m->E) : 0;
  return a > b ? a : b;
}
// The supernode scratch of a model about to run.
static ggnn_status check_super_ws(const ggnn_model* m) {
  const size_t need = super_model_ws(m);
  if (need == 0) return GGNN_OK;
  if (m->super_ws == nullptr || m->super_ws_bytes < need || !aligned16(m->super_ws))
    return fail(GGNN_ERR_WORKSPACE, "supernodes need a 16-byte aligned model.super_ws of %zu bytes (got %zu)", need,
                m->super_ws ? m->super_ws_bytes : (size_t)0);
  return GGNN_OK;
}

static ggnn_status check_acts(const ggnn_model* m, const ggnn_activations* act) {
  GGNN_CHECK_ARG(act != nullptr, "activations is NULL");
  CHECK_PTR(act->X, "act.X");
  CHECK_PTR(act->a, "act.a");
  CHECK_PTR(act->saved, "act.saved");
  if (m->band_format == GGNN_BAND_DENSE) CHECK_PTR(act->M, "act.M");
  return GGNN_OK;
}


size_t ggnn_super_model_workspace_bytes(const ggnn_model* m) {
  if (m == nullptr || check_model(m) != GGNN_OK) {
    clear_error();
    return 0;
  }
  return super_model_ws(m);
}

int32_t ggnn_super_fusable(ggnn_dtype dt, int32_t n_pad, int32_t B, int32_t H, int32_t E, int32_t n_super_active) {
  if (check_banded(dt, n_pad, B, H, E) != GGNN_OK) {
    clear_error();
    return 0;
  }
  return (n_super_active == 16 || n_super_active == 32) && dt == GGNN_BF16 && H <= 64 &&
                 impl_bf16::step_sn_fusable(n_pad, B, H, E)
             ? 1
             : 0;
}

size_t ggnn_backward_workspace_bytes(const ggnn_model* m) {
  if (m == nullptr || check_model(m) != GGNN_OK) {
    clear_error();
    return 0;
  }
  return bwd_layout(m).total;
}

ggnn_status ggnn_forward(const ggnn_model* m, const ggnn_activations* act, void* stream) {
  clear_error();
  ggnn_status st = check_model(m);
  if (st != GGNN_OK) return st;
  st = check_acts(m, act);
  if (st != GGNN_OK) return st;
  st = check_super_ws(m);
  if (st != GGNN_OK) return st;
  const size_t es = dtype_bytes(m->dtype);
  const size_t xs = (size_t)m->n_pad * m->H;
  hipStream_t s = as_stream(stream);
  const void* gru_pk = gru_pack_bytes(m->dtype, m->H) ? m->gru_packed : nullptr;
  const bool sn = m->n_super > 0 && m->n_super_active > 0;
  const bool snf = sn && super_fused(m);
  float* sn_rec = static_cast<float*>(m->super_ws);
  float* sn_scr = snf ? sn_rec + super_fused_record_floats(m->H, m->E) : nullptr;
  for (int t = 0; t < m->T; ++t) {
    const char* Xt = static_cast<const char*>(act->X) + t * xs * es;
    char* Xn = static_cast<char*>(act->X) + (t + 1) * xs * es;
    float* at = act->a + t * xs;
    char* sv = static_cast<char*>(act->saved) + t * 3 * xs * es;
    hipError_t err;
    bool fused = false;   // the bit-band step also ran the GRU update
    if (snf) {
      // supernode rows: R_e X over all nodes; then the fused step with the
      // column slice as a fourth block
      prof_begin(s);
      err = impl_bf16::launch_super_long_fused(m->n_pad, m->H, m->E, m->n_super, m->n_super_active, m->super_rows,
                                               Xt, false, sn_scr, sn_rec, s);
      prof_end(s, PROF_SUPER_RECORD);
      if (err == hipSuccess) {
        prof_begin(s);
        err = impl_bf16::launch_step_fwd_bits_gru_sn(m->n_pad, m->B, m->H, m->E, m->band, Xt, m->W, m->Wt, m->bias,
                                                     at, m->Wi, m->U, m->b, Xn, sv,
                                                     SnStep{m->super_cols, sn_rec, m->n_super, m->n_super_active},
                                                     s);
        prof_end(s, PROF_STEP_FWD_GRU);
        fused = true;
      }
    } else if (m->band_format == GGNN_BAND_BITS) {
      // with stand-alone supernode slices the GRU waits for their share of a
      prof_begin(s);
      err = launch_step_fwd_bits_gru(m->dtype, m->n_pad, m->B, m->H, m->E, m->band, Xt, m->W, m->Wt, m->bias, at,
                                     sn ? nullptr : m->Wi, m->U, m->b, Xn, sv, &fused, s);
      prof_end(s, fused ? PROF_STEP_FWD_GRU : PROF_STEP_FWD);
      if (err == hipSuccess && sn) {
        prof_begin(s);
        err = launch_super_fwd(m->dtype, m->n_pad, m->H, m->E, m->n_super, m->super_rows, m->super_cols, Xt, m->W,
                               m->bias, at, m->super_ws, s);
        prof_end(s, PROF_SUPER);
      }
    } else {
      prof_begin(s);
      err = launch_transform_fwd(m->dtype, m->n_pad, m->H, m->E, Xt, m->W, m->bias, act->M, s);
      prof_end(s, PROF_TRANSFORM_FWD);
      if (err == hipSuccess) {
        prof_begin(s);
        err = launch_banded_fwd(m->dtype, m->n_pad, m->B, m->H, m->E, m->band, act->M, at, s);
        prof_end(s, PROF_BANDED_FWD);
      }
    }
    if (err == hipSuccess && !fused) {
      prof_begin(s);
      err = launch_gru_fwd(m->dtype, m->n_pad, m->H, at, Xt, m->Wi, m->U, m->b, Xn, sv, s, gru_pk);
      prof_end(s, PROF_GRU_FWD);
    }
    if (err != hipSuccess) return device_status(err, "forward");
  }
  return GGNN_OK;
}

ggnn_status ggnn_backward(const ggnn_model* m, const ggnn_activations* act, const ggnn_grads* gr, void* stream) {
  clear_error();
  ggnn_status st = check_model(m);
  if (st != GGNN_OK) return st;
  st = check_acts(m, act);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(gr != nullptr, "grads is NULL");
  CHECK_PTR(gr->dX, "grads.dX");
  CHECK_PTR(gr->dW, "grads.dW");
  CHECK_PTR(gr->dWi, "grads.dWi");
  CHECK_PTR(gr->dU, "grads.dU");
  CHECK_PTR(gr->db, "grads.db");
  CHECK_PTR(gr->da, "grads.da");
  CHECK_PTR(gr->dM, "grads.dM");
  CHECK_PTR(gr->dh, "grads.dh");
  if (m->bias) CHECK_PTR(gr->dbias, "grads.dbias");
  st = check_super_ws(m);
  if (st != GGNN_OK) return st;
  const BwdLayout L = bwd_layout(m);
  if (gr->workspace == nullptr || gr->workspace_bytes < L.total || !aligned16(gr->workspace))
    return fail(GGNN_ERR_WORKSPACE, "backward needs a 16-byte aligned workspace of %zu bytes (got %zu)", L.total,
                gr->workspace ? gr->workspace_bytes : (size_t)0);
  const size_t es = dtype_bytes(m->dtype);
  const size_t xs = (size_t)m->n_pad * m->H;
  const long K = (long)m->T * m->n_pad;   // rows of the weight-gradient contractions; also the dM row length
  hipStream_t s = as_stream(stream);
  float* dbias = m->bias ? gr->dbias : nullptr;
  const void* gru_pk = gru_pack_bytes(m->dtype, m->H) ? m->gru_packed : nullptr;
  char* ws = static_cast<char*>(gr->workspace);
  char* ghat = ws + L.ghat;
  // Node passes, t = T-1..0.  The weight gradients are sums over steps and
  // nodes of products of per-step quantities, so each step only stores its
  // factors (G^ of step t; dM of step t at offset t * n_pad) and the sums
  // run once, over all T * n_pad rows, after the loop.
  auto Xs = [&](int t) { return static_cast<const char*>(act->X) + t * xs * es; };
  auto Ss = [&](int t) { return static_cast<const char*>(act->saved) + t * 3 * xs * es; };
  auto Gs = [&](int t) { return ghat + t * 3 * xs * es; };
  if (m->band_format == GGNN_BAND_BITS) {
    // Bit band: the reverse step of t also runs the GRU reverse of t-1 when
    // the kernel shape allows (one launch per step); da and dh alternate
    // between two buffers (step t's are read while t-1's are written).
    void* da_b[2] = {gr->da, ws + L.da2};
    float* dh_b[2] = {gr->dh, reinterpret_cast<float*>(ws + L.dh2)};
    int cur = 0;
    const bool sn = m->n_super > 0 && m->n_super_active > 0;
    const bool snf = sn && super_fused(m);
    float* sn_rec = static_cast<float*>(m->super_ws);
    float* sn_scr = snf ? sn_rec + super_fused_record_floats(m->H, m->E) : nullptr;

    prof_begin(s);
    hipError_t err = launch_gru_bwd_nodes(m->dtype, m->n_pad, m->H, gr->dX, Xs(m->T - 1), Ss(m->T - 1), m->Wi, m->U,
                                          da_b[0], dh_b[0], Gs(m->T - 1), s, gru_pk);
    prof_end(s, PROF_GRU_REV);
    if (err != hipSuccess) return device_status(err, "backward");
    for (int t = m->T - 1; t >= 0; --t) {
      char* dMr = static_cast<char*>(gr->dM) + (size_t)t * m->n_pad * m->H * es;   // node-major rows of step t
      if (snf) {
        // supernode rows: C_e^T da over all nodes; then the fused reverse step
        // with the transposed row slice as a fourth block
        prof_begin(s);
        if (impl_bf16::super_gather_rev_applies(m->n_pad, m->H))
          err = impl_bf16::launch_super_gather_rev(m->n_pad, m->H, m->E, m->n_super, m->n_super_active,
                                                   m->super_cols_t, Gs(t), m->Wi, sn_rec, s);
        else
          err = impl_bf16::launch_super_long_fused(m->n_pad, m->H, m->E, m->n_super, m->n_super_active,
                                                   m->super_cols_t, da_b[cur], true, sn_scr, sn_rec, s);
        prof_end(s, PROF_SUPER_RECORD);
        if (err == hipSuccess) {
          const bool prev = t > 0;
          prof_begin(s);
          err = impl_bf16::launch_step_bwd_bits_sn(
              m->n_pad, m->B, m->H, m->E, m->band_t, da_b[cur], m->W, dh_b[cur], gr->dX, dMr, K, m->Wi, m->U,
              prev ? Xs(t - 1) : nullptr, prev ? Ss(t - 1) : nullptr, prev ? da_b[1 - cur] : nullptr,
              prev ? dh_b[1 - cur] : nullptr, prev ? Gs(t - 1) : nullptr,
              SnStep{m->super_rows_t, sn_rec, m->n_super, m->n_super_active}, s);
          prof_end(s, prev ? PROF_STEP_REV_GRU : PROF_STEP_REV);
        }
        if (err != hipSuccess) return device_status(err, "backward");
        cur ^= 1;
        continue;
      }
      if (sn) {
        // stand-alone slices: their share of dX goes into dh (the step's
        // dX_in), of dW and dbias straight into the gradients
        prof_begin(s);
        err = launch_super_bwd(m->dtype, m->n_pad, m->H, m->E, m->n_super, m->super_rows, m->super_rows_t,
                               m->super_cols_t, Xs(t), m->W, da_b[cur], dh_b[cur], gr->dW, dbias, m->super_ws, s);
        prof_end(s, PROF_SUPER);
        if (err != hipSuccess) return device_status(err, "backward");
      }
      if (t > 0) {
        bool fused = false;
        prof_begin(s);
        err = launch_step_bwd_bits_gru(m->dtype, m->n_pad, m->B, m->H, m->E, m->band_t, da_b[cur], m->W, dh_b[cur],
                                       gr->dX, dMr, K, m->Wi, m->U, Xs(t - 1), Ss(t - 1), da_b[1 - cur],
                                       dh_b[1 - cur], Gs(t - 1), &fused, s);
        prof_end(s, fused ? PROF_STEP_REV_GRU : PROF_STEP_REV);
        if (err == hipSuccess && !fused) {
          prof_begin(s);
          err = launch_gru_bwd_nodes(m->dtype, m->n_pad, m->H, gr->dX, Xs(t - 1), Ss(t - 1), m->Wi, m->U,
                                     da_b[1 - cur], dh_b[1 - cur], Gs(t - 1), s, gru_pk);
          prof_end(s, PROF_GRU_REV);
        }
      } else {
        prof_begin(s);
        err = launch_step_bwd_bits(m->dtype, m->n_pad, m->B, m->H, m->E, m->band_t, da_b[cur], m->W, dh_b[cur],
                                   gr->dX, dMr, K, s);
        prof_end(s, PROF_STEP_REV);
      }
      if (err != hipSuccess) return device_status(err, "backward");
      cur ^= 1;
    }
  } else {
    for (int t = m->T - 1; t >= 0; --t) {
      char* dMt = static_cast<char*>(gr->dM) + (size_t)t * m->n_pad * es;   // feature-major columns of step t
      prof_begin(s);
      hipError_t err = launch_gru_bwd_nodes(m->dtype, m->n_pad, m->H, gr->dX, Xs(t), Ss(t), m->Wi, m->U, gr->da,
                                            gr->dh, Gs(t), s, gru_pk);
      prof_end(s, PROF_GRU_REV);
      if (err == hipSuccess) {
        prof_begin(s);
        err = launch_banded_bwd(m->dtype, m->n_pad, m->B, m->H, m->E, m->band, gr->da, dMt, K, s);
        prof_end(s, PROF_BANDED_REV);
      }
      if (err == hipSuccess) {
        prof_begin(s);
        err = launch_transform_bwd_dx(m->dtype, m->n_pad, m->H, m->E, m->W, dMt, K, gr->dh, gr->dX, s);
        prof_end(s, PROF_TRANSFORM_REV_DX);
      }
      if (err != hipSuccess) return device_status(err, "backward");
    }
  }
  // The weight-gradient contractions leave per-split partials; their
  // fixed-order reductions then run as one launch.
  ReduceList red;
  prof_begin(s);
  hipError_t err = launch_gru_wgrad(m->dtype, K, m->H, act->a, act->X, act->saved, ghat, gr->dWi, gr->dU, gr->db,
                                    ws + L.gru_part, s, &red);
  prof_end(s, PROF_WGRAD_GRU);
  if (err == hipSuccess) {
    prof_begin(s);
    err = m->band_format == GGNN_BAND_BITS
              ? launch_transform_wgrad_nm(m->dtype, K, m->H, m->E, act->X, gr->dM, K, gr->dW, dbias, ws + L.tr_part, s,
                                          &red)
              : launch_transform_wgrad(m->dtype, K, m->H, m->E, act->X, gr->dM, K, gr->dW, dbias, ws + L.tr_part, s);
    prof_end(s, PROF_WGRAD_TRANSFORM);
  }
  if (err == hipSuccess) {
    prof_begin(s);
    err = launch_reduce_multi(red, s);
    prof_end(s, PROF_REDUCE);
  }
  return device_status(err, "backward");
}

ggnn_status ggnn_readout_loss(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t n_graphs, int32_t n_cand,
                              const void* X, const float* w_out, const float* b_out, const int32_t* cand_node,
                              const int32_t* cand_ptr, const int32_t* target, float* logits, float* loss,
                              float* dlogit, void* stream) {
  clear_error();
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(n_graphs >= 1, "n_graphs=%d must be at least 1", n_graphs);
  GGNN_CHECK_ARG(n_cand >= 0, "n_cand=%d must not be negative", n_cand);
  CHECK_PTR(X, "X");
  CHECK_PTR(w_out, "w_out");
  CHECK_PTR(b_out, "b_out");
  CHECK_PTR(cand_ptr, "cand_ptr");
  CHECK_PTR(target, "target");
  CHECK_PTR(loss, "loss");
  if (n_cand > 0) {
    CHECK_PTR(cand_node, "cand_node");
    CHECK_PTR(logits, "logits");
    CHECK_PTR(dlogit, "dlogit");
  }
  return device_status(launch_readout_loss(dt, H, n_graphs, X, w_out, b_out, cand_node, cand_ptr, target, logits,
                                           loss, dlogit, as_stream(stream)),
                       "readout_loss");
}

size_t ggnn_readout_loss_bwd_workspace_bytes(int32_t H, int32_t n_cand) {
  if (!supported_H(H) || n_cand < 0) return 0;
  return readout_bwd_workspace(H, n_cand);
}

}  // extern "C"

namespace {
ggnn_status check_readout_bwd(int32_t dt, int32_t n_pad, int32_t H, int32_t n_cand, const void* X,
                              const float* w_out, const int32_t* cand_node, const float* dlogit, float* dX,
                              float* dw_out, float* db_out) {
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(n_cand >= 0, "n_cand=%d must not be negative", n_cand);
  CHECK_PTR(X, "X");
  CHECK_PTR(w_out, "w_out");
  CHECK_PTR(dX, "dX");
  CHECK_PTR(dw_out, "dw_out");
  CHECK_PTR(db_out, "db_out");
  if (n_cand > 0) {
    CHECK_PTR(cand_node, "cand_node");
    CHECK_PTR(dlogit, "dlogit");
  }
  return GGNN_OK;
}
}  // namespace

extern "C" {

ggnn_status ggnn_readout_loss_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t n_cand, const void* X,
                                  const float* w_out, const int32_t* cand_node, const float* dlogit, float* dX,
                                  float* dw_out, float* db_out, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  clear_error();
  ggnn_status st = check_readout_bwd(dt, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out);
  if (st != GGNN_OK) return st;
  const size_t need = readout_bwd_workspace(H, n_cand);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))
    return fail(GGNN_ERR_WORKSPACE, "readout_loss_bwd needs a 16-byte aligned workspace of %zu bytes (got %zu)",
                need, workspace ? workspace_bytes : (size_t)0);
  return device_status(launch_readout_bwd(dt, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out,
                                          workspace, as_stream(stream)),
                       "readout_loss_bwd");
}

ggnn_status ggnn_sgd_momentum(int64_t count, float* param, float* velocity, const float* grad, float lr,
                              float momentum, float weight_decay, int32_t nesterov, ggnn_dtype copy_dtype,
                              void* param_copy, void* stream) {
  clear_error();
  GGNN_CHECK_ARG(count >= 0, "count=%lld must not be negative", (long long)count);
  GGNN_CHECK_ARG(std::isfinite(lr) && std::isfinite(momentum) && std::isfinite(weight_decay),
                 "lr, momentum and weight_decay must be finite");
  GGNN_CHECK_ARG(momentum >= 0.f && weight_decay >= 0.f, "momentum and weight_decay must not be negative");
  if (count == 0) return GGNN_OK;
  CHECK_PTR(param, "param");
  CHECK_PTR(velocity, "velocity");
  CHECK_PTR(grad, "grad");
  CHECK_OPT_PTR(param_copy, "param_copy");
  if (param_copy != nullptr) {
    GGNN_CHECK_ARG(supported_dtype(copy_dtype), "unknown copy dtype %d", copy_dtype);
    GGNN_CHECK_ARG(param_copy != param, "param_copy must not be param");
  }
  GGNN_CHECK_ARG(velocity != param && grad != param && grad != velocity,
                 "param, velocity and grad must be distinct buffers");
  return device_status(launch_sgd_momentum(count, param, velocity, grad, lr, momentum, weight_decay,
                                           nesterov != 0, copy_dtype, param_copy, as_stream(stream)),
                       "sgd_momentum");
}

ggnn_status ggnn_sparse_step(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, const int32_t* row_ptr,
                             const int32_t* col, int64_t nnz, const void* X, const void* Wt, const float* bias,
                             float* a, void* stream) {
  clear_error();
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  GGNN_CHECK_ARG(nnz >= 0 && nnz < ((int64_t)1 << 31), "nnz=%lld must be in [0, 2^31)", (long long)nnz);
  CHECK_PTR(row_ptr, "row_ptr");
  if (nnz > 0) CHECK_PTR(col, "col");
  CHECK_PTR(X, "X");
  CHECK_PTR(Wt, "Wt");
  CHECK_OPT_PTR(bias, "bias");
  CHECK_PTR(a, "a");
  return device_status(launch_sparse_step(dt, n_pad, H, E, row_ptr, col, X, Wt, bias, a, as_stream(stream)),
                       "sparse_step");
}

}  // extern "C"

namespace {
ggnn_status check_super(int32_t dt, int32_t n_pad, int32_t H, int32_t E, int32_t s) {
  ggnn_status st = check_common(dt, n_pad, H);
  if (st != GGNN_OK) return st;
  GGNN_CHECK_ARG(n_pad % 64 == 0, "n_pad=%d must be a multiple of 64", n_pad);
  GGNN_CHECK_ARG(E >= 1 && E <= 64, "E=%d must be in [1, 64]", E);
  GGNN_CHECK_ARG(s >= 32 && s <= 128 && s % 32 == 0 && s <= n_pad, "s=%d must be 32, 64, 96 or 128 (<= n_pad)", s);
  return GGNN_OK;
}
}  // namespace

extern "C" {

size_t ggnn_super_workspace_bytes(int32_t n_pad, int32_t H, int32_t E, int32_t s) {
  if (n_pad <= 0 || n_pad % 64 != 0 || !supported_H(H) || E < 1 || E > 64 || s < 32 || s > 128 || s % 32 != 0 ||
      s > n_pad)
    return 0;
  return super_workspace(n_pad, H, E, s);
}

ggnn_status ggnn_super_propagate(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, int32_t s, const void* rows,
                                 const void* cols, const void* X, const void* W, const float* bias, float* a,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  ggnn_status st = check_super(dt, n_pad, H, E, s);
  if (st != GGNN_OK) return st;
  CHECK_PTR(rows, "rows");
  CHECK_PTR(cols, "cols");
  CHECK_PTR(X, "X");
  CHECK_PTR(W, "W");
  CHECK_OPT_PTR(bias, "bias");
  CHECK_PTR(a, "a");
  const size_t need = super_workspace(n_pad, H, E, s);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))
    return fail(GGNN_ERR_WORKSPACE, "super_propagate needs a 16-byte aligned workspace of %zu bytes (got %zu)", need,
                workspace ? workspace_bytes : (size_t)0);
  return device_status(launch_super_fwd(dt, n_pad, H, E, s, rows, cols, X, W, bias, a, workspace, as_stream(stream)),
                       "super_propagate");
}

ggnn_status ggnn_super_propagate_bwd(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t E, int32_t s,
                                     const void* rows, const void* rows_t, const void* cols_t, const void* X,
                                     const void* W, const void* da, float* dX, float* dW, float* dbias,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  ggnn_status st = check_super(dt, n_pad, H, E, s);
  if (st != GGNN_OK) return st;
  CHECK_PTR(rows, "rows");
  CHECK_PTR(rows_t, "rows_t");
  CHECK_PTR(cols_t, "cols_t");
  CHECK_PTR(X, "X");
  CHECK_PTR(W, "W");
  CHECK_PTR(da, "da");
  CHECK_PTR(dX, "dX");
  CHECK_PTR(dW, "dW");
  CHECK_OPT_PTR(dbias, "dbias");
  const size_t need = super_workspace(n_pad, H, E, s);
  if (workspace == nullptr || workspace_bytes < need || !aligned16(workspace))
    return fail(GGNN_ERR_WORKSPACE, "super_propagate_bwd needs a 16-byte aligned workspace of %zu bytes (got %zu)",
                need, workspace ? workspace_bytes : (size_t)0);
  return device_status(launch_super_bwd(dt, n_pad, H, E, s, rows, rows_t, cols_t, X, W, da, dX, dW, dbias, workspace,
                                        as_stream(stream)),
                       "super_propagate_bwd");
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free readout reverse.  Its per-block partial sums live in a
// file-scope device array that the library holds on every device it runs on
// (until the process ends) instead of a caller workspace.  In host code the
// array's name is only a stand-in: its device address on each device is
// looked up once, with that device current, and kept.
// ---------------------------------------------------------------------------
static constexpr size_t kNoAllocScratchBytes = (size_t)GGNN_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device that runs `stream`.
ggnn_status scratch_address(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = hipStreamGetDevice(stream, &dev);
  if (e != hipSuccess) return fail(GGNN_ERR_DEVICE, "device of the stream: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(GGNN_ERR_UNSUPPORTED, "device %d beyond the %d supported", dev,
                                                 kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || p == nullptr)
      return fail(GGNN_ERR_DEVICE, "address of the scratch array on device %d: %s", dev,
                  e != hipSuccess ? hipGetErrorString(e) : "null");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GGNN_OK;
}
}  // namespace

extern "C" {

ggnn_status ggnn_readout_loss_bwd_noalloc(ggnn_dtype dt, int32_t n_pad, int32_t H, int32_t n_cand, const void* X,
                                          const float* w_out, const int32_t* cand_node, const float* dlogit,
                                          float* dX, float* dw_out, float* db_out, void* stream) {
  clear_error();
  ggnn_status st = check_readout_bwd(dt, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out);
  if (st != GGNN_OK) return st;
  const size_t need = readout_bwd_workspace(H, n_cand);
  if (need > kNoAllocScratchBytes)
    return fail(GGNN_ERR_UNSUPPORTED,
                "readout_loss_bwd_noalloc: %d candidates at H=%d need %zu bytes of partial sums, more than the "
                "library's %zu-byte scratch; use ggnn_readout_loss_bwd with a workspace",
                n_cand, H, need, kNoAllocScratchBytes);
  void* part = nullptr;
  st = scratch_address(as_stream(stream), &part);
  if (st != GGNN_OK) return st;
  return device_status(launch_readout_bwd(dt, n_pad, H, n_cand, X, w_out, cand_node, dlogit, dX, dw_out, db_out,
                                          part, as_stream(stream)),
                       "readout_loss_bwd_noalloc");
}

}  // extern "C"
