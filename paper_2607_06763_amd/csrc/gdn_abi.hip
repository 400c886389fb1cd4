// gdn_abi.hip -- the extern "C" boundary of libgdntree (declared in
// include/gdn_tree.h): argument validation on the host, dispatch to the
// templated kernel launchers, and the thread-local error message.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <set>
#include <utility>

#include "gdn_internal.h"

namespace gdn {

static thread_local char g_err[512] = "";

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ensure_dynamic_lds(const void* fn, int bytes, const char* who) {
  static std::mutex mu;
  static std::set<std::pair<const void*, int>> done;  // (kernel, device)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(GDN_EHIP, "%s: hipGetDevice failed", who);
  std::lock_guard<std::mutex> lock(mu);
  if (done.count({fn, dev})) return GDN_OK;
  const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return set_error(GDN_EHIP, "%s: LDS attribute: %s", who, hipGetErrorString(e));
  done.insert({fn, dev});
  return GDN_OK;
}

static bool head_dim_ok(int d) { return d == 16 || d == 32 || d == 64 || d == 128; }

// Shape checks shared by verify and commit.
static int check_dims(const gdn_dims* d, const char* who) {
  if (!d) return set_error(GDN_EINVAL, "%s: dims is NULL", who);
  if (d->B < 0 || d->T < 0 || d->Hk < 1 || d->Hv < 1)
    return set_error(GDN_EINVAL, "%s: bad sizes B=%d T=%d Hk=%d Hv=%d", who, d->B, d->T, d->Hk,
                     d->Hv);
  if (d->Hv % d->Hk != 0)
    return set_error(GDN_EINVAL, "%s: Hv=%d is not a multiple of Hk=%d", who, d->Hv, d->Hk);
  if (d->in_dtype != GDN_F32 && d->in_dtype != GDN_BF16)
    return set_error(GDN_EINVAL, "%s: in_dtype=%d", who, d->in_dtype);
  if (!(d->scale >= 0.0f) || isinf(d->scale))
    return set_error(GDN_EINVAL, "%s: scale must be finite and >= 0", who);
  if (!head_dim_ok(d->dk) || !head_dim_ok(d->dv))
    return set_error(GDN_EUNSUPPORTED, "%s: dk=%d dv=%d (supported 16, 32, 64, 128)", who, d->dk,
                     d->dv);
  if (d->T > GDN_MAX_T) return set_error(GDN_EUNSUPPORTED, "%s: T=%d > %d", who, d->T, GDN_MAX_T);
  return GDN_OK;
}

// Verification at any supported T: the LDS-resident kernel up to 128 slots,
// the feature workspace + gathered pull-back above.
static int verify_any(const VerifyArgs& a, hipStream_t stream) {
  if (a.T <= kSmallMaxT) return launch_verify(a, stream);
  const size_t bytes = large_workspace_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv);
  int rc = GDN_OK;
  void* ws = stream_workspace(bytes, stream, &rc);
  if (!ws) return rc;
  return launch_verify_large(a, ws, bytes, stream);
}

}  // namespace gdn

using namespace gdn;

extern "C" {

size_t gdn_tree_meta_bytes(int32_t B, int32_t T) {
  if (B <= 0 || T <= 0) return 0;
  return meta_layout(B, T).total;
}

int gdn_tree_prepare(const gdn_dims* dims, const int32_t* parent, void* meta,
                     int32_t* tree_status, hipStream_t stream) {
  if (!dims) return set_error(GDN_EINVAL, "prepare: dims is NULL");
  if (dims->B < 0 || dims->T < 0)
    return set_error(GDN_EINVAL, "prepare: bad sizes B=%d T=%d", dims->B, dims->T);
  if (dims->T > GDN_MAX_T)
    return set_error(GDN_EUNSUPPORTED, "prepare: T=%d > %d", dims->T, GDN_MAX_T);
  if (dims->B == 0 || dims->T == 0) return GDN_OK;
  if (!parent || !meta) return set_error(GDN_EINVAL, "prepare: NULL parent or meta");
  return launch_prepare(dims->B, dims->T, parent, meta, tree_status, stream);
}

int gdn_tree_verify(const gdn_dims* dims, const void* meta, const void* q, const void* k,
                    const void* v, const void* alpha, const void* beta, const float* conv_w,
                    const float* conv_state, const float* S0, float* out, hipStream_t stream) {
  int rc = check_dims(dims, "verify");
  if (rc != GDN_OK) return rc;
  if (dims->B == 0 || dims->T == 0) return GDN_OK;
  if (!meta || !q || !k || !v || !alpha || !beta || !conv_w || !conv_state || !S0 || !out)
    return set_error(GDN_EINVAL, "verify: NULL tensor pointer");
  VerifyArgs a;
  a.B = dims->B;
  a.T = dims->T;
  a.Hk = dims->Hk;
  a.Hv = dims->Hv;
  a.dk = dims->dk;
  a.dv = dims->dv;
  a.in_dtype = dims->in_dtype;
  a.scale = dims->scale > 0.0f ? dims->scale : 1.0f / sqrtf(float(dims->dk));
  a.meta = meta;
  a.q = q;
  a.k = k;
  a.v = v;
  a.alpha = alpha;
  a.beta = beta;
  a.conv_w = conv_w;
  a.conv_state = conv_state;
  a.S0 = S0;
  a.out = out;
  return verify_any(a, stream);
}

int gdn_tree_verify_noalloc(const gdn_dims* dims, const void* meta, const void* q, const void* k,
                            const void* v, const void* alpha, const void* beta, const float* conv_w,
                            const float* conv_state, const float* S0, float* out, hipStream_t stream) {
  int rc = check_dims(dims, "verify_noalloc");
  if (rc != GDN_OK) return rc;
  if (dims->B == 0 || dims->T == 0) return GDN_OK;
  const size_t need = dims->T > kSmallMaxT ? large_workspace_bytes(dims->B, dims->T, dims->Hk, dims->Hv,
                                                                   dims->dk, dims->dv)
                                           : 0;
  if (need > size_t(GDN_NOALLOC_SCRATCH_BYTES))
    return set_error(GDN_EUNSUPPORTED, "verify_noalloc: B=%d T=%d needs %zu workspace bytes, above %zu",
                     dims->B, dims->T, need, size_t(GDN_NOALLOC_SCRATCH_BYTES));
  if (!meta || !q || !k || !v || !alpha || !beta || !conv_w || !conv_state || !S0 || !out)
    return set_error(GDN_EINVAL, "verify_noalloc: NULL tensor pointer");
  VerifyArgs a;
  a.B = dims->B;
  a.T = dims->T;
  a.Hk = dims->Hk;
  a.Hv = dims->Hv;
  a.dk = dims->dk;
  a.dv = dims->dv;
  a.in_dtype = dims->in_dtype;
  a.scale = dims->scale > 0.0f ? dims->scale : 1.0f / sqrtf(float(dims->dk));
  a.meta = meta;
  a.q = q;
  a.k = k;
  a.v = v;
  a.alpha = alpha;
  a.beta = beta;
  a.conv_w = conv_w;
  a.conv_state = conv_state;
  a.S0 = S0;
  a.out = out;
  return launch_verify_noalloc(a, stream);
}

int gdn_tree_verify_chunked(const gdn_dims* dims, const void* meta, const void* q, const void* k,
                            const void* v, const void* alpha, const void* beta, const float* conv_w,
                            const float* conv_state, const float* S0, float* out, hipStream_t stream) {
  int rc = check_dims(dims, "verify_chunked");
  if (rc != GDN_OK) return rc;
  if (dims->B == 0 || dims->T == 0) return GDN_OK;
  if (!meta || !q || !k || !v || !alpha || !beta || !conv_w || !conv_state || !S0 || !out)
    return set_error(GDN_EINVAL, "verify_chunked: NULL tensor pointer");
  VerifyArgs a;
  a.B = dims->B;
  a.T = dims->T;
  a.Hk = dims->Hk;
  a.Hv = dims->Hv;
  a.dk = dims->dk;
  a.dv = dims->dv;
  a.in_dtype = dims->in_dtype;
  a.scale = dims->scale > 0.0f ? dims->scale : 1.0f / sqrtf(float(dims->dk));
  a.meta = meta;
  a.q = q;
  a.k = k;
  a.v = v;
  a.alpha = alpha;
  a.beta = beta;
  a.conv_w = conv_w;
  a.conv_state = conv_state;
  a.S0 = S0;
  a.out = out;
  const size_t bytes = chunked_workspace_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv);
  void* ws = stream_workspace(bytes, stream, &rc);
  if (!ws) return rc;
  return launch_verify_chunked(a, ws, bytes, stream);
}

int gdn_tree_commit(const gdn_dims* dims, const void* meta, const int32_t* accepted,
                    const void* q, const void* k, const void* v, const void* alpha,
                    const void* beta, const float* conv_w, float* conv_state, float* S,
                    int32_t* commit_status, hipStream_t stream) {
  int rc = check_dims(dims, "commit");
  if (rc != GDN_OK) return rc;
  if (dims->B == 0 || dims->T == 0) return GDN_OK;
  if (!meta || !accepted || !q || !k || !v || !alpha || !beta || !conv_w || !conv_state || !S)
    return set_error(GDN_EINVAL, "commit: NULL tensor pointer");
  CommitArgs a;
  a.B = dims->B;
  a.T = dims->T;
  a.Hk = dims->Hk;
  a.Hv = dims->Hv;
  a.dk = dims->dk;
  a.dv = dims->dv;
  a.in_dtype = dims->in_dtype;
  a.meta = meta;
  a.accepted = accepted;
  a.q = q;
  a.k = k;
  a.v = v;
  a.alpha = alpha;
  a.beta = beta;
  a.conv_w = conv_w;
  a.conv_state = conv_state;
  a.S = S;
  a.commit_status = commit_status;
  return launch_commit(a, stream);
}

int gdn_tree_step(const gdn_dims* dims, const void* prev_meta, const int32_t* prev_accepted,
                  const void* prev_q, const void* prev_k, const void* prev_v, const void* prev_alpha,
                  const void* prev_beta, int32_t* commit_status, const void* meta, const void* q,
                  const void* k, const void* v, const void* alpha, const void* beta,
                  const float* conv_w, const float* conv_state, float* conv_state_out, float* S,
                  float* out, hipStream_t stream) {
  int rc = check_dims(dims, "step");
  if (rc != GDN_OK) return rc;
  if (dims->B == 0 || dims->T == 0) return GDN_OK;
  if (!prev_meta || !prev_accepted || !prev_q || !prev_k || !prev_v || !prev_alpha || !prev_beta ||
      !meta || !q || !k || !v || !alpha || !beta || !conv_w || !conv_state || !conv_state_out || !S ||
      !out)
    return set_error(GDN_EINVAL, "step: NULL tensor pointer");
  const size_t cs_bytes =
      size_t(dims->B) * 3 * (2 * size_t(dims->Hk) * dims->dk + size_t(dims->Hv) * dims->dv) * sizeof(float);
  const char* ci = reinterpret_cast<const char*>(conv_state);
  const char* co = reinterpret_cast<const char*>(conv_state_out);
  if (ci < co + cs_bytes && co < ci + cs_bytes)
    return set_error(GDN_EINVAL, "step: conv_state and conv_state_out overlap");
  VerifyArgs a;
  a.B = dims->B;
  a.T = dims->T;
  a.Hk = dims->Hk;
  a.Hv = dims->Hv;
  a.dk = dims->dk;
  a.dv = dims->dv;
  a.in_dtype = dims->in_dtype;
  a.scale = dims->scale > 0.0f ? dims->scale : 1.0f / sqrtf(float(dims->dk));
  a.meta = meta;
  a.q = q;
  a.k = k;
  a.v = v;
  a.alpha = alpha;
  a.beta = beta;
  a.conv_w = conv_w;
  a.conv_state = conv_state;
  a.S0 = S;
  a.out = out;
  a.fused = true;
  a.pmeta = prev_meta;
  a.paccepted = prev_accepted;
  a.pq = prev_q;
  a.pk = prev_k;
  a.pv = prev_v;
  a.palpha = prev_alpha;
  a.pbeta = prev_beta;
  a.conv_state_out = conv_state_out;
  a.S = S;
  a.commit_status = commit_status;
  // up to 128 slots the verify kernel commits; above, the pull-back commits
  // each head's rows (heads of at least 512 state elements)
  if (a.T <= kSmallMaxT || a.dk * a.dv >= 512) return verify_any(a, stream);
  // tiny heads above 128 slots: the commit kernels (conv state into
  // conv_state_out), then the verification against the committed state
  CommitArgs c;
  c.B = a.B;
  c.T = a.T;
  c.Hk = a.Hk;
  c.Hv = a.Hv;
  c.dk = a.dk;
  c.dv = a.dv;
  c.in_dtype = a.in_dtype;
  c.meta = prev_meta;
  c.accepted = prev_accepted;
  c.q = prev_q;
  c.k = prev_k;
  c.v = prev_v;
  c.alpha = prev_alpha;
  c.beta = prev_beta;
  c.conv_w = conv_w;
  c.conv_state = conv_state_out;
  c.conv_state_in = conv_state;
  c.S = S;
  c.commit_status = commit_status;
  rc = launch_commit(c, stream);
  if (rc != GDN_OK) return rc;
  VerifyArgs v2 = a;
  v2.fused = false;
  v2.conv_state = conv_state_out;
  return verify_any(v2, stream);
}

const char* gdn_last_error(void) { return g_err; }

const char* gdn_version(void) { return "gdntree 0.1 (gfx950)"; }

}  // extern "C"
