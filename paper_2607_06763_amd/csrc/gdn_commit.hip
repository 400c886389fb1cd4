// gdn_commit.hip -- conv-state shift of the commit (Sec. 3.4.2: once the
// accepted node is known its path is committed; the state part runs on MFMA
// in gdn_coef.hip).
//
// Grid ceil(C/256) x B: the new conv-state slots are the last three raw
// inputs of (old slots | path root..a).  The kernel runs after the state
// kernel on the same stream, because that kernel reads the old conv state.
#include "gdn_internal.h"

namespace gdn {

struct CommitParams {
  int B, T, Hk, Hv;
  const void* meta;
  const int32_t* accepted;
  const void *q, *k, *v, *alpha, *beta;
  const float* conv_w;
  float* conv_state;
  float* S;
  int32_t* commit_status;
};

// status of the commit of sequence b: tree status, bad accepted slot, or ok
__device__ __forceinline__ int commit_check(const MetaPtrs& m, int b, int T, int a) {
  const int st = m.status[b];
  if (st != GDN_TREE_OK) return st;
  if (a == -1) return GDN_TREE_OK;
  if (a < -1 || a >= T) return GDN_TREE_BAD_ACCEPTED;
  if (m.depth[size_t(b) * T + a] < 0) return GDN_TREE_BAD_ACCEPTED;
  return GDN_TREE_OK;
}

template <typename TIn>
__global__ __launch_bounds__(256) void commit_conv_kernel(CommitParams p, int DK, int DV) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int C = 2 * Hk * DK + Hv * DV;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int a = p.accepted[b];
  if (commit_check(m, b, T, a) != GDN_TREE_OK || a == -1 || c >= C) return;
  const int L = m.depth[size_t(b) * T + a] + 1;
  int n[3];  // path nodes at distance 0, 1, 2 from the accepted slot
  n[0] = a;
  n[1] = L >= 2 ? m.parent[size_t(b) * T + a] : -1;
  n[2] = L >= 3 ? m.parent[size_t(b) * T + n[1]] : -1;
  float* cs = p.conv_state + size_t(b) * 3 * C;
  float old[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) old[s] = cs[size_t(s) * C + c];
  const int nq = Hk * DK;
  float nw[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    if (L + s >= 3) {
      const size_t t = n[2 - s];
      float x;
      if (c < nq)
        x = ld(static_cast<const TIn*>(p.q), (size_t(b) * T + t) * nq + c);
      else if (c < 2 * nq)
        x = ld(static_cast<const TIn*>(p.k), (size_t(b) * T + t) * nq + (c - nq));
      else
        x = ld(static_cast<const TIn*>(p.v), (size_t(b) * T + t) * size_t(Hv) * DV + (c - 2 * nq));
      nw[s] = x;
    } else {
      nw[s] = old[L + s];
    }
  }
#pragma unroll
  for (int s = 0; s < 3; ++s) cs[size_t(s) * C + c] = nw[s];
}

int launch_commit(const CommitArgs& a, hipStream_t stream) {
  // the state (MFMA WY form, gdn_coef.hip), then the conv-state shift, which
  // must run after the state kernel has read the old conv state
  int rc = launch_coef_commit(a, stream);
  if (rc != GDN_OK) return rc;
  CommitParams p;
  p.B = a.B;
  p.T = a.T;
  p.Hk = a.Hk;
  p.Hv = a.Hv;
  p.meta = a.meta;
  p.accepted = a.accepted;
  p.q = a.q;
  p.k = a.k;
  p.v = a.v;
  p.alpha = a.alpha;
  p.beta = a.beta;
  p.conv_w = a.conv_w;
  p.conv_state = a.conv_state;
  p.S = a.S;
  p.commit_status = a.commit_status;
  const int C = 2 * a.Hk * a.dk + a.Hv * a.dv;
  if (a.in_dtype == GDN_BF16)
    hipLaunchKernelGGL((commit_conv_kernel<BF16>), dim3((C + 255) / 256, a.B), dim3(256), 0, stream, p, a.dk, a.dv);
  else
    hipLaunchKernelGGL((commit_conv_kernel<float>), dim3((C + 255) / 256, a.B), dim3(256), 0, stream, p, a.dk, a.dv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "commit conv launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

}  // namespace gdn
