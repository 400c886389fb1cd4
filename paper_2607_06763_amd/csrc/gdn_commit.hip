// gdn_commit.hip -- commit of the accepted node (Sec. 3.4.2).  Verification
// leaves the cached state untouched; after the decoder has chosen the
// accepted slot, these kernels advance S and the conv state over the slot's
// path root..a (Eq. 7 per path node), the one place the state changes.
//
// Kernel 1 (grid Hv x B, 512 threads): the path root..a of the accepted slot
// a is read off its ancestor bitmask; one thread per (feature channel, half
// of a chunk of 32 path nodes) slides the width-4 conv window along the path
// (conv-state slots above the root) into LDS, its raw inputs loaded before
// the state rows; the key norms are reduced per path node;
// each row of S[b][h] (dv rows of dk) lives in the registers of LPR lanes
// (a thread holds pieces of R rows that share the key slice) and takes one
// rank-1 step per path node,
//     S_r <- alpha S_r + beta (v_r - alpha (S_r . k)) k^T,
// which is Eq. 7 in the stored orientation S <- alpha S (I - beta k k^T) + beta v k^T.
// The rows are kept as S = gamma * S_stored with gamma the running product of
// alpha, so a step is two FMAs per element (dot and write); when gamma would
// fall below 2^-60 (or alpha is 0) the rows are first rescaled to the true
// frame, so no step divides by a vanishing decay (replay_rows).  Paths of up
// to 512 nodes: the path is read off the bitmask (up to 8 words) in one load
// wave, and features are built in chunks of 32 path nodes.
// Kernel 2 (grid ceil(C/256) x B) shifts the conv state: the new slots are
// the last three raw inputs of (old slots | path root..a).  It runs after
// kernel 1 on the same stream because kernel 1 reads the old conv state; it
// may write to a separate output buffer (the step above 128 slots), which
// then also receives the unchanged slots of sequences that commit nothing.
#include "gdn_commit_rows.h"

namespace gdn {

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(commit_threads(DK, DV)) void commit_state_kernel(CommitParams p) {
  constexpr int kCT = commit_threads(DK, DV);
  using CS = CommitSplit<DK, DV, kCT>;
  __shared__ __align__(16) unsigned char s_lds[commit_lds_bytes<DK, DV>()];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  float srow[CS::EPT];
  if (commit_rows<DK, DV, TIn, kCT, false>(p, b, h, tid, commit_lds<DK, DV>(s_lds), srow))
    store_rows<DK, DV, kCT>(p.S, b, h, p.Hv, tid, srow);
}

template <typename TIn>
__global__ __launch_bounds__(256) void commit_conv_kernel(CommitParams p, int DK, int DV) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int C = 2 * Hk * DK + Hv * DV;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  if (c >= C) return;
  const int a = p.accepted[b];
  const float* ci = p.cs_in + size_t(b) * 3 * C;
  float* co = p.cs_out + size_t(b) * 3 * C;
  float old[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) old[s] = ci[size_t(s) * C + c];
  if (commit_check(m, b, T, a) != GDN_TREE_OK || a == -1) {  // nothing committed
    if (co != ci) {
#pragma unroll
      for (int s = 0; s < 3; ++s) co[size_t(s) * C + c] = old[s];
    }
    return;
  }
  const int L = m.depth[size_t(b) * T + a] + 1;
  int n[3];  // path nodes at distance 0, 1, 2 from the accepted slot
  n[0] = a;
  n[1] = L >= 2 ? m.parent[size_t(b) * T + a] : -1;
  n[2] = L >= 3 ? m.parent[size_t(b) * T + n[1]] : -1;
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
  for (int s = 0; s < 3; ++s) co[size_t(s) * C + c] = nw[s];
}

template <int DK, int DV, typename TIn>
static int launch_commit_t(const CommitParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((commit_state_kernel<DK, DV, TIn>), dim3(p.Hv, p.B), dim3(commit_threads(DK, DV)), 0,
                     stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "commit launch: %s", hipGetErrorString(e));
  const int C = 2 * p.Hk * DK + p.Hv * DV;
  hipLaunchKernelGGL((commit_conv_kernel<TIn>), dim3((C + 255) / 256, p.B), dim3(256), 0, stream, p,
                     DK, DV);
  e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "commit conv launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

template <int DK, typename TIn>
static int commit_dv(const CommitArgs& a, const CommitParams& p, hipStream_t s) {
  switch (a.dv) {
    case 16: return launch_commit_t<DK, 16, TIn>(p, s);
    case 32: return launch_commit_t<DK, 32, TIn>(p, s);
    case 64: return launch_commit_t<DK, 64, TIn>(p, s);
    case 128: return launch_commit_t<DK, 128, TIn>(p, s);
  }
  return set_error(GDN_EUNSUPPORTED, "commit: dv=%d unsupported", a.dv);
}

template <typename TIn>
static int commit_dk(const CommitArgs& a, const CommitParams& p, hipStream_t s) {
  switch (a.dk) {
    case 16: return commit_dv<16, TIn>(a, p, s);
    case 32: return commit_dv<32, TIn>(a, p, s);
    case 64: return commit_dv<64, TIn>(a, p, s);
    case 128: return commit_dv<128, TIn>(a, p, s);
  }
  return set_error(GDN_EUNSUPPORTED, "commit: dk=%d unsupported", a.dk);
}

int launch_commit_conv(const CommitParams& p, int dk, int dv, int in_dtype, hipStream_t stream) {
  const int C = 2 * p.Hk * dk + p.Hv * dv;
  if (in_dtype == GDN_BF16)
    hipLaunchKernelGGL((commit_conv_kernel<BF16>), dim3((C + 255) / 256, p.B), dim3(256), 0, stream, p, dk, dv);
  else
    hipLaunchKernelGGL((commit_conv_kernel<float>), dim3((C + 255) / 256, p.B), dim3(256), 0, stream, p, dk, dv);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "commit conv launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

int launch_commit(const CommitArgs& a, hipStream_t stream) {
  if (a.T > kCMaxT) return set_error(GDN_EUNSUPPORTED, "commit: T=%d exceeds %d", a.T, kCMaxT);
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
  p.cs_in = a.conv_state_in ? a.conv_state_in : a.conv_state;
  p.cs_out = a.conv_state;
  p.S = a.S;
  p.commit_status = a.commit_status;
  if (a.in_dtype == GDN_BF16) return commit_dk<BF16>(a, p, stream);
  return commit_dk<float>(a, p, stream);
}

}  // namespace gdn
