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
#include "gdn_internal.h"

namespace gdn {

// threads per state workgroup: 512, or one per state element for tiny heads
constexpr int commit_threads(int dk, int dv) { return dk * dv >= 512 ? 512 : dk * dv; }
constexpr int kCMaxT = 512;    // tree slots supported
constexpr int kMH = kMC / 2;   // path nodes per feature half

struct CommitParams {
  int B, T, Hk, Hv;
  const void* meta;
  const int32_t* accepted;
  const void *q, *k, *v, *alpha, *beta;
  const float* conv_w;
  const float* cs_in;  // conv state before the commit
  float* cs_out;       // conv state after it (may equal cs_in)
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

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(commit_threads(DK, DV)) void commit_state_kernel(CommitParams p) {
  constexpr int kCT = commit_threads(DK, DV);
  constexpr int EPT = DV * DK / kCT;  // state elements per thread
  constexpr int R = EPT >= 16 ? 2 : 1;  // rows per thread (rows q and q + RS)
  constexpr int CPT = EPT / R;          // columns per thread and row
  constexpr int LPR = DK / CPT;         // lanes per state row (power of 2)
  constexpr int RS = DV / R;
  static_assert(EPT >= 1 && (EPT < 4 || EPT % 4 == 0) && DV % R == 0, "state split");
  static_assert(LPR >= 1 && LPR <= 32 && (LPR & (LPR - 1)) == 0, "row lanes");
  static_assert(2 * (DK + DV) <= kCT, "one feature task per thread");

  __shared__ int s_path[kCMaxT];
  __shared__ int s_dep[kCMaxT];
  __shared__ float s_al[kCMaxT], s_be[kCMaxT];    // gates by path index
  __shared__ __align__(16) float s_fk[kMC][DK];  // SiLU(conv) keys of a path chunk (unnormalised)
  __shared__ __align__(16) float s_fv[kMC][DV];  // SiLU(conv) values of a path chunk
  __shared__ float s_inv[kMC];                    // 1 / ||k|| per path node of the chunk

  const int h = blockIdx.x, b = blockIdx.y;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int g = h * Hk / Hv;
  const int tid = threadIdx.x;
  const int C = 2 * Hk * DK + Hv * DV;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);

  // ---- first load wave: status, depths and gates of this thread's slots (raw
  //      gates are converted only once the path is known)
  constexpr int kSl = (kCMaxT + kCT - 1) / kCT;  // slots per thread
  const int a = p.accepted[b];
  const int tree_st = m.status[b];
  int dep[kSl];
  TIn alr[kSl], ber[kSl];
#pragma unroll
  for (int sl = 0; sl < kSl; ++sl) {
    const int j = tid + sl * kCT;
    const int jj = j < T ? j : T - 1;
    dep[sl] = m.depth[size_t(b) * T + jj];
    alr[sl] = alpha[(size_t(b) * T + jj) * Hv + h];
    ber[sl] = beta[(size_t(b) * T + jj) * Hv + h];
  }
  if (tree_st != GDN_TREE_OK || a < 0 || a >= T) {
    if (h == 0 && tid == 0 && p.commit_status)
      p.commit_status[b] = tree_st != GDN_TREE_OK ? tree_st : (a == -1 ? GDN_TREE_OK : GDN_TREE_BAD_ACCEPTED);
    return;
  }
  // ---- second load wave: the ancestor bitmask of a -> the path root..a
  uint64_t word[kSl];
#pragma unroll
  for (int sl = 0; sl < kSl; ++sl) {
    const int j = tid + sl * kCT;
    word[sl] = m.anc[(size_t(b) * T + a) * m.W + ((j < T ? j : T - 1) >> 6)];
    if (j < T) s_dep[j] = dep[sl];
  }
  __syncthreads();
  const int d = s_dep[a];
  if (h == 0 && tid == 0 && p.commit_status)
    p.commit_status[b] = d < 0 ? GDN_TREE_BAD_ACCEPTED : GDN_TREE_OK;
  if (d < 0) return;  // accepted slot is padding
#pragma unroll
  for (int sl = 0; sl < kSl; ++sl) {
    const int j = tid + sl * kCT;
    if (j < T && (j == a || ((word[sl] >> (j & 63)) & 1ull))) {
      s_path[dep[sl]] = j;
      s_al[dep[sl]] = to_f32(alr[sl]);
      s_be[dep[sl]] = to_f32(ber[sl]);
    }
  }
  __syncthreads();
  const int L = d + 1;  // path length

  // ---- feature task of this thread: value channel (tid < 2 DV) or key
  //      channel (2 DV <= tid < 2 (DV + DK)); fhalf picks the half of a chunk
  const bool vtask = tid < 2 * DV;
  const bool ktask = !vtask && tid < 2 * (DV + DK);
  const int tt = vtask ? tid : tid - 2 * DV;
  const int fc = vtask ? tt % DV : tt % DK;
  const int fhalf = vtask ? tt / DV : tt / DK;
  const int fch = vtask ? 2 * Hk * DK + h * DV + fc : Hk * DK + g * DK + fc;  // conv channel
  const TIn* fsrc = vtask ? static_cast<const TIn*>(p.v) + size_t(b) * T * Hv * DV + size_t(h) * DV + fc
                          : static_cast<const TIn*>(p.k) + size_t(b) * T * Hk * DK + size_t(g) * DK + fc;
  const size_t fstride = vtask ? size_t(Hv) * DV : size_t(Hk) * DK;
  const float* fcs = p.cs_in + size_t(b) * 3 * C + fch;
  FeatWindow<TIn, kMH> win;
  if (vtask || ktask) win.load(fsrc, fstride, fcs, C, p.conv_w + size_t(fch) * 4, s_path, fhalf * kMH, L);

  // ---- the state rows load behind the first windows
  const int row = tid / LPR;
  const int col0 = (tid % LPR) * CPT;
  float* Sbh = p.S + (size_t(b) * Hv + h) * size_t(DV) * DK + size_t(row) * DK + col0;
  float srow[EPT];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float piece[CPT];
    ld_slice<CPT>(Sbh + size_t(i) * RS * DK, piece);
#pragma unroll
    for (int e = 0; e < CPT; ++e) srow[i * CPT + e] = piece[e];
  }

  // S_true = gamma * srow: one step costs one FMA for S.k and one for the
  // rank-1 write, S_true <- alpha S_true + c k  <=>  srow += c / (alpha gamma) k
  float gamma = 1.0f;
  for (int base = 0; base < L; base += kMC) {
    if (base > 0 && (vtask || ktask))  // long paths: later chunks load here
      win.load(fsrc, fstride, fcs, C, p.conv_w + size_t(fch) * 4, s_path, base + fhalf * kMH, L);
    // features of the chunk (window element q is path node m0 - 3 + q)
    if (vtask || ktask) {
      const int m0 = base + fhalf * kMH;
#pragma unroll
      for (int mr = 0; mr < kMH; ++mr) {
        const float y = silu(win.w.x * win.x(mr, m0, L) + win.w.y * win.x(mr + 1, m0, L) +
                             win.w.z * win.x(mr + 2, m0, L) + win.w.w * win.x(mr + 3, m0, L));
        if (vtask)
          s_fv[fhalf * kMH + mr][fc] = y;
        else
          s_fk[fhalf * kMH + mr][fc] = y;
      }
    }
    __syncthreads();
    // key norms: 16 lanes per path node, DK / 16 channels per lane
#pragma unroll
    for (int nd0 = 0; nd0 < kMC; nd0 += kCT / 16) {
      constexpr int CPL = DK / 16;
      const int nd = nd0 + (tid >> 4), ln = tid & 15;
      float ss = 0.0f;
      if (nd < kMC) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const float y = s_fk[nd][ln * CPL + c];
          ss += y * y;
        }
      }
      ss = group_sum<16>(ss);
      if (nd < kMC && ln == 0) s_inv[nd] = rsqrt_hw(ss + 1e-6f);
    }
    __syncthreads();
    const int cnt = L - base < kMC ? L - base : kMC;
    for (int mr = 0; mr < cnt; ++mr) {
      float kk[CPT], vr[R];
      ld_slice<CPT>(&s_fk[mr][col0], kk);
#pragma unroll
      for (int i = 0; i < R; ++i) vr[i] = s_fv[mr][row + i * RS];
      gamma = replay_rows<R, CPT, LPR>(srow, kk, vr, s_al[base + mr], s_be[base + mr], s_inv[mr], gamma);
    }
    __syncthreads();  // chunk features consumed
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float* dst = Sbh + size_t(i) * RS * DK;
    if constexpr (CPT % 4 == 0) {
#pragma unroll
      for (int e = 0; e < CPT; e += 4)
        *reinterpret_cast<float4*>(dst + e) =
            make_float4(srow[i * CPT + e] * gamma, srow[i * CPT + e + 1] * gamma, srow[i * CPT + e + 2] * gamma,
                        srow[i * CPT + e + 3] * gamma);
    } else {
#pragma unroll
      for (int e = 0; e < CPT; ++e) dst[e] = srow[i * CPT + e] * gamma;
    }
  }
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
