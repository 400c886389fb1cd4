// gdn_commit.hip -- commit of the accepted node (paper Sec. 3.4.2: once the
// accepted leaf is known a single pass replays Eq. 7 along its path and
// writes the state; it is the only state write of the decode step).
//
// Kernel 1 (grid Hv x B, 512 threads): the state loads are issued first; the
// path root..a of the accepted slot a is read off its ancestor bitmask; each
// half of the workgroup featurises half of a chunk of kChunk path nodes (one
// thread per feature channel, width-4 conv window along the path, conv-state
// slots above the root) into LDS, with the key norms reduced across waves;
// each row of S[b][h] (dv rows of dk) lives in the registers of LPR lanes and
// takes one rank-1 step per path node,
//     S_r <- alpha S_r + beta (v_r - alpha (S_r . k)) k^T,
// which is Eq. 7 in the stored orientation S <- alpha S (I - beta k k^T) + beta v k^T.
// The rows are kept as S = gamma * S_stored with gamma the running product of
// alpha, so a step is two FMAs per element (dot and write).
// Kernel 2 (grid ceil(C/256) x B) shifts the conv state: the new slots are
// the last three raw inputs of (old slots | path root..a).  It runs after
// kernel 1 on the same stream because kernel 1 reads the old conv state.
#include "gdn_internal.h"

namespace gdn {

// threads per state workgroup: 512, or one per state element for tiny heads
constexpr int commit_threads(int dk, int dv) { return dk * dv >= 512 ? 512 : dk * dv; }
constexpr int kChunk = 16;   // path nodes featurised per LDS chunk
constexpr int kCMaxT = 128;  // tree slots supported

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

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(commit_threads(DK, DV)) void commit_state_kernel(CommitParams p) {
  constexpr int kCT = commit_threads(DK, DV);
  constexpr int EPT = DV * DK / kCT;  // state elements per thread
  constexpr int LPR = DK / EPT;       // lanes per state row (power of 2)
  constexpr int NCH = DK + DV;        // feature channels: k of key head g, v of head h
  constexpr int HALF = kCT / 2;       // threads per feature half
  constexpr int CPT = (NCH + HALF - 1) / HALF;  // feature channels per thread
  constexpr int MH = kChunk / 2;      // path nodes per half and chunk
  static_assert(EPT >= 1 && (EPT < 4 || EPT % 4 == 0), "state split");
  static_assert(LPR >= 1 && LPR <= 32 && (LPR & (LPR - 1)) == 0, "row lanes");

  __shared__ int s_path[kCMaxT];
  __shared__ int s_dep[kCMaxT];
  __shared__ float s_al[kCMaxT], s_be[kCMaxT];
  __shared__ __align__(16) float s_f[kChunk][NCH];  // conv+SiLU features of a path chunk
  __shared__ float s_part[kChunk][kCT / kWave];     // per-wave partial sums of k^2
  __shared__ float s_inv[kChunk];                   // 1 / ||k|| per path node

  const int h = blockIdx.x, b = blockIdx.y;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int g = h * Hk / Hv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = 2 * Hk * DK + Hv * DV;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);

  // first round of loads: nothing here depends on the accepted slot
  const int a = p.accepted[b];
  const int tree_st = m.status[b];
  int dep_j = -1;
  float al_j = 0.0f, be_j = 0.0f;
  if (tid < T) {
    dep_j = m.depth[size_t(b) * T + tid];
    const size_t ab = (size_t(b) * T + tid) * Hv + h;
    al_j = ld(alpha, ab);
    be_j = ld(beta, ab);
  }
  if (tree_st != GDN_TREE_OK || a < 0 || a >= T) {
    if (h == 0 && tid == 0 && p.commit_status)
      p.commit_status[b] = tree_st != GDN_TREE_OK ? tree_st : (a == -1 ? GDN_TREE_OK : GDN_TREE_BAD_ACCEPTED);
    return;
  }
  const int row = tid / LPR;
  const int col0 = (tid % LPR) * EPT;
  float* Sbh = p.S + (size_t(b) * Hv + h) * size_t(DV) * DK;
  float srow[EPT];  // state rows in registers; the loads overlap the path work
  if constexpr (EPT % 4 == 0) {
#pragma unroll
    for (int e = 0; e < EPT; e += 4) {
      const float4 x = *reinterpret_cast<const float4*>(Sbh + size_t(row) * DK + col0 + e);
      srow[e] = x.x;
      srow[e + 1] = x.y;
      srow[e + 2] = x.z;
      srow[e + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < EPT; ++e) srow[e] = Sbh[size_t(row) * DK + col0 + e];
  }
  if (tid < T) s_dep[tid] = dep_j;
  __syncthreads();
  const int d = s_dep[a];
  if (h == 0 && tid == 0 && p.commit_status)
    p.commit_status[b] = d < 0 ? GDN_TREE_BAD_ACCEPTED : GDN_TREE_OK;
  if (d < 0) return;  // accepted slot is padding

  // second round: the path root..a from the ancestor bitmask of a
  if (tid < T) {
    const uint64_t word = m.anc[(size_t(b) * T + a) * m.W + (tid >> 6)];
    if (tid == a || ((word >> (tid & 63)) & 1ull)) {
      s_path[dep_j] = tid;
      s_al[dep_j] = al_j;
      s_be[dep_j] = be_j;
    }
  }

  // feature channels of this thread: c < DK -> k[g][c], else v[h][c - DK]
  const int half = tid / HALF, ht = tid % HALF;
  const TIn* kin = static_cast<const TIn*>(p.k);
  const TIn* vin = static_cast<const TIn*>(p.v);
  const size_t krow = size_t(Hk) * DK, vrow = size_t(Hv) * DV;
  float wt[CPT][4];
  const TIn* src[CPT];
  size_t sstride[CPT];
  const float* csrc[CPT];
#pragma unroll
  for (int u = 0; u < CPT; ++u) {
    const int c = ht + u * HALF;
    const int cc = c < NCH ? c : 0;
    const int ch = cc < DK ? Hk * DK + g * DK + cc : 2 * Hk * DK + h * DV + (cc - DK);
    src[u] = cc < DK ? kin + size_t(b) * T * krow + size_t(g) * DK + cc
                     : vin + size_t(b) * T * vrow + size_t(h) * DV + (cc - DK);
    sstride[u] = cc < DK ? krow : vrow;
    csrc[u] = p.conv_state + size_t(b) * 3 * C + ch;
    const float4 w4 = *reinterpret_cast<const float4*>(p.conv_w + size_t(ch) * 4);
    wt[u][0] = w4.x;
    wt[u][1] = w4.y;
    wt[u][2] = w4.z;
    wt[u][3] = w4.w;
  }
  __syncthreads();  // s_path ready

  // S_true = gamma * srow: one step costs one FMA for S.k and one for the
  // rank-1 write, S_true <- alpha S_true + c k  <=>  srow += c / (alpha gamma) k
  float gamma = 1.0f;
  for (int base = 0; base <= d; base += kChunk) {
    const int cnt = (d - base + 1) < kChunk ? (d - base + 1) : kChunk;
    // this half featurises path nodes base + half * MH .. + MH - 1; the
    // window before its first node comes from the path or the conv state
    const int m0 = base + half * MH;
    float ksq[MH];
#pragma unroll
    for (int mr = 0; mr < MH; ++mr) ksq[mr] = 0.0f;
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int c = ht + u * HALF;
      float xs[MH + 3];
#pragma unroll
      for (int q = 0; q < MH + 3; ++q) {
        const int mi = m0 - 3 + q;  // path index of this window element
        xs[q] = mi < 0 ? csrc[u][size_t(3 + mi) * C]
                       : (mi <= d ? ld(src[u], size_t(s_path[mi]) * sstride[u]) : 0.0f);
      }
#pragma unroll
      for (int mr = 0; mr < MH; ++mr) {
        const float y = silu(wt[u][0] * xs[mr] + wt[u][1] * xs[mr + 1] + wt[u][2] * xs[mr + 2] +
                             wt[u][3] * xs[mr + 3]);
        if (c < NCH) s_f[half * MH + mr][c] = y;
        if (c < DK) ksq[mr] += y * y;
      }
    }
    // ||k||^2 per path node: wave sums, then across the waves of the half
#pragma unroll
    for (int mr = 0; mr < MH; ++mr) {
      const float v = wave_sum(ksq[mr]);
      if (lane == 0) s_part[half * MH + mr][wave % (HALF / kWave)] = v;
    }
    __syncthreads();
    if (tid < kChunk) {
      float v = 0.0f;
#pragma unroll
      for (int wv = 0; wv < HALF / kWave; ++wv) v += s_part[tid][wv];
      s_inv[tid] = rsqrt_hw(v + 1e-6f);
    }
    __syncthreads();
    for (int mr = 0; mr < cnt; ++mr) {
      const int mi = base + mr;
      const float al = s_al[mi], be = s_be[mi], inv = s_inv[mr];
      float kk[EPT];  // un-normalised key; 1 / ||k|| is folded into the scalars
      if constexpr (EPT % 4 == 0) {
#pragma unroll
        for (int e = 0; e < EPT; e += 4) {
          const float4 x = *reinterpret_cast<const float4*>(&s_f[mr][col0 + e]);
          kk[e] = x.x;
          kk[e + 1] = x.y;
          kk[e + 2] = x.z;
          kk[e + 3] = x.w;
        }
      } else {
#pragma unroll
        for (int e = 0; e < EPT; ++e) kk[e] = s_f[mr][col0 + e];
      }
      float u0 = 0.0f, u1 = 0.0f;
#pragma unroll
      for (int e = 0; e + 1 < EPT; e += 2) {
        u0 += srow[e] * kk[e];
        u1 += srow[e + 1] * kk[e + 1];
      }
      if (EPT & 1) u0 += srow[EPT - 1] * kk[EPT - 1];
      const float uu = group_sum<LPR>(u0 + u1) * inv;  // S_stored . k_hat
      // c = beta (v_r - alpha S_true.k_hat), scaled into the stored frame and
      // multiplied by 1 / ||k|| so that it applies to the raw key
      const float ag = al * gamma;
      const float c = be * (s_f[mr][DK + row] - ag * uu) * __builtin_amdgcn_rcpf(ag) * inv;
#pragma unroll
      for (int e = 0; e < EPT; ++e) srow[e] += c * kk[e];
      gamma = ag;
      if (gamma < 0x1p-60f) {  // keep the stored frame in range (uniform branch)
#pragma unroll
        for (int e = 0; e < EPT; ++e) srow[e] *= gamma;
        gamma = 1.0f;
      }
    }
    __syncthreads();  // chunk features consumed
  }
  if constexpr (EPT % 4 == 0) {
#pragma unroll
    for (int e = 0; e < EPT; e += 4)
      *reinterpret_cast<float4*>(Sbh + size_t(row) * DK + col0 + e) =
          make_float4(srow[e] * gamma, srow[e + 1] * gamma, srow[e + 2] * gamma, srow[e + 3] * gamma);
  } else {
#pragma unroll
    for (int e = 0; e < EPT; ++e) Sbh[size_t(row) * DK + col0 + e] = srow[e] * gamma;
  }
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
  p.conv_state = a.conv_state;
  p.S = a.S;
  p.commit_status = a.commit_status;
  if (a.in_dtype == GDN_BF16) return commit_dk<BF16>(a, p, stream);
  return commit_dk<float>(a, p, stream);
}

}  // namespace gdn
