// gdn_commit.hip -- commit of the accepted node (paper Sec. 3.4.2: once the
// accepted leaf is known a single pass replays Eq. 7 along its path and
// writes the state; it is the only state write of the decode step).
//
// Kernel 1 (grid Hv x B, 256 threads): the path root..a of the accepted slot
// a is read off its ancestor bitmask; the conv + SiLU + L2-norm features of
// the path nodes are computed in chunks of kChunk nodes into LDS; each row of
// S[b][h] (dv rows of dk) lives in the registers of LPR lanes and takes one
// rank-1 step per path node,
//     S_r <- alpha S_r + beta (v_r - alpha (S_r . k)) k^T,
// which is Eq. 7 in the stored orientation S <- alpha S (I - beta k k^T) + beta v k^T.
// Kernel 2 (grid ceil(C/256) x B) shifts the conv state: the new slots are
// the last three raw inputs of (old slots | path root..a).  It runs after
// kernel 1 on the same stream because kernel 1 reads the old conv state.
#include "gdn_internal.h"

namespace gdn {

constexpr int kCT = 256;     // threads per state workgroup
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
__global__ __launch_bounds__(kCT) void commit_state_kernel(CommitParams p) {
  constexpr int EPT = DV * DK / kCT;       // state elements per thread
  constexpr int LPR = DK / EPT;            // lanes per state row (power of 2)
  constexpr int KPL = DK / kWave > 0 ? DK / kWave : 1;  // k channels per lane
  constexpr int VPL = DV / kWave > 0 ? DV / kWave : 1;  // v channels per lane
  static_assert(EPT >= 1 && (EPT < 4 || EPT % 4 == 0), "state split");
  static_assert(LPR >= 1 && LPR <= kWave && (LPR & (LPR - 1)) == 0, "row lanes");

  __shared__ int s_path[kCMaxT];
  __shared__ float s_al[kCMaxT], s_be[kCMaxT];
  __shared__ __align__(16) float s_k[kChunk][DK];
  __shared__ float s_v[kChunk][DV];

  const int h = blockIdx.x, b = blockIdx.y;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int g = h * Hk / Hv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = 2 * Hk * DK + Hv * DV;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int a = p.accepted[b];
  const int st = commit_check(m, b, T, a);
  if (h == 0 && tid == 0 && p.commit_status) p.commit_status[b] = st;
  if (st != GDN_TREE_OK || a == -1) return;

  const int d = m.depth[size_t(b) * T + a];
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  for (int j = tid; j < T; j += kCT) {
    const uint64_t word = m.anc[(size_t(b) * T + a) * m.W + (j >> 6)];
    if (j == a || ((word >> (j & 63)) & 1ull)) {
      const int dj = m.depth[size_t(b) * T + j];
      s_path[dj] = j;
      const size_t ab = (size_t(b) * T + j) * Hv + h;
      s_al[dj] = ld(alpha, ab);
      s_be[dj] = ld(beta, ab);
    }
  }

  // state rows in registers
  const int row = tid / LPR;
  const int col0 = (tid % LPR) * EPT;
  float* Sbh = p.S + (size_t(b) * Hv + h) * size_t(DV) * DK;
  float srow[EPT];
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
  __syncthreads();

  const TIn* kin = static_cast<const TIn*>(p.k);
  const TIn* vin = static_cast<const TIn*>(p.v);
  const int kch0 = Hk * DK + g * DK;    // conv channel of k[g][0]
  const int vch0 = 2 * Hk * DK + h * DV;  // conv channel of v[h][0]
  for (int base = 0; base <= d; base += kChunk) {
    // features of path nodes base .. base+kChunk-1: one wave per node
    for (int mrel = wave; mrel < kChunk; mrel += kCT / kWave) {
      const int mi = base + mrel;
      if (mi > d) break;
      float yk[KPL], yv[VPL];
      float ss = 0.0f;
#pragma unroll
      for (int e = 0; e < KPL; ++e) {
        const int c = lane * KPL + e;
        float y = 0.0f;
        if (c < DK) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int mm = mi - 3 + w;
            const float x = mm >= 0
                                ? ld(kin, (size_t(b) * T + s_path[mm]) * Hk * DK + size_t(g) * DK + c)
                                : p.conv_state[(size_t(b) * 3 + (3 + mm)) * C + kch0 + c];
            y += p.conv_w[size_t(kch0 + c) * 4 + w] * x;
          }
          y = silu(y);
        }
        yk[e] = y;
        ss += y * y;
      }
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) ss += __shfl_xor(ss, o);
      const float inv = rsqrt_hw(ss + 1e-6f);
#pragma unroll
      for (int e = 0; e < KPL; ++e) {
        const int c = lane * KPL + e;
        if (c < DK) s_k[mrel][c] = yk[e] * inv;
      }
#pragma unroll
      for (int e = 0; e < VPL; ++e) {
        const int c = lane * VPL + e;
        if (c < DV) {
          float y = 0.0f;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int mm = mi - 3 + w;
            const float x = mm >= 0
                                ? ld(vin, (size_t(b) * T + s_path[mm]) * Hv * DV + size_t(h) * DV + c)
                                : p.conv_state[(size_t(b) * 3 + (3 + mm)) * C + vch0 + c];
            y += p.conv_w[size_t(vch0 + c) * 4 + w] * x;
          }
          yv[e] = silu(y);
          s_v[mrel][c] = yv[e];
        }
      }
    }
    __syncthreads();
    const int cnt = (d - base + 1) < kChunk ? (d - base + 1) : kChunk;
    for (int mrel = 0; mrel < cnt; ++mrel) {
      const int mi = base + mrel;
      const float al = s_al[mi], be = s_be[mi];
      float kk[EPT];
      if constexpr (EPT % 4 == 0) {
#pragma unroll
        for (int e = 0; e < EPT; e += 4) {
          const float4 x = *reinterpret_cast<const float4*>(&s_k[mrel][col0 + e]);
          kk[e] = x.x;
          kk[e + 1] = x.y;
          kk[e + 2] = x.z;
          kk[e + 3] = x.w;
        }
      } else {
#pragma unroll
        for (int e = 0; e < EPT; ++e) kk[e] = s_k[mrel][col0 + e];
      }
      float u = 0.0f;
#pragma unroll
      for (int e = 0; e < EPT; ++e) u += srow[e] * kk[e];
#pragma unroll
      for (int o = 1; o < LPR; o <<= 1) u += __shfl_xor(u, o);
      const float c = be * (s_v[mrel][row] - al * u);
#pragma unroll
      for (int e = 0; e < EPT; ++e) srow[e] = al * srow[e] + c * kk[e];
    }
    __syncthreads();
  }
  if constexpr (EPT % 4 == 0) {
#pragma unroll
    for (int e = 0; e < EPT; e += 4)
      *reinterpret_cast<float4*>(Sbh + size_t(row) * DK + col0 + e) =
          make_float4(srow[e], srow[e + 1], srow[e + 2], srow[e + 3]);
  } else {
#pragma unroll
    for (int e = 0; e < EPT; ++e) Sbh[size_t(row) * DK + col0 + e] = srow[e];
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
  hipLaunchKernelGGL((commit_state_kernel<DK, DV, TIn>), dim3(p.Hv, p.B), dim3(kCT), 0, stream, p);
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
