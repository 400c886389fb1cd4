// gdn_large.hip -- read-only verification of trees of 129..512 slots.
//
// The verification of one node is the query pull-back of the T <= 128
// kernel (an exact rearrangement of Eq. 7-8): walking the path of i from
// the node to the root with
//     x <- q~_i, r <- 1, acc <- 0;   for t = i, parent(i), ..., root:
//         s = k~_t.x;  acc += r beta_t s v~_t;  x <- x - beta_t s k~_t;  r <- r alpha_t
// gives o_i = scale (S0 (r x) + acc) in the stored orientation.  With up to
// 512 slots the post-conv features of a tree no longer fit in LDS, so the
// work is split in two launches:
//   feat_kernel   one workgroup per (2048 channels, 32 positions, sequence):
//                 the width-4 conv along each node's path (conv-state slots
//                 above the root), SiLU, and the per-head L2 norm of q and
//                 k; written to a workspace of fp16 features FH[B][T][C]
//                 (canonical position order, channels as in conv_w; q~
//                 and k~ have unit norm, each v~ row of a value head is
//                 scaled by the power of two that puts its largest
//                 magnitude in [1, 2), the inverse scale kept in
//                 Vs[B][T][Hv]).  The chunked form reads the same features
//                 as fp32 (launch_features).
//   pull_kernel   one workgroup per (value head, sequence), 512 threads:
//                 the head's S0 as one fp16 plane in LDS (each row scaled by
//                 the power of two that puts its largest magnitude in [1, 2),
//                 exact, undone on the output), then tiles of 32 positions:
//                 16 lanes per node walk the paths with the features of the
//                 path nodes gathered from FH (fp16 operands into fp32
//                 accumulators by mixed-precision FMAs), the value heads of
//                 one key head on one XCD so that they share its k~ rows in
//                 L2, r x -> an fp16 tile, O^T = S0 (r X)^T on
//                 v_mfma_f32_16x16x32_f16 (fp32 accumulation), plus acc.
// The fused decode step (Sec. 3.4.2) runs the conv-state shift of the
// previous step's commit first, the features on the committed conv state,
// and pull_kernel<..., FUSED>, which commits the previous accepted path into
// its head's state rows (commit_rows) and converts the committed rows
// straight into its plane.
#include <map>
#include <type_traits>
#include <mutex>

#include "gdn_commit_rows.h"

namespace gdn {

constexpr int kLT = 512;      // threads of a pull-back workgroup (8 waves)
constexpr int kLTile = 32;    // positions per readout tile (4 per wave)
constexpr int kLMaxT = 512;   // tree slots supported
constexpr int kFT = 256;      // threads of a feature workgroup

struct LargeParams {
  int B, T, Hk, Hv;
  float scale;
  const void* meta;
  const void *q, *k, *v, *alpha, *beta;
  const float *conv_w, *conv_state, *S0;
  float* out;
  float* F;       // fp32 features [B][T][C] (chunked form)
  _Float16* FH;   // fp16 features [B][T][C] (pull-back)
  float* Vs;      // inverse v~ row scales [B][T][Hv] (pull-back)
  // fused step: the previous step's commit, run by the pull-back on the rows
  // it reads (conv_state above is then the conv state after the commit)
  CommitParams cp;
};

static size_t fh_bytes(int B, int T, int Hk, int Hv, int dk, int dv) {
  return (size_t(B) * size_t(T) * size_t(2 * Hk * dk + Hv * dv) * 2 + 255) & ~size_t(255);
}

size_t large_workspace_bytes(int B, int T, int Hk, int Hv, int dk, int dv) {
  return fh_bytes(B, T, Hk, Hv, dk, dv) + size_t(B) * size_t(T) * size_t(Hv) * sizeof(float);
}

size_t features_f32_bytes(int B, int T, int Hk, int Hv, int dk, int dv) {
  return size_t(B) * size_t(T) * size_t(2 * Hk * dk + Hv * dv) * sizeof(float);
}

// ---------------------------------------------------------------------------
// Features: conv taps along the path, SiLU, L2 norm (q, k).  One workgroup
// per (kFT CPT channels, block of kFP positions, sequence): each thread keeps
// the conv weights of its CPT channels in registers, the block's conv taps
// are resolved once into LDS, and the raw rows of the next positions are in
// flight while the current ones are computed.  CPT = 8 channels per thread
// for the fp16 workspace (one 16-byte row load and store per tap and
// position), 4 for the fp32 features, whose 16-byte stores then stay
// contiguous across the lanes.
// ---------------------------------------------------------------------------
constexpr int kFP = 32;  // positions per feature workgroup

// First thread (in units of CPT channels) of the value channels: the q / k
// threads come first, the value threads start on a wave boundary, so that
// every wave reads rows of one row stride (the q and k rows have Hk dk
// elements, the v rows Hv dv) and the dv / CPT lanes of a value head are
// aligned consecutive lanes of one wave.
__host__ __device__ inline int feat_vbase(int Hk, int dk, int cpt) {
  const int nqk = 2 * Hk * dk / cpt;
  return (nqk + 63) & ~63;
}

// N raw channels of one row (N = 4 or 8), kept as loaded until they are used
template <typename TIn, int N>
struct RawRow;
template <int N>
struct RawRow<BF16, N> {
  uint32_t u[N / 2];
  __device__ __forceinline__ void load(const BF16* p) {
    if constexpr (N == 8) {
      const uint4 v = *reinterpret_cast<const uint4*>(p);
      u[0] = v.x, u[1] = v.y, u[2] = v.z, u[3] = v.w;
    } else {
      const uint2 v = *reinterpret_cast<const uint2*>(p);
      u[0] = v.x, u[1] = v.y;
    }
  }
  __device__ __forceinline__ void get(float (&x)[N]) const {
#pragma unroll
    for (int j = 0; j < N / 2; ++j) {
      x[2 * j] = __uint_as_float(u[j] << 16);
      x[2 * j + 1] = __uint_as_float(u[j] & 0xffff0000u);
    }
  }
};
template <int N>
struct RawRow<float, N> {
  float4 a[N / 4];
  __device__ __forceinline__ void load(const float* p) {
#pragma unroll
    for (int h = 0; h < N / 4; ++h) a[h] = reinterpret_cast<const float4*>(p)[h];
  }
  __device__ __forceinline__ void get(float (&x)[N]) const {
#pragma unroll
    for (int h = 0; h < N / 4; ++h) x[4 * h] = a[h].x, x[4 * h + 1] = a[h].y, x[4 * h + 2] = a[h].z, x[4 * h + 3] = a[h].w;
  }
};

// Largest |x| over aligned groups of N lanes, on the bit patterns of the
// magnitudes (the same order as the floats; a NaN counts as 0, as fmaxf
// would skip it), one DPP max per step.
template <int N>
__device__ __forceinline__ float group_absmax(float v) {
  uint32_t u = __float_as_uint(v) & 0x7fffffffu;
  u = u > 0x7f800000u ? 0u : u;
  auto mx = [&](uint32_t a, uint32_t o) { return a > o ? a : o; };
  if constexpr (N >= 2) u = mx(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), kDppQuadXor1, 0xF, 0xF, false)));
  if constexpr (N >= 4) u = mx(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), kDppQuadXor2, 0xF, 0xF, false)));
  if constexpr (N >= 8) u = mx(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), kDppRowHalfMirror, 0xF, 0xF, false)));
  if constexpr (N >= 16) u = mx(u, uint32_t(__builtin_amdgcn_update_dpp(0, int(u), kDppRowMirror, 0xF, 0xF, false)));
  if constexpr (N >= 32) u = mx(u, uint32_t(__shfl_xor(int(u), 16)));
  static_assert(N <= 32, "group size");
  return __uint_as_float(u);
}

// VG = 0: fp32 features into p.F; VG = DV / CPT: fp16 features into p.FH
// with the v~ rows of each head scaled (inverse scales into p.Vs).
template <typename TIn, int DK, int VG, int CPT>
__global__ __launch_bounds__(kFT) void feat_kernel(LargeParams p, int DV, int ncb) {
  constexpr bool kHalf = VG > 0;
  static_assert(CPT == 4 || CPT == 8, "channels per thread");
  // positions per register buffer: 32 registers of raw rows (4 taps each)
  constexpr int kFU = 32 / (int(sizeof(TIn)) * CPT);
  __shared__ int s_tap[kFP][4];  // node of each tap, or -1 - conv-state slot
  // Blocks go round-robin over the 8 XCDs.  The grid is one-dimensional and
  // renumbered so that each XCD takes a contiguous range of (position block,
  // channel block, sequence) in that order: the position blocks of one
  // channel block of a sequence run on one XCD, where the rows that some of
  // them load are still in L2 when others gather them as ancestor taps
  // (measured: 1.5x fewer HBM bytes fetched).
  const int nblk = gridDim.x, per = nblk / 8;
  const int id = blockIdx.x;
  const int L = id < 8 * per ? (id % 8) * per + id / 8 : id;
  const int nyb = (p.T + kFP - 1) / kFP;
  const int yb = L % nyb, bx = (L / nyb) % ncb, b = L / (nyb * ncb);
  const int tid = threadIdx.x;
  const int p0 = yb * kFP;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int nval = m.status[b] == GDN_TREE_OK ? m.nvalid[b] : 0;
  if (p0 >= nval) return;  // uniform
  const int np = nval - p0 < kFP ? nval - p0 : kFP;
  const size_t bt = size_t(b) * T;
  if (tid < np) {
    // the 4 taps of position p0 + tid (3 = the node itself): a path node's
    // raw row, or the conv-state slot d + w for taps above the root
    const int pos = p0 + tid;
    const int d = m.pdep[bt + pos];
    const int t2 = m.ppos[bt + pos];
    const int t1 = t2 >= 0 ? m.ppos[bt + t2] : -1;
    const int t0 = t1 >= 0 ? m.ppos[bt + t1] : -1;
    const int tp[4] = {t0, t1, t2, pos};
#pragma unroll
    for (int w = 0; w < 4; ++w) s_tap[tid][w] = d - 3 + w >= 0 ? m.order[bt + tp[w]] : -1 - (d + w);
  }
  const int nq = Hk * DK;
  const int C = 2 * nq + Hv * DV;
  const int vb = feat_vbase(Hk, DK, CPT);
  const int nqkt = 2 * nq / CPT, nvt = Hv * DV / CPT;
  const int ct = bx * kFT + tid;
  const bool isv = ct >= vb;  // the same for the whole wave
  const bool ok = isv ? ct - vb < nvt : ct < nqkt;
  // this thread's first channel; lanes past the channels of their kind
  // compute on the last group of that kind (in bounds) and store nothing
  const int c = isv ? 2 * nq + CPT * (ct - vb < nvt ? ct - vb : nvt - 1) : CPT * (ct < nqkt ? ct : nqkt - 1);
  const TIn* src;
  int off;
  if (c < nq) {
    src = static_cast<const TIn*>(p.q), off = c;
  } else if (c < 2 * nq) {
    src = static_cast<const TIn*>(p.k), off = c - nq;
  } else {
    src = static_cast<const TIn*>(p.v), off = c - 2 * nq;
  }
  // row stride of this wave's tensor (wave-uniform: node offsets are scalar)
  const int rs = __builtin_amdgcn_readfirstlane(isv ? Hv * DV : nq);
  src += bt * size_t(rs) + off;
  float4 wv[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) wv[j] = reinterpret_cast<const float4*>(p.conv_w + size_t(c) * 4)[j];
  const bool qk = !isv;
  // the conv-state slots of this thread's channels (taps above the root),
  // kept in LDS: read under a branch, an LDS load does not make the row
  // loads in flight wait
  __shared__ float4 s_cs[3][CPT / 4][kFT];
  {
    const float* cs = p.conv_state + size_t(b) * 3 * C + c;
#pragma unroll
    for (int sl = 0; sl < 3; ++sl)
#pragma unroll
      for (int h = 0; h < CPT / 4; ++h) s_cs[sl][h][tid] = ld4(cs + size_t(sl) * C + 4 * h);
  }
  float* dst = kHalf ? nullptr : p.F + (bt + p0) * size_t(C) + c;
  _Float16* dsth = kHalf ? p.FH + (bt + p0) * size_t(C) + c : nullptr;
  // the first lane of each value head writes the head's inverse scale
  const bool vs_lane = kHalf && ok && isv && (ct - vb) % (kHalf ? VG : 1) == 0;
  float* vs = vs_lane ? p.Vs + (bt + p0) * size_t(Hv) + (ct - vb) / (kHalf ? VG : 1) : nullptr;
  __syncthreads();
  // Two register buffers of kFU positions each: the rows of the next group
  // are in flight while the current one is computed.  Group indices past
  // the block are clamped to its last position (loaded again, not stored).
  RawRow<TIn, CPT> ra[kFU][4], rb[kFU][4];
  int ca[kFU], cb[kFU];  // tap 0's code: negative iff the position is within 3 of the root
  auto load_group = [&](RawRow<TIn, CPT> (&xr)[kFU][4], int (&code)[kFU], int g0) {
#pragma unroll
    for (int u = 0; u < kFU; ++u) {
      const int i = g0 + u < np ? g0 + u : np - 1;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int nd = __builtin_amdgcn_readfirstlane(s_tap[i][w]);
        if (w == 0) code[u] = nd;
        xr[u][w].load(src + (nd >= 0 ? nd : 0) * rs);
      }
    }
  };
  auto compute_group = [&](const RawRow<TIn, CPT> (&xr)[kFU][4], const int (&code)[kFU], int g0) {
#pragma unroll
    for (int u = 0; u < kFU; ++u) {
      float x[4][CPT];
#pragma unroll
      for (int w = 0; w < 4; ++w) xr[u][w].get(x[w]);
      if (code[u] < 0) {
        // taps above the root read the conv-state slots (uniform; only near
        // the start of a tree, as the canonical order sorts by depth)
        const int i = g0 + u < np ? g0 + u : np - 1;
#pragma unroll
        for (int w = 0; w < 3; ++w) {
          const int cd = __builtin_amdgcn_readfirstlane(s_tap[i][w]);
          if (cd < 0) {
#pragma unroll
            for (int h = 0; h < CPT / 4; ++h) {
              const float4 a = s_cs[-1 - cd][h][tid];
              x[w][4 * h] = a.x, x[w][4 * h + 1] = a.y, x[w][4 * h + 2] = a.z, x[w][4 * h + 3] = a.w;
            }
          }
        }
      }
      float y[CPT];
      float ss = 0.0f;
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        y[j] = silu(fmaf(wv[j].w, x[3][j], fmaf(wv[j].z, x[2][j], fmaf(wv[j].y, x[1][j], wv[j].x * x[0][j]))));
        ss = fmaf(y[j], y[j], ss);
      }
      // the DK / CPT lanes of a q or k head are consecutive lanes of one wave
      ss = group_sum<DK / CPT>(ss);
      const float f = qk ? rsqrt_hw(ss + 1e-6f) : 1.0f;
      const bool st = ok && g0 + u < np;
      if constexpr (kHalf) {
        // v~: one power-of-two scale per (position, head) from the row max
        float mx = 0.0f;
#pragma unroll
        for (int j = 0; j < CPT; ++j) mx = fmaxf(mx, fabsf(y[j]));
        mx = group_absmax<VG>(mx);
        float sc, inv;
        row_scale(mx, sc, inv);
        const float g = qk ? f : sc;
        uint2 h4[CPT / 4];
#pragma unroll
        for (int h = 0; h < CPT / 4; ++h) h4[h] = to_f16x4(make_float4(y[4 * h], y[4 * h + 1], y[4 * h + 2], y[4 * h + 3]), g);
        if (st) {
          if constexpr (CPT == 8)
            *reinterpret_cast<uint4*>(dsth + size_t(g0 + u) * C) = make_uint4(h4[0].x, h4[0].y, h4[1].x, h4[1].y);
          else
            *reinterpret_cast<uint2*>(dsth + size_t(g0 + u) * C) = h4[0];
          if (vs_lane) vs[size_t(g0 + u) * Hv] = inv;
        }
      } else {
        if (st) {
          float4* d4 = reinterpret_cast<float4*>(dst + size_t(g0 + u) * C);
#pragma unroll
          for (int h = 0; h < CPT / 4; ++h)
            d4[h] = make_float4(y[4 * h] * f, y[4 * h + 1] * f, y[4 * h + 2] * f, y[4 * h + 3] * f);
        }
      }
    }
  };
  load_group(ra, ca, 0);
  for (int i0 = 0;;) {
    load_group(rb, cb, i0 + kFU);
    compute_group(ra, ca, i0);
    i0 += kFU;
    if (i0 >= np) break;
    load_group(ra, ca, i0 + kFU);
    compute_group(rb, cb, i0);
    i0 += kFU;
    if (i0 >= np) break;
  }
}

// ---------------------------------------------------------------------------
// Pull-back along gathered features + fp16 MFMA readout
// ---------------------------------------------------------------------------
template <int DK, int DV>
struct PullSmem {
  static constexpr int KP = (DK < 32 ? 32 : DK) + 8;  // fp16 row (zero beyond DK)
  static constexpr int PP = DV + 4;                    // fp32 row of the product tile
  static constexpr size_t plane = size_t(DV) * KP * 2;
  static constexpr size_t xt = size_t(2) * kLTile * KP * 2;  // r x as fp16 hi and lo planes
  static constexpr size_t pt = size_t(kLTile) * PP * 4;
  // the plane and the two tiles; in the fused step the commit's LDS first
  static constexpr size_t front = plane + xt + pt > commit_lds_bytes<DK, DV>() ? plane + xt + pt
                                                                              : commit_lds_bytes<DK, DV>();
  static constexpr size_t inv = size_t(DV) * 4;
  static constexpr size_t meta = size_t(kLMaxT) * (2 + 4 + 4 + 4 + 4);
  static constexpr size_t total = front + inv + meta;
};

template <int N>
__device__ __forceinline__ void ld_f(const float* src, float (&x)[N]) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int e = 0; e < N; e += 4) {
      const float4 u = *reinterpret_cast<const float4*>(src + e);
      x[e] = u.x;
      x[e + 1] = u.y;
      x[e + 2] = u.z;
      x[e + 3] = u.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < N; ++e) x[e] = src[e];
  }
}

// N consecutive fp16 values (N = 1, 2, 4, 8, aligned to 2 N bytes) as one
// load, kept packed in registers.
template <int N>
struct HalfVec {
  typedef _Float16 type __attribute__((ext_vector_type(N)));
};
template <int N>
__device__ __forceinline__ typename HalfVec<N>::type ld_h(const _Float16* src) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8, "fp16 vector width");
  return *reinterpret_cast<const typename HalfVec<N>::type*>(src);
}

// the same at a 32-bit byte offset from a wave-uniform base (a scalar base
// plus a vector offset: no 64-bit address arithmetic per load)
template <int N>
__device__ __forceinline__ typename HalfVec<N>::type ld_hb(const _Float16* base, uint32_t byte_off) {
  return *reinterpret_cast<const typename HalfVec<N>::type*>(reinterpret_cast<const char*>(base) + byte_off);
}

template <int DK, int DV, typename TIn, bool FUSED>
__global__ __launch_bounds__(kLT) void pull_kernel(LargeParams p) {
  using SM = PullSmem<DK, DV>;
  constexpr int KP = SM::KP, PP = SM::PP;
  constexpr int CK = DK / 16, CV = DV / 16;  // channels per lane (16 lanes per node)
  constexpr int KS = (DK < 32 ? 32 : DK) / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16* s_plane = reinterpret_cast<_Float16*>(smem);
  _Float16* s_x = reinterpret_cast<_Float16*>(smem + SM::plane);  // [2][kLTile][KP]: hi, lo
  float* s_p = reinterpret_cast<float*>(smem + SM::plane + SM::xt);
  float* s_inv = reinterpret_cast<float*>(smem + SM::front);
  int* s_ppos = reinterpret_cast<int*>(smem + SM::front + SM::inv);
  float* s_al = reinterpret_cast<float*>(s_ppos + kLMaxT);
  float* s_be = s_al + kLMaxT;
  float* s_vs = s_be + kLMaxT;  // inverse v~ row scales by position
  int16_t* s_ord = reinterpret_cast<int16_t*>(s_vs + kLMaxT);

  // Blocks go round-robin over the 8 XCDs: the G value heads of unit u =
  // (sequence, key head), which gather the same k~ rows, take blocks
  // u % 8 + 8 j of their group of 8 G, i.e. one XCD and one L2.
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int G = Hv / Hk;
  const int grp = blockIdx.x / (8 * G), rem = blockIdx.x % (8 * G);
  const int unit = 8 * grp + rem % 8;
  if (unit >= p.B * Hk) return;  // uniform
  const int b = unit / Hk, g = unit % Hk, h = g * G + rem / 8;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int nq = Hk * DK;
  const size_t C = size_t(2 * nq + Hv * DV);
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const size_t bt = size_t(b) * T;
  const int nval = m.status[b] == GDN_TREE_OK ? m.nvalid[b] : 0;
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);

  // ---- tree metadata and this head's gates by position
  for (int j = tid; j < T; j += kLT) {
    const int nd = m.order[bt + j];
    s_ord[j] = int16_t(nd);
    // a parent sits at a smaller position (depth order); anything else
    // (corrupt metadata) ends the walk, so every walk terminates
    const int pp = j < nval ? m.ppos[bt + j] : -1;
    s_ppos[j] = pp >= 0 && pp < j ? pp : -1;
    s_al[j] = j < nval ? ld(alpha, (bt + nd) * Hv + h) : 0.0f;
    s_be[j] = j < nval ? ld(beta, (bt + nd) * Hv + h) : 0.0f;
    s_vs[j] = j < nval ? p.Vs[(bt + j) * Hv + h] : 0.0f;
  }
  if constexpr (FUSED) {
    // ---- fused step: the previous step's accepted path is committed into
    //      this head's rows (its LDS in the plane and tile region), the rows
    //      go back to S and straight into the fp16 plane
    using CS = CommitSplit<DK, DV, kLT>;
    float srow[CS::EPT];
    const bool changed = commit_rows<DK, DV, TIn, kLT, true>(p.cp, b, h, tid, commit_lds<DK, DV>(smem), srow);
    if (changed) store_rows<DK, DV, kLT>(p.cp.S, b, h, Hv, tid, srow);
    const int row = tid / CS::LPR, col0 = (tid % CS::LPR) * CS::CPT;
#pragma unroll
    for (int i = 0; i < CS::R; ++i) {
      float mx = 0.0f;
#pragma unroll
      for (int e = 0; e < CS::CPT; ++e) mx = fmaxf(mx, fabsf(srow[i * CS::CPT + e]));
      mx = group_max<CS::LPR>(mx);
      float sc, inv;
      row_scale(mx, sc, inv);
      const int r = row + i * CS::RS;
#pragma unroll
      for (int e = 0; e < CS::CPT; ++e) s_plane[r * KP + col0 + e] = (_Float16)(srow[i * CS::CPT + e] * sc);
      if (tid % CS::LPR == 0) s_inv[r] = inv;
    }
    if constexpr (DK < 32) {
      for (int i = tid; i < DV * (32 - DK); i += kLT)
        s_plane[(i / (32 - DK)) * KP + DK + i % (32 - DK)] = (_Float16)0.0f;
      for (int i = tid; i < 2 * kLTile * (32 - DK); i += kLT)
        s_x[(i / (32 - DK)) * KP + DK + i % (32 - DK)] = (_Float16)0.0f;
    }
  } else if (nval > 0) {
    // ---- S0 -> fp16 plane (16 lanes per row), zero columns past DK
    const float* S0 = p.S0 + (size_t(b) * Hv + h) * size_t(DV) * DK;
    const int ln = tid & 15;
    for (int r0 = 0; r0 < DV; r0 += kLT / 16) {
      const int r = r0 + (tid >> 4);
      if (r < DV) {  // uniform per 16-lane group
        float xs[CK];
        ld_f<CK>(S0 + size_t(r) * DK + ln * CK, xs);
        float mx = 0.0f;
#pragma unroll
        for (int e = 0; e < CK; ++e) mx = fmaxf(mx, fabsf(xs[e]));
        mx = group_max<16>(mx);
        float sc, inv;
        row_scale(mx, sc, inv);
#pragma unroll
        for (int e = 0; e < CK; ++e) s_plane[r * KP + ln * CK + e] = (_Float16)(xs[e] * sc);
        if (ln == 0) s_inv[r] = inv;
      }
    }
    if constexpr (DK < 32) {
      for (int i = tid; i < DV * (32 - DK); i += kLT)
        s_plane[(i / (32 - DK)) * KP + DK + i % (32 - DK)] = (_Float16)0.0f;
      for (int i = tid; i < 2 * kLTile * (32 - DK); i += kLT)
        s_x[(i / (32 - DK)) * KP + DK + i % (32 - DK)] = (_Float16)0.0f;
    }
  }
  __syncthreads();

  const float scale = p.scale;
  const int jn = wave * 4 + (lane >> 4);  // node slot of this lane in a tile
  const int ln = lane & 15;
  const _Float16* Fb = p.FH + bt * C;
  using HK = typename HalfVec<CK>::type;
  using HVv = typename HalfVec<CV>::type;
  for (int n0 = 0; n0 < T; n0 += kLTile) {
    const int pos = n0 + jn;
    const bool real = pos < nval;
    float x[CK], acc[CV];
    float r = 1.0f;
#pragma unroll
    for (int e = 0; e < CV; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int e = 0; e < CK; ++e) x[e] = 0.0f;
    if (real) {
      {
        const HK q0 = ld_h<CK>(Fb + size_t(pos) * C + g * DK + ln * CK);
#pragma unroll
        for (int e = 0; e < CK; ++e) x[e] = (float)q0[e];
      }
      // walk to the root.  The gathers of the path rows are what bounds this
      // loop (L2 / MALL bandwidth, 16 resident waves per CU hide their
      // latency): loading rows ahead, which past the root means loading
      // rows that are never used, measured slower.
      // uniform row bases and a 32-bit lane offset (rows of one sequence
      // span B T C / B < 2^31 halves)
      const _Float16* Fk = Fb + nq + g * DK;
      const _Float16* Fv = Fb + 2 * nq + h * DV;
      const uint32_t Cu = uint32_t(C);
      for (int t = pos; t >= 0; t = s_ppos[t]) {  // uniform per 16-lane node group
        const uint32_t ro = uint32_t(t) * Cu;  // byte offsets below in 32 bits
        const HK kt = ld_hb<CK>(Fk, 2 * (ro + uint32_t(ln * CK)));
        const HVv vt = ld_hb<CV>(Fv, 2 * (ro + uint32_t(ln * CV)));
        float s0 = 0.0f, s1 = 0.0f;  // two chains
#pragma unroll
        for (int e = 0; e < CK; e += 2) {
          s0 = fmaf((float)kt[e], x[e], s0);
          if (e + 1 < CK) s1 = fmaf((float)kt[e + 1], x[e + 1], s1);
        }
        const float s = group_sum<16>(s0 + s1);
        const float c = s_be[t] * s;
        const float rc = r * c * s_vs[t];
#pragma unroll
        for (int e = 0; e < CV; ++e) acc[e] = fmaf(rc, (float)vt[e], acc[e]);
#pragma unroll
        for (int e = 0; e < CK; ++e) x[e] = fmaf(-c, (float)kt[e], x[e]);
        r *= s_al[t];
      }
    }
    // r x -> tile row jn (zero for padding positions) as fp16 hi + lo: the
    // product takes both, so x contributes no rounding beyond ~2^-22 (with
    // fp16 features the key dims are short, and an x rounded once to 11 bits
    // cost up to 3e-4 of max|o| on 16-dim heads)
#pragma unroll
    for (int e = 0; e < CK; ++e) {
      const float rx = r * x[e];
      const _Float16 hi = (_Float16)rx;
      s_x[jn * KP + ln * CK + e] = hi;
      s_x[(kLTile + jn) * KP + ln * CK + e] = (_Float16)(rx - (float)hi);
    }
    __syncthreads();
    // O^T tiles (16 value rows x 16 positions), K = key channels
    {
      const int l16 = lane & 15, lg = lane >> 4;
      for (int task = wave; task < (DV / 16) * (kLTile / 16); task += kLT / 64) {
        const int rt = task / (kLTile / 16), ct = task % (kLTile / 16);
        f32x4 acc4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const f16x8 a = *reinterpret_cast<const f16x8*>(s_plane + (16 * rt + l16) * KP + 32 * ks + 8 * lg);
          const f16x8 bx = *reinterpret_cast<const f16x8*>(s_x + (16 * ct + l16) * KP + 32 * ks + 8 * lg);
          const f16x8 bl = *reinterpret_cast<const f16x8*>(s_x + (kLTile + 16 * ct + l16) * KP + 32 * ks + 8 * lg);
          acc4 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bx, acc4, 0, 0, 0);
          acc4 = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bl, acc4, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 16 * rt + 4 * lg + i;
          s_p[(16 * ct + l16) * PP + row] = acc4[i] * s_inv[row];
        }
      }
    }
    __syncthreads();
    if (pos < T) {
      float o[CV];
#pragma unroll
      for (int e = 0; e < CV; ++e) o[e] = real ? scale * (s_p[jn * PP + ln * CV + e] + acc[e]) : 0.0f;
      float* dst = p.out + (bt + s_ord[pos]) * size_t(Hv) * DV + size_t(h) * DV + ln * CV;
      if constexpr (CV % 4 == 0) {
#pragma unroll
        for (int e = 0; e < CV; e += 4)
          *reinterpret_cast<float4*>(dst + e) = make_float4(o[e], o[e + 1], o[e + 2], o[e + 3]);
      } else {
#pragma unroll
        for (int e = 0; e < CV; ++e) dst[e] = o[e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------
// channels per thread of the feature kernel: 8 for the fp16 workspace, 4
// for the fp32 features
constexpr int kFCHalf = 8, kFCF32 = 4;

// channel blocks of the feature kernel
static int feat_cblocks(const LargeParams& p, int dk, int dv, int cpt) {
  const int nt = feat_vbase(p.Hk, dk, cpt) + p.Hv * dv / cpt;
  return (nt + kFT - 1) / kFT;
}

static dim3 feat_grid(const LargeParams& p, int dk, int dv, int cpt) {
  return dim3(feat_cblocks(p, dk, dv, cpt) * ((p.T + kFP - 1) / kFP) * p.B);
}

template <int DK, int DV, typename TIn, bool FUSED>
static int launch_pull(const LargeParams& p, hipStream_t stream) {
  using SM = PullSmem<DK, DV>;
  const int rc = ensure_dynamic_lds(reinterpret_cast<const void*>(&pull_kernel<DK, DV, TIn, FUSED>),
                                    int(SM::total), "verify (T > 128)");
  if (rc != GDN_OK) return rc;
  const int units = p.B * p.Hk, G = p.Hv / p.Hk;
  hipLaunchKernelGGL((pull_kernel<DK, DV, TIn, FUSED>), dim3((units + 7) / 8 * 8 * G), dim3(kLT), SM::total,
                     stream, p);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "verify (T > 128) launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

// fused: the conv-state part of the previous step's commit first (the
// features read the conv state after it), the state rows inside the
// pull-back
template <int DK, int DV, typename TIn>
static int launch_large_t(const LargeParams& p, bool fused, hipStream_t stream) {
  constexpr bool kCanFuse = commit_threads(DK, DV) == kLT;
  if (fused) {
    if (!kCanFuse) return set_error(GDN_EUNSUPPORTED, "step (T > 128): dk * dv = %d below 512", DK * DV);
    const int rc = launch_commit_conv(p.cp, DK, DV, std::is_same<TIn, BF16>::value ? GDN_BF16 : GDN_F32, stream);
    if (rc != GDN_OK) return rc;
  }
  hipLaunchKernelGGL((feat_kernel<TIn, DK, DV / kFCHalf, kFCHalf>), feat_grid(p, DK, DV, kFCHalf), dim3(kFT), 0, stream,
                     p, DV, feat_cblocks(p, DK, DV, kFCHalf));
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "verify (T > 128) feature launch: %s", hipGetErrorString(e));
  if constexpr (kCanFuse)
    if (fused) return launch_pull<DK, DV, TIn, true>(p, stream);
  return launch_pull<DK, DV, TIn, false>(p, stream);
}

template <int DK, typename TIn>
static int large_dv(const VerifyArgs& a, const LargeParams& p, hipStream_t s) {
  switch (a.dv) {
    case 16: return launch_large_t<DK, 16, TIn>(p, a.fused, s);
    case 32: return launch_large_t<DK, 32, TIn>(p, a.fused, s);
    case 64: return launch_large_t<DK, 64, TIn>(p, a.fused, s);
    case 128: return launch_large_t<DK, 128, TIn>(p, a.fused, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify: dv=%d unsupported", a.dv);
}

template <typename TIn>
static int large_dk(const VerifyArgs& a, const LargeParams& p, hipStream_t s) {
  switch (a.dk) {
    case 16: return large_dv<16, TIn>(a, p, s);
    case 32: return large_dv<32, TIn>(a, p, s);
    case 64: return large_dv<64, TIn>(a, p, s);
    case 128: return large_dv<128, TIn>(a, p, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify: dk=%d unsupported", a.dk);
}

// ws: the pull-back workspace (fp16 features, then the v~ scales) or, for
// launch_features, the fp32 feature array
static LargeParams large_params(const VerifyArgs& a, void* ws, bool half) {
  LargeParams p;
  p.B = a.B;
  p.T = a.T;
  p.Hk = a.Hk;
  p.Hv = a.Hv;
  p.scale = a.scale;
  p.meta = a.meta;
  p.q = a.q;
  p.k = a.k;
  p.v = a.v;
  p.alpha = a.alpha;
  p.beta = a.beta;
  p.conv_w = a.conv_w;
  p.conv_state = a.conv_state;
  p.S0 = a.S0;
  p.out = a.out;
  p.F = half ? nullptr : static_cast<float*>(ws);
  p.FH = half ? static_cast<_Float16*>(ws) : nullptr;
  p.Vs = half ? reinterpret_cast<float*>(static_cast<unsigned char*>(ws) + fh_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv))
              : nullptr;
  p.cp = CommitParams{};
  if (a.fused) {
    p.conv_state = a.conv_state_out;  // the features see the committed conv state
    p.cp.B = a.B;
    p.cp.T = a.T;
    p.cp.Hk = a.Hk;
    p.cp.Hv = a.Hv;
    p.cp.meta = a.pmeta;
    p.cp.accepted = a.paccepted;
    p.cp.q = a.pq;
    p.cp.k = a.pk;
    p.cp.v = a.pv;
    p.cp.alpha = a.palpha;
    p.cp.beta = a.pbeta;
    p.cp.conv_w = a.conv_w;
    p.cp.cs_in = a.conv_state;
    p.cp.cs_out = a.conv_state_out;
    p.cp.S = a.S;
    p.cp.commit_status = a.commit_status;
  }
  return p;
}

int launch_verify_large(const VerifyArgs& a, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (a.T > kLMaxT) return set_error(GDN_EUNSUPPORTED, "verify: T=%d exceeds %d", a.T, kLMaxT);
  if (ws_bytes < large_workspace_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv))
    return set_error(GDN_EINVAL, "verify: workspace of %zu bytes is too small", ws_bytes);
  const LargeParams p = large_params(a, ws, true);
  if (a.in_dtype == GDN_BF16) return large_dk<BF16>(a, p, stream);
  return large_dk<float>(a, p, stream);
}

template <typename TIn>
static int launch_features_t(const VerifyArgs& a, const LargeParams& p, hipStream_t stream) {
  switch (a.dk) {
    case 16: hipLaunchKernelGGL((feat_kernel<TIn, 16, 0, kFCF32>), feat_grid(p, 16, a.dv, kFCF32), dim3(kFT), 0, stream,
                                  p, a.dv, feat_cblocks(p, 16, a.dv, kFCF32)); break;
    case 32: hipLaunchKernelGGL((feat_kernel<TIn, 32, 0, kFCF32>), feat_grid(p, 32, a.dv, kFCF32), dim3(kFT), 0, stream,
                                  p, a.dv, feat_cblocks(p, 32, a.dv, kFCF32)); break;
    case 64: hipLaunchKernelGGL((feat_kernel<TIn, 64, 0, kFCF32>), feat_grid(p, 64, a.dv, kFCF32), dim3(kFT), 0, stream,
                                  p, a.dv, feat_cblocks(p, 64, a.dv, kFCF32)); break;
    case 128: hipLaunchKernelGGL((feat_kernel<TIn, 128, 0, kFCF32>), feat_grid(p, 128, a.dv, kFCF32), dim3(kFT), 0, stream,
                                  p, a.dv, feat_cblocks(p, 128, a.dv, kFCF32)); break;
    default: return set_error(GDN_EUNSUPPORTED, "features: dk=%d unsupported", a.dk);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "feature launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

int launch_features(const VerifyArgs& a, float* F, hipStream_t stream) {
  if (a.T > kLMaxT) return set_error(GDN_EUNSUPPORTED, "features: T=%d exceeds %d", a.T, kLMaxT);
  const LargeParams p = large_params(a, F, false);
  if (a.in_dtype == GDN_BF16) return launch_features_t<BF16>(a, p, stream);
  return launch_features_t<float>(a, p, stream);
}

// ---------------------------------------------------------------------------
// Allocation-free variant: the workspace is a file-scope device array of
// GDN_NOALLOC_SCRATCH_BYTES (every device the library runs on holds one
// copy until the process ends).  In host code `scratch` only names the
// symbol; its device address is looked up once per device with
// hipGetSymbolAddress and only that address is passed to kernels.  Calls
// that overlap on one device share the array and race.  The features are
// written before they are read, so nothing needs clearing.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[GDN_NOALLOC_SCRATCH_BYTES];

static void* scratch_address(int* rc) {
  static std::mutex mu;
  static std::map<int, void*> addr;  // device -> address of its copy
  *rc = GDN_OK;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    *rc = set_error(GDN_EHIP, "verify_noalloc: hipGetDevice failed");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(dev);
  if (it != addr.end()) return it->second;
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || ptr == nullptr) {
    *rc = set_error(GDN_EHIP, "verify_noalloc: hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    return nullptr;
  }
  addr[dev] = ptr;
  return ptr;
}

int launch_verify_noalloc(const VerifyArgs& a, hipStream_t stream) {
  if (a.T <= kSmallMaxT) return launch_verify(a, stream);  // uses no workspace
  const size_t bytes = large_workspace_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv);
  if (bytes > size_t(GDN_NOALLOC_SCRATCH_BYTES))
    return set_error(GDN_EUNSUPPORTED,
                     "verify_noalloc: B=%d T=%d needs %zu workspace bytes, above the static %zu (call "
                     "gdn_tree_verify, or split the batch)",
                     a.B, a.T, bytes, size_t(GDN_NOALLOC_SCRATCH_BYTES));
  int rc = GDN_OK;
  void* ws = scratch_address(&rc);
  if (!ws) return rc;
  return launch_verify_large(a, ws, size_t(GDN_NOALLOC_SCRATCH_BYTES), stream);
}

// ---------------------------------------------------------------------------
// Workspace of the T > 128 path: one device buffer per (device, stream),
// grown on demand and kept until the process ends.
// ---------------------------------------------------------------------------
void* stream_workspace(size_t bytes, hipStream_t stream, int* rc) {
  static std::mutex mu;
  static std::map<std::pair<int, hipStream_t>, std::pair<void*, size_t>> bufs;
  *rc = GDN_OK;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    *rc = set_error(GDN_EHIP, "workspace: hipGetDevice failed");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  auto& e = bufs[{dev, stream}];
  if (e.second >= bytes) return e.first;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
    *rc = set_error(GDN_EUNSUPPORTED,
                    "workspace: %zu bytes needed while the stream is captured; run the same sizes once "
                    "uncaptured first",
                    bytes);
    return nullptr;
  }
  if (e.first) {  // only this stream used it
    if (hipStreamSynchronize(stream) != hipSuccess || hipFree(e.first) != hipSuccess) {
      *rc = set_error(GDN_EHIP, "workspace: release of %zu bytes failed", e.second);
      return nullptr;
    }
    e.first = nullptr;
    e.second = 0;
  }
  if (hipMalloc(&e.first, bytes) != hipSuccess) {
    e.first = nullptr;
    *rc = set_error(GDN_EHIP, "workspace: hipMalloc of %zu bytes failed", bytes);
    return nullptr;
  }
  e.second = bytes;
  return e.first;
}

}  // namespace gdn
