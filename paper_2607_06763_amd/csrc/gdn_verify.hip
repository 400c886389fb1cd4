// gdn_verify.hip -- read-only tree verification through one GDN layer.
//
// For every node i of a draft tree the output is the gated delta rule
// (Eq. 7) applied along i's own path root..i starting from the cached state
// S0, then read out with q_i (Eq. 8); S0 is never written (Sec. 3.4).
//
// Instead of the paper's masked triangular solve (Eq. 9-13) this kernel uses
// an exact rearrangement of Eq. 7-8 that needs one contraction with S0 per
// node.  In the stored orientation (S in R^{dv x dk}, o = scale S q), one
// step gives S_t x = alpha_t S_{t-1} (x - beta_t (k_t.x) k_t) + beta_t (k_t.x) v_t
// for any vector x, so walking i's path from the leaf to the root with
//     x <- q_i, r <- 1;   for t = i, parent(i), ..., root:
//         s = k_t.x;  c_t = r beta_t s;  x <- x - beta_t s k_t;  r <- r alpha_t
// yields  o_i = scale * ( r S0 x + sum_t c_t v_t ),  r = a_i = prod alpha.
// The leaf-to-root walk ("query pull-back") is O(depth * dk) vector work per
// node; the rest is one dense product per (sequence, value head):
//     O = scale * [ diag(a) X~ | C ] . [ S0^T ; V ]
// with X~ the pulled-back queries (T x dk) and C the ancestor-masked
// coefficients (T x T, lower triangular in the canonical order).  That
// product runs on the MFMA units with a bf16 hi/lo split of both operands
// (three bf16 products per tile, fp32 accumulation, ~1e-5 relative error).
//
// Workgroup = (dv slice, value head h, sequence b); 256 threads.
//   phase 0  metadata of the tree in canonical order -> LDS
//   phase 1  conv + SiLU + L2-norm of q, k along each node's path; k~ -> LDS,
//            q~ stays in the registers of the node's lane quad
//   phase 2  pull-back (4 lanes per node, quad reductions), coefficients -> LDS
//   phase 3  MFMA product; v~ is computed from the raw values on the fly in
//            the B-operand registers.
#include "gdn_internal.h"

namespace gdn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kVT = 256;                // threads per workgroup
constexpr int kVMaxT = 128;             // tree slots supported
constexpr int kQuads = kVT / 4;         // lane quads = nodes in flight
constexpr int kNPR = kVMaxT / kQuads;   // nodes per quad
constexpr int kKPad = 4;                // row padding (floats) of the k~/x~ tile

struct VerifyParams {
  int B, T, Hk, Hv, nslices;
  float scale;
  const void* meta;
  const void *q, *k, *v, *alpha, *beta;
  const float *conv_w, *conv_state, *S0;
  float* out;
};

// bf16 hi/lo split by truncation: x = hi + lo + O(2^-16 |x|).
__device__ __forceinline__ void split8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
  u32x4 h, l;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t u0 = __float_as_uint(x[2 * e]), u1 = __float_as_uint(x[2 * e + 1]);
    uint32_t h0 = u0 & 0xffff0000u, h1 = u1 & 0xffff0000u;
    float r0 = x[2 * e] - __uint_as_float(h0);
    float r1 = x[2 * e + 1] - __uint_as_float(h1);
    h[e] = (h0 >> 16) | h1;
    l[e] = (__float_as_uint(r0) >> 16) | (__float_as_uint(r1) & 0xffff0000u);
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

__device__ __forceinline__ f32x4 mfma3(const bf16x8& ah, const bf16x8& al, const bf16x8& bh,
                                       const bf16x8& bl, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, c, 0, 0, 0);
  return c;
}

__host__ __device__ inline int verify_ncoef(int T) { return ((T * (T + 1) / 2) + 3) & ~3; }

// LDS bytes for a tree of T slots and key dim DK.
__host__ __device__ inline size_t verify_smem_bytes(int T, int DK) {
  int TP2 = (T + 31) & ~31;
  size_t b = size_t(TP2) * (DK + kKPad) * 4;  // k~ / x~ tile
  b += size_t(4 * kVMaxT + 4) * 4;            // order, parent pos, depth, offsets
  b += size_t(2 * kVMaxT + 8 * DK) * 4;       // alpha, beta, q/k conv weights
  b += size_t(verify_ncoef(T)) * 8;           // coefficients + their positions
  return b;
}

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(kVT) void verify_kernel(VerifyParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int KROW = DK + kKPad;
  constexpr int CPL = DK / 4;   // channels per lane
  constexpr int NCH = DK / 16;  // 4-channel chunks per lane
  constexpr int KS1 = (DK + 31) / 32;
  constexpr int NPW_MAX = DV / 64 > 1 ? DV / 64 : 1;
  constexpr int MPW_MAX = kVMaxT / 16;

  const int T = p.T;
  const int slice = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int Hk = p.Hk, Hv = p.Hv;
  const int g = h * Hk / Hv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int DVS = DV / p.nslices;
  const int TP2 = (T + 31) & ~31;
  const int C = 2 * Hk * DK + Hv * DV;
  const size_t orow = size_t(Hv) * DV;

  float* s_x = reinterpret_cast<float*>(smem);
  int* s_ord = reinterpret_cast<int*>(s_x + TP2 * KROW);
  int* s_ppos = s_ord + kVMaxT;
  int* s_dep = s_ppos + kVMaxT;
  int* s_off = s_dep + kVMaxT;
  float* s_al = reinterpret_cast<float*>(s_off + kVMaxT + 4);
  float* s_be = s_al + kVMaxT;
  float* s_w = s_be + kVMaxT;  // [2][DK][4]
  float* s_coef = s_w + 8 * DK;
  int* s_cpos = reinterpret_cast<int*>(s_coef + verify_ncoef(T));

  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int status = m.status[b];
  const int nv = m.nvalid[b];
  if (status != GDN_TREE_OK) {
    for (int idx = tid; idx < T * DVS; idx += kVT) {
      int i = idx / DVS, c = idx % DVS;
      p.out[(size_t(b) * T + i) * orow + size_t(h) * DV + slice * DVS + c] = 0.0f;
    }
    return;
  }

  // ---------------- phase 0: tree metadata in canonical order --------------
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  if (tid < T) {
    const int i = tid;
    int node = m.order[b * T + i];
    node = (node >= 0 && node < T) ? node : 0;  // metadata written by prepare is a permutation
    const bool real = i < nv;
    s_ord[i] = node;
    s_dep[i] = real ? m.depth[b * T + node] : -1;
    const int par = m.parent[b * T + node];
    s_ppos[i] = (real && par >= 0 && par < T) ? m.pos[b * T + par] : -1;
    const size_t ab = (size_t(b) * T + node) * Hv + h;
    s_al[i] = ld(alpha, ab);
    s_be[i] = ld(beta, ab);
  }
  for (int i = tid; i < 8 * DK; i += kVT) {
    const int part = i / (4 * DK), rem = i % (4 * DK);
    const int ch = part * Hk * DK + g * DK + rem / 4;
    s_w[i] = p.conv_w[size_t(ch) * 4 + (rem & 3)];
  }
  __syncthreads();
  if (wave == 0) {  // exclusive scan of (depth + 1) over real positions
    const int i0 = 2 * lane, i1 = 2 * lane + 1;
    const int v0 = i0 < nv ? s_dep[i0] + 1 : 0;
    const int v1 = i1 < nv ? s_dep[i1] + 1 : 0;
    int sum = v0 + v1;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      int t = __shfl_up(sum, o);
      if (lane >= o) sum += t;
    }
    const int excl = sum - v0 - v1;
    s_off[i0] = excl;
    s_off[i1] = excl + v0;
  }
  __syncthreads();

  // ---------------- phase 1: conv / SiLU / L2-norm of q and k --------------
  const int quad = tid >> 2, q4 = tid & 3;
  const TIn* qin = static_cast<const TIn*>(p.q);
  const TIn* kin = static_cast<const TIn*>(p.k);
  const size_t qk_row = size_t(Hk) * DK;
  float qh[kNPR][CPL];
#pragma unroll
  for (int r = 0; r < kNPR; ++r) {
    const int pp = quad + r * kQuads;
#pragma unroll
    for (int c = 0; c < CPL; ++c) qh[r][c] = 0.0f;
    if (pp < nv) {
      const int d = s_dep[pp];
      int tap[4];
      tap[3] = pp;
      tap[2] = s_ppos[pp];
      tap[1] = tap[2] >= 0 ? s_ppos[tap[2]] : -1;
      tap[0] = tap[1] >= 0 ? s_ppos[tap[1]] : -1;
      float yq[CPL], yk[CPL];
#pragma unroll
      for (int c = 0; c < CPL; ++c) yq[c] = yk[c] = 0.0f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int mm = d - 3 + w;
        const TIn* qrow = nullptr;
        const TIn* krow = nullptr;
        const float* cs = nullptr;
        if (mm >= 0) {
          const size_t node = s_ord[tap[w]];
          qrow = qin + (size_t(b) * T + node) * qk_row + size_t(g) * DK;
          krow = kin + (size_t(b) * T + node) * qk_row + size_t(g) * DK;
        } else {
          cs = p.conv_state + (size_t(b) * 3 + (3 + mm)) * C;
        }
#pragma unroll
        for (int u = 0; u < NCH; ++u) {
          const int c = 16 * u + 4 * q4;
          float4 xq, xk;
          if (mm >= 0) {
            xq = ld4(qrow + c);
            xk = ld4(krow + c);
          } else {
            xq = ld4(cs + g * DK + c);
            xk = ld4(cs + Hk * DK + g * DK + c);
          }
          const float xqa[4] = {xq.x, xq.y, xq.z, xq.w};
          const float xka[4] = {xk.x, xk.y, xk.z, xk.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            yq[4 * u + e] += s_w[(c + e) * 4 + w] * xqa[e];
            yk[4 * u + e] += s_w[4 * DK + (c + e) * 4 + w] * xka[e];
          }
        }
      }
      float sq = 0.0f, sk = 0.0f;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        yq[c] = silu(yq[c]);
        yk[c] = silu(yk[c]);
        sq += yq[c] * yq[c];
        sk += yk[c] * yk[c];
      }
      sq += __shfl_xor(sq, 1);
      sq += __shfl_xor(sq, 2);
      sk += __shfl_xor(sk, 1);
      sk += __shfl_xor(sk, 2);
      const float iq = 1.0f / sqrtf(sq + 1e-6f);
      const float ik = 1.0f / sqrtf(sk + 1e-6f);
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int c = 16 * u + 4 * q4;
#pragma unroll
        for (int e = 0; e < 4; ++e) qh[r][4 * u + e] = yq[4 * u + e] * iq;
        *reinterpret_cast<float4*>(s_x + pp * KROW + c) =
            make_float4(yk[4 * u] * ik, yk[4 * u + 1] * ik, yk[4 * u + 2] * ik, yk[4 * u + 3] * ik);
      }
    }
  }
  __syncthreads();

  // ---------------- phase 2: query pull-back along each path ----------------
#pragma unroll
  for (int r = 0; r < kNPR; ++r) {
    const int pp = quad + r * kQuads;
    if (pp < nv) {
      float rr = 1.0f;
      int t = pp;
      const int off = s_off[pp];
      // a path has at most T nodes; the bound also ends the walk on corrupt metadata
      for (int step = 0; t >= 0 && step < T; ++step) {
        const float* krow = s_x + t * KROW;
        float kv[CPL];
        float s = 0.0f;
#pragma unroll
        for (int u = 0; u < NCH; ++u) {
          const float4 k4 = *reinterpret_cast<const float4*>(krow + 16 * u + 4 * q4);
          kv[4 * u] = k4.x;
          kv[4 * u + 1] = k4.y;
          kv[4 * u + 2] = k4.z;
          kv[4 * u + 3] = k4.w;
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) s += kv[c] * qh[r][c];
        s += __shfl_xor(s, 1);
        s += __shfl_xor(s, 2);
        const float bs = s_be[t] * s;
        if (q4 == 0) {
          const int slot = off + s_dep[t];
          s_coef[slot] = rr * bs;
          s_cpos[slot] = t;
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) qh[r][c] -= bs * kv[c];
        rr *= s_al[t];
        t = s_ppos[t];
      }
#pragma unroll
      for (int c = 0; c < CPL; ++c) qh[r][c] *= rr;  // a_i * x~_i
    }
  }
  __syncthreads();  // every pull-back has finished reading k~
#pragma unroll
  for (int r = 0; r < kNPR; ++r) {
    const int pp = quad + r * kQuads;
    if (pp < TP2) {
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int c = 16 * u + 4 * q4;
        *reinterpret_cast<float4*>(s_x + pp * KROW + c) =
            make_float4(qh[r][4 * u], qh[r][4 * u + 1], qh[r][4 * u + 2], qh[r][4 * u + 3]);
      }
    }
  }
  __syncthreads();

  // ---------------- phase 3: O = scale [a X~ | C] [S0^T ; V~] on MFMA -------
  const int NTS = DVS / 16;
  const int WN = NTS >= 4 ? 4 : NTS;
  const int WM = 4 / WN;
  const int wn = wave % WN, wm = wave / WN;
  const int NPW = NTS / WN;
  const int MT = TP2 / 16;
  const int l16 = lane & 15, lg = lane >> 4;

  f32x4 acc[NPW_MAX][MPW_MAX];
#pragma unroll
  for (int ni = 0; ni < NPW_MAX; ++ni)
#pragma unroll
    for (int mi = 0; mi < MPW_MAX; ++mi) acc[ni][mi] = f32x4{0.f, 0.f, 0.f, 0.f};

  // part 1: a X~ S0^T   (K = dk)
  const float* S0bh = p.S0 + (size_t(b) * Hv + h) * size_t(DV) * DK;
#pragma unroll
  for (int ks = 0; ks < KS1; ++ks) {
    const int k0 = ks * 32 + 8 * lg;
    bf16x8 bh[NPW_MAX], bl[NPW_MAX];
#pragma unroll
    for (int ni = 0; ni < NPW_MAX; ++ni) {
      if (ni < NPW) {
        const int rcol = slice * DVS + (wn + ni * WN) * 16 + l16;
        float xs[8];
        if (k0 < DK) {
          const float4 a0 = ld4(S0bh + size_t(rcol) * DK + k0);
          const float4 a1 = ld4(S0bh + size_t(rcol) * DK + k0 + 4);
          xs[0] = a0.x; xs[1] = a0.y; xs[2] = a0.z; xs[3] = a0.w;
          xs[4] = a1.x; xs[5] = a1.y; xs[6] = a1.z; xs[7] = a1.w;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) xs[e] = 0.0f;
        }
        split8(xs, bh[ni], bl[ni]);
      }
    }
#pragma unroll
    for (int mi = 0; mi < MPW_MAX; ++mi) {
      const int mt = wm + mi * WM;
      if (mt < MT) {
        const int row = mt * 16 + l16;
        float xa[8];
        if (k0 < DK) {
          const float4 a0 = *reinterpret_cast<const float4*>(s_x + row * KROW + k0);
          const float4 a1 = *reinterpret_cast<const float4*>(s_x + row * KROW + k0 + 4);
          xa[0] = a0.x; xa[1] = a0.y; xa[2] = a0.z; xa[3] = a0.w;
          xa[4] = a1.x; xa[5] = a1.y; xa[6] = a1.z; xa[7] = a1.w;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) xa[e] = 0.0f;
        }
        bf16x8 ah, al;
        split8(xa, ah, al);
#pragma unroll
        for (int ni = 0; ni < NPW_MAX; ++ni)
          if (ni < NPW) acc[ni][mi] = mfma3(ah, al, bh[ni], bl[ni], acc[ni][mi]);
      }
    }
  }

  // part 2: C V~   (K = tree positions; C lower triangular)
  const TIn* vin = static_cast<const TIn*>(p.v);
  const int vbase = 2 * Hk * DK + h * DV;  // conv channel of v[h][0]
  for (int ks = 0; ks < TP2 / 32; ++ks) {
    const int j0 = ks * 32 + 8 * lg;
    bf16x8 bh[NPW_MAX], bl[NPW_MAX];
#pragma unroll
    for (int ni = 0; ni < NPW_MAX; ++ni) {
      if (ni < NPW) {
        const int rcol = slice * DVS + (wn + ni * WN) * 16 + l16;
        const float4 wv = ld4(p.conv_w + size_t(vbase + rcol) * 4);
        const float wva[4] = {wv.x, wv.y, wv.z, wv.w};
        float xs[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = j0 + e;
          float y = 0.0f;
          if (j < nv) {
            const int d = s_dep[j];
            int t = j;
#pragma unroll
            for (int w = 3; w >= 0; --w) {
              const int mm = d - 3 + w;
              float x;
              if (mm >= 0) {
                x = ld(vin, (size_t(b) * T + s_ord[t]) * orow + size_t(h) * DV + rcol);
                if (w > 0) t = s_ppos[t];
              } else {
                x = p.conv_state[(size_t(b) * 3 + (3 + mm)) * C + vbase + rcol];
              }
              y += wva[w] * x;
            }
            y = silu(y);
          }
          xs[e] = y;
        }
        split8(xs, bh[ni], bl[ni]);
      }
    }
#pragma unroll
    for (int mi = 0; mi < MPW_MAX; ++mi) {
      const int mt = wm + mi * WM;
      if (mt < MT && ks * 32 <= mt * 16 + 15) {
        const int i = mt * 16 + l16;
        const int di = i < nv ? s_dep[i] : -1;
        const int offi = s_off[i];
        float xa[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = j0 + e;
          float cv = 0.0f;
          if (di >= 0 && j <= i) {
            const int dj = s_dep[j];
            if (dj <= di) {
              const int slot = offi + dj;
              if (s_cpos[slot] == j) cv = s_coef[slot];
            }
          }
          xa[e] = cv;
        }
        bf16x8 ah, al;
        split8(xa, ah, al);
#pragma unroll
        for (int ni = 0; ni < NPW_MAX; ++ni)
          if (ni < NPW) acc[ni][mi] = mfma3(ah, al, bh[ni], bl[ni], acc[ni][mi]);
      }
    }
  }

  // store: tile row 4*lg+e, column l16
#pragma unroll
  for (int ni = 0; ni < NPW_MAX; ++ni) {
    if (ni >= NPW) continue;
    const int rcol = slice * DVS + (wn + ni * WN) * 16 + l16;
#pragma unroll
    for (int mi = 0; mi < MPW_MAX; ++mi) {
      const int mt = wm + mi * WM;
      if (mt >= MT) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = mt * 16 + 4 * lg + e;
        if (i < T) {
          const size_t node = s_ord[i];
          p.out[(size_t(b) * T + node) * orow + size_t(h) * DV + rcol] = acc[ni][mi][e] * p.scale;
        }
      }
    }
  }
}

template <int DK, int DV, typename TIn>
static int launch_verify_t(const VerifyArgs& a, hipStream_t stream) {
  VerifyParams p;
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
  // split the value dim across workgroups while the grid is small
  int ns = 1;
  while (size_t(a.B) * a.Hv * ns < 256 && DV / (2 * ns) >= 32) ns *= 2;
  p.nslices = ns;
  const size_t smem = verify_smem_bytes(a.T, DK);
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&verify_kernel<DK, DV, TIn>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(verify_smem_bytes(kVMaxT, DK)));
    if (e != hipSuccess)
      return set_error(GDN_EHIP, "verify: LDS attribute: %s", hipGetErrorString(e));
    attr_done = true;
  }
  hipLaunchKernelGGL((verify_kernel<DK, DV, TIn>), dim3(ns, a.Hv, a.B), dim3(kVT), smem, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "verify launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

template <int DK, typename TIn>
static int dispatch_dv(const VerifyArgs& a, hipStream_t s) {
  switch (a.dv) {
    case 16: return launch_verify_t<DK, 16, TIn>(a, s);
    case 32: return launch_verify_t<DK, 32, TIn>(a, s);
    case 64: return launch_verify_t<DK, 64, TIn>(a, s);
    case 128: return launch_verify_t<DK, 128, TIn>(a, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify: dv=%d unsupported", a.dv);
}

template <typename TIn>
static int dispatch_dk(const VerifyArgs& a, hipStream_t s) {
  switch (a.dk) {
    case 16: return dispatch_dv<16, TIn>(a, s);
    case 32: return dispatch_dv<32, TIn>(a, s);
    case 64: return dispatch_dv<64, TIn>(a, s);
    case 128: return dispatch_dv<128, TIn>(a, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify: dk=%d unsupported", a.dk);
}

int launch_verify(const VerifyArgs& a, hipStream_t stream) {
  if (a.T > kVMaxT) return set_error(GDN_EUNSUPPORTED, "verify: T=%d exceeds %d", a.T, kVMaxT);
  if (a.in_dtype == GDN_BF16) return dispatch_dk<BF16>(a, stream);
  return dispatch_dk<float>(a, stream);
}

}  // namespace gdn
