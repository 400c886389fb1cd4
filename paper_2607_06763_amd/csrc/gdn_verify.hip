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
//     x <- q_i, r <- 1, acc <- 0;   for t = i, parent(i), ..., root:
//         s = k_t.x;  acc += r beta_t s v_t;  x <- x - beta_t s k_t;  r <- r alpha_t
// yields  o_i = scale * ( r S0 x + acc ),  r = a_i = prod of alpha on the path.
// The leaf-to-root walk ("query pull-back") is O(depth (2 dk + dv)) vector
// work per node on the VALU; the one dense product left is
//     O^T = S0 X~^T + ACC^T      (dv x T, K = dk)
// per (sequence, value head), which runs on the MFMA units with a bf16 hi/lo
// split of both operands (three bf16 products per tile, fp32 accumulation,
// ~1e-5 relative error).
//
// Workgroup = (dv slice, key head g with HPW of its value heads, sequence b),
// 512 threads.  Wave w owns the 16 tree positions [16w, 16w+16) of the
// canonical (depth, index) order; lane (l16, lg) of a wave holds, for node
// 16w + l16, the key channels 32kb + 8lg + e and the value channels
// 16n + 4lg + e.  That is exactly the MFMA B-operand layout of X~^T and the
// accumulator layout of O^T for v_mfma_f32_16x16x32_bf16, so the pulled-back
// queries and the value accumulators never leave registers.
//   phase 0  tree metadata in canonical order -> LDS; prefetch S0 and raw v
//            of the first head into registers
//   phase 1  conv + SiLU + L2-norm of q and k along each node's path (raw
//            rows staged in LDS); q~ stays in registers, k~ -> LDS (fp32)
//   per value head:
//     2a/b   raw v -> LDS, conv + SiLU -> v~ in LDS (fp32); prefetch the next
//            head's raw v
//     2c     pull-back with k~, v~ gathered from LDS (4 lanes per node)
//     2d     S0 (prefetched) -> LDS as bf16 hi/lo planes; prefetch next S0
//     2e     MFMA O^T = S0 X~^T + ACC^T, store
#include "gdn_internal.h"

namespace gdn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kVT = 512;        // threads per workgroup (8 waves)
constexpr int kVMaxT = 128;     // tree slots supported = 8 waves x 16 nodes
constexpr int kKPad = 4;        // fp32 row padding of the k~ and v~ tiles
constexpr int kSPad = 8;        // bf16 row padding of the S0 planes

struct VerifyParams {
  int B, T, Hk, Hv, DV, hpw;
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

// 4 floats -> packed bf16 hi (2 dwords) and lo (2 dwords), truncation split
__device__ __forceinline__ void split4(float4 x, uint2& hi, uint2& lo) {
  const float xs[4] = {x.x, x.y, x.z, x.w};
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t u = __float_as_uint(xs[e]);
    h[e] = u & 0xffff0000u;
    l[e] = __float_as_uint(xs[e] - __uint_as_float(h[e])) & 0xffff0000u;
  }
  hi = make_uint2((h[0] >> 16) | h[1], (h[2] >> 16) | h[3]);
  lo = make_uint2((l[0] >> 16) | l[1], (l[2] >> 16) | l[3]);
}

__device__ __forceinline__ f32x4 mfma3(const bf16x8& ah, const bf16x8& al, const bf16x8& bh,
                                       const bf16x8& bl, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, c, 0, 0, 0);
  return c;
}

// 8 consecutive input elements as floats (16 B for bf16, 32 B for fp32)
__device__ __forceinline__ void ld8(const float* p, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void ld8(const BF16* p, float (&x)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(w[e] << 16);
    x[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
  }
}


// Sum over the 4 lanes of a quad (DPP quad permutations, no LDS traffic).
__device__ __forceinline__ float quad_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // [1,0,3,2]
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // [2,3,0,1]
  return v;
}

// Value of v held by lane src of this wave (ds_bpermute).
__device__ __forceinline__ float lane_gather(float v, int src) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(v)));
}

// LDS regions (bytes) for a tree of T slots, key dim DK and value slice DVS
struct VerifySmem {
  size_t rk, rv, meta, total;
};
__host__ __device__ inline VerifySmem verify_smem(int T, int DK, int DVS) {
  const int TP = (T + 15) & ~15;
  const int kappa = DK >= 32 ? DK : 32;
  const size_t rows = size_t(TP > T + 3 ? TP : T + 3);
  VerifySmem s;
  s.rk = rows * (DK + kKPad) * 4;                           // q staging [T+3][DK+pad], then k~ [TP][DK+pad]
  const size_t k_stage = rows * (DK + kKPad) * 4;           // k staging [T+3][DK+pad]
  const size_t v_tile = rows * (DVS + kKPad) * 4;           // v staging [T+3][DVS+pad], then v~
  const size_t s_tile = size_t(DVS) * (kappa + kSPad) * 2 * 2;  // S0 bf16 hi + lo planes
  s.rv = k_stage > v_tile ? k_stage : v_tile;
  s.rv = s.rv > s_tile ? s.rv : s_tile;
  s.meta = size_t(3 * kVMaxT) * 4                           // order, parent pos, depth
           + size_t(2 * kVMaxT) * 4                         // alpha, beta of the current head
           + size_t(8 * DK) * 4 + size_t(4 * DVS) * 4;      // q/k and v conv weights
  s.total = s.rk + s.rv + s.meta;
  return s;
}

// Issue the loads of this thread's share of S0[b][h][c0 .. c0+DVS][0 .. DK).
template <int DK, int DVS, int NS0>
__device__ __forceinline__ void prefetch_s0(const float* S0bh, int tid, float4 (&pf)[NS0]) {
  constexpr int n4 = DVS * DK / 4;
#pragma unroll
  for (int j = 0; j < NS0; ++j) {
    const int idx = j * kVT + tid;
    pf[j] = idx < n4 ? reinterpret_cast<const float4*>(S0bh)[idx] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// Issue the loads of this thread's share of the raw values v[b][.][h][c0 .. c0+DVS)
// for the T nodes (16-byte chunks, node-major).
template <typename TIn, int DVS, int NVC>
__device__ __forceinline__ void prefetch_v(const TIn* vin, size_t node_stride, const int* s_ord,
                                           int T, int tid, uint4 (&pf)[NVC]) {
  constexpr int EPC = 16 / sizeof(TIn);  // elements per 16-byte chunk
  constexpr int CPR = DVS / EPC;         // chunks per node row
#pragma unroll
  for (int j = 0; j < NVC; ++j) {
    const int idx = j * kVT + tid;
    const int p = idx / CPR, c = idx % CPR;
    pf[j] = p < T ? *reinterpret_cast<const uint4*>(vin + size_t(s_ord[p]) * node_stride + c * EPC)
                  : make_uint4(0, 0, 0, 0);
  }
}

// Write one 16-byte chunk of raw inputs (8 bf16 or 4 fp32) to LDS as fp32.
__device__ __forceinline__ void store_chunk_f32(float* dst, uint4 u, const BF16*) {
  *reinterpret_cast<float4*>(dst) = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                                                __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  *reinterpret_cast<float4*>(dst + 4) = make_float4(__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xffff0000u),
                                                    __uint_as_float(u.w << 16), __uint_as_float(u.w & 0xffff0000u));
}
__device__ __forceinline__ void store_chunk_f32(float* dst, uint4 u, const float*) {
  *reinterpret_cast<float4*>(dst) =
      make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z), __uint_as_float(u.w));
}

template <int DK, int DVS, typename TIn>
__global__ __launch_bounds__(kVT) void verify_kernel(VerifyParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int KPL = DK / 4;                 // key channels per lane: 16 j + 4 lg + e
  constexpr int KB = DK >= 32 ? DK / 32 : 1;  // 32-wide MFMA k blocks (dk = 16 is zero-padded)
  constexpr int KAPPA = 32 * KB;              // MFMA k extent
  constexpr int KROW = DK + kKPad;            // k~ / staging row stride (floats)
  constexpr int NT = DVS / 16;                // 16-row value tiles of this slice
  constexpr int VROW = DVS + kKPad;           // v~ / staging row stride (floats)
  constexpr int EPC = 16 / sizeof(TIn);
  constexpr int NS0 = (DVS * DK / 4 + kVT - 1) / kVT;        // S0 float4 per thread
  constexpr int NVC = (kVMaxT * DVS / EPC + kVT - 1) / kVT;  // raw-v chunks per thread
  constexpr int QCPR = DK / EPC;                             // raw q/k chunks per row
  constexpr int NQC = (kVMaxT * QCPR + kVT - 1) / kVT;       // raw q (or k) chunks per thread

  const int T = p.T;
  const int TP = (T + 15) & ~15;
  const int Hk = p.Hk, Hv = p.Hv, DV = p.DV;
  const int G = Hv / Hk;
  const int nhg = G / p.hpw;
  const int b = blockIdx.z;
  const int g = blockIdx.y / nhg;
  const int h0 = g * G + (blockIdx.y % nhg) * p.hpw;
  const int c0 = blockIdx.x * DVS;  // first value channel of this slice
  const int C = 2 * Hk * DK + Hv * DV;
  const size_t orow = size_t(Hv) * DV;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // quad layout (conv, pull-back): node = 16 wave + lane / 4, channel group lg = lane % 4
  const int qlg = lane & 3;
  const int pos = wave * 16 + (lane >> 2);
  // MFMA layout (product, store): node = 16 wave + lane % 16, channel group = lane / 16
  const int l16 = lane & 15, mlg = lane >> 4;
  const int mpos = wave * 16 + l16;

  const VerifySmem L = verify_smem(T, DK, DVS);
  float* s_k = reinterpret_cast<float*>(smem);  // q staging, then k~ [TP][KROW]
  unsigned char* s_rv = smem + L.rk;            // k staging / v staging / v~ / S0 planes
  float* s_v = reinterpret_cast<float*>(s_rv);  // [.][VROW]
  int* s_ord = reinterpret_cast<int*>(smem + L.rk + L.rv);
  int* s_ppos = s_ord + kVMaxT;
  int* s_dep = s_ppos + kVMaxT;
  float* s_al = reinterpret_cast<float*>(s_dep + kVMaxT);
  float* s_be = s_al + kVMaxT;
  float* s_wqk = s_be + kVMaxT;  // [2][4][DK] tap-major
  float* s_wv = s_wqk + 8 * DK;  // [4][DVS] tap-major

  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int status = m.status[b];
  const int nv = m.nvalid[b];
  if (status != GDN_TREE_OK) {
    for (int hh = 0; hh < p.hpw; ++hh)
      for (int idx = tid; idx < T * DVS; idx += kVT) {
        const int i = idx / DVS, c = idx % DVS;
        p.out[(size_t(b) * T + i) * orow + size_t(h0 + hh) * DV + c0 + c] = 0.0f;
      }
    return;
  }

  // ---------------- phase 0: per-position metadata, prefetches ----------------
  if (tid < T) {
    int node = m.order[b * T + tid];
    node = (node >= 0 && node < T) ? node : 0;  // prepare writes a permutation
    const int pp = m.ppos[b * T + tid];
    s_ord[tid] = node;
    s_dep[tid] = tid < nv ? m.pdep[b * T + tid] : -1;
    s_ppos[tid] = (tid < nv && pp >= 0 && pp < T) ? pp : -1;
  }
  for (int i = tid; i < 8 * DK; i += kVT) {
    const int part = i / (4 * DK), w = (i / DK) & 3, c = i % DK;
    s_wqk[i] = p.conv_w[size_t(part * Hk * DK + g * DK + c) * 4 + w];
  }
  float4 s0pf[NS0];
  prefetch_s0<DK, DVS>(p.S0 + (size_t(b) * Hv + h0) * DV * DK + size_t(c0) * DK, tid, s0pf);
  __syncthreads();
  const TIn* vin = static_cast<const TIn*>(p.v);
  uint4 vpf[NVC];
  prefetch_v<TIn, DVS>(vin + size_t(b) * T * orow + size_t(h0) * DV + c0, orow, s_ord, T, tid, vpf);

  // ---------------- phase 1: q~ and k~ ----------------
  // Raw rows are staged in LDS as fp32, in canonical order, followed by the
  // three conv-state slots, so that every conv tap is an LDS row: tap w of a
  // node at depth d is row tap[w] if d - 3 + w >= 0, else conv-state row
  // T + d + w (slot d + w; slot 2 is the most recent token).  q is staged
  // in the k~ region and k in the value region; all loads are issued first.
  {
    const size_t qk_row = size_t(Hk) * DK;
    const TIn* qsrc = static_cast<const TIn*>(p.q) + size_t(b) * T * qk_row + size_t(g) * DK;
    const TIn* ksrc = static_cast<const TIn*>(p.k) + size_t(b) * T * qk_row + size_t(g) * DK;
    uint4 qpf[NQC], kpf[NQC];
#pragma unroll
    for (int j = 0; j < NQC; ++j) {
      const int idx = j * kVT + tid;
      const int row = idx / QCPR, c = (idx % QCPR) * EPC;
      if (row < T) {
        const size_t off = size_t(s_ord[row]) * qk_row + c;
        qpf[j] = *reinterpret_cast<const uint4*>(qsrc + off);
        kpf[j] = *reinterpret_cast<const uint4*>(ksrc + off);
      }
    }
    float* s_kst = reinterpret_cast<float*>(s_rv);
#pragma unroll
    for (int j = 0; j < NQC; ++j) {
      const int idx = j * kVT + tid;
      const int row = idx / QCPR, c = (idx % QCPR) * EPC;
      if (row < T) {
        store_chunk_f32(s_k + row * KROW + c, qpf[j], static_cast<const TIn*>(nullptr));
        store_chunk_f32(s_kst + row * KROW + c, kpf[j], static_cast<const TIn*>(nullptr));
      }
    }
    const float* csq = p.conv_state + size_t(b) * 3 * C + g * DK;
    for (int i = tid; i < 3 * DK; i += kVT) {
      const int sl = i / DK, c = i % DK;
      s_k[(T + sl) * KROW + c] = csq[size_t(sl) * C + c];
      s_kst[(T + sl) * KROW + c] = csq[size_t(sl) * C + Hk * DK + c];
    }
  }
  __syncthreads();
  const bool active = pos < nv;
  int trow[4] = {0, 0, 0, 0};
  if (active) {
    const int dep = s_dep[pos];
    const int t2 = s_ppos[pos];
    const int t1 = t2 >= 0 ? s_ppos[t2] : -1;
    const int t0 = t1 >= 0 ? s_ppos[t1] : -1;
    const int tp[4] = {t0, t1, t2, pos};
#pragma unroll
    for (int w = 0; w < 4; ++w) trow[w] = (dep - 3 + w >= 0) ? tp[w] : T + dep + w;
  }
  float qh[KPL];  // q~ of this lane's node (channels 16 j + 4 lg + e)
  float kh[KPL];
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const float* stage = part == 0 ? s_k : reinterpret_cast<const float*>(s_rv);
    float y[KPL];
#pragma unroll
    for (int c = 0; c < KPL; ++c) y[c] = 0.0f;
    if (active) {
      const float* wpart = s_wqk + part * 4 * DK;
#pragma unroll
      for (int j = 0; j < DK / 16; ++j) {
        const int c = 16 * j + 4 * qlg;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float4 x = *reinterpret_cast<const float4*>(stage + trow[w] * KROW + c);
          const float4 wt = *reinterpret_cast<const float4*>(wpart + w * DK + c);
          y[4 * j] += wt.x * x.x;
          y[4 * j + 1] += wt.y * x.y;
          y[4 * j + 2] += wt.z * x.z;
          y[4 * j + 3] += wt.w * x.w;
        }
      }
    }
    float ss = 0.0f;
#pragma unroll
    for (int c = 0; c < KPL; ++c) {
      y[c] = silu(y[c]);
      ss += y[c] * y[c];
    }
    ss = quad_sum(ss);
    const float inv = rsqrt_hw(ss + 1e-6f);
#pragma unroll
    for (int c = 0; c < KPL; ++c) {
      if (part == 0)
        qh[c] = active ? y[c] * inv : 0.0f;
      else
        kh[c] = active ? y[c] * inv : 0.0f;
    }
  }
  __syncthreads();  // staged rows consumed
  if (active) {
#pragma unroll
    for (int j = 0; j < DK / 16; ++j)
      *reinterpret_cast<float4*>(s_k + pos * KROW + 16 * j + 4 * qlg) =
          make_float4(kh[4 * j], kh[4 * j + 1], kh[4 * j + 2], kh[4 * j + 3]);
  }

  // ---------------- phase 2: one value head at a time ----------------
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  const int src_lane = 4 * l16 + mlg;  // quad-layout lane holding this MFMA lane's data
  for (int hh = 0; hh < p.hpw; ++hh) {
    const int h = h0 + hh;
    // 2a: raw v rows (prefetched) + 3 conv-state rows -> LDS as fp32
    //     [T + 3][VROW]; gates and v conv weights -> LDS
    const int vch0 = 2 * Hk * DK + h * DV + c0;  // conv channel of v[h][c0]
    {
      constexpr int CPR = DVS / EPC;
#pragma unroll
      for (int j = 0; j < NVC; ++j) {
        const int idx = j * kVT + tid;
        if (idx < T * CPR) {
          const int row = idx / CPR, c = (idx % CPR) * EPC;
          store_chunk_f32(s_v + row * VROW + c, vpf[j], static_cast<const TIn*>(nullptr));
        }
      }
      const float* cs = p.conv_state + size_t(b) * 3 * C + vch0;
      for (int i = tid; i < 3 * DVS; i += kVT)
        s_v[(T + i / DVS) * VROW + i % DVS] = cs[size_t(i / DVS) * C + i % DVS];
    }
    if (tid < T) {
      const size_t ab = (size_t(b) * T + s_ord[tid]) * Hv + h;
      s_al[tid] = ld(alpha, ab);
      s_be[tid] = ld(beta, ab);
    }
    for (int i = tid; i < 4 * DVS; i += kVT)
      s_wv[i] = p.conv_w[size_t(vch0 + i % DVS) * 4 + i / DVS];
    __syncthreads();
    // 2b: v~ for this lane's node and value channels 16 n + 4 lg + e
    float vt[4 * NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) {
#pragma unroll
      for (int e = 0; e < 4; ++e) vt[4 * n + e] = 0.0f;
      if (active) {
        const int c = 16 * n + 4 * qlg;
        float y[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float4 x = *reinterpret_cast<const float4*>(s_v + trow[w] * VROW + c);
          const float4 wt = *reinterpret_cast<const float4*>(s_wv + w * DVS + c);
          y[0] += wt.x * x.x;
          y[1] += wt.y * x.y;
          y[2] += wt.z * x.z;
          y[3] += wt.w * x.w;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) vt[4 * n + e] = silu(y[e]);
      }
    }
    __syncthreads();  // staged rows consumed
    if (active) {
#pragma unroll
      for (int n = 0; n < NT; ++n)
          *reinterpret_cast<float4*>(s_v + pos * VROW + 16 * n + 4 * qlg) =
              make_float4(vt[4 * n], vt[4 * n + 1], vt[4 * n + 2], vt[4 * n + 3]);
    }
    if (hh + 1 < p.hpw)
      prefetch_v<TIn, DVS>(vin + size_t(b) * T * orow + size_t(h + 1) * DV + c0, orow, s_ord, T, tid, vpf);
    __syncthreads();

    // 2c: query pull-back along the path, leaf to root (quad layout)
    float x[KPL];
    float acc[4 * NT];
#pragma unroll
    for (int c = 0; c < KPL; ++c) x[c] = qh[c];
#pragma unroll
    for (int c = 0; c < 4 * NT; ++c) acc[c] = 0.0f;
    float r = 1.0f;
    {
      int t = active ? pos : -1;
      // a path has at most T nodes; the bound also ends the walk on corrupt metadata
      for (int step = 0; step < T && t >= 0; ++step) {
        float kt[KPL];
#pragma unroll
        for (int j = 0; j < DK / 16; ++j) {
          const float4 k4 = *reinterpret_cast<const float4*>(s_k + t * KROW + 16 * j + 4 * qlg);
          kt[4 * j] = k4.x;
          kt[4 * j + 1] = k4.y;
          kt[4 * j + 2] = k4.z;
          kt[4 * j + 3] = k4.w;
        }
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int c = 0; c < KPL; c += 2) {
          s0 += kt[c] * x[c];
          s1 += kt[c + 1] * x[c + 1];
        }
        const float s = quad_sum(s0 + s1);
        const float bs = s_be[t] * s;
        const float rbs = r * bs;
#pragma unroll
        for (int c = 0; c < KPL; ++c) x[c] -= bs * kt[c];
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          const float4 v4 = *reinterpret_cast<const float4*>(s_v + t * VROW + 16 * n + 4 * qlg);
          acc[4 * n] += rbs * v4.x;
          acc[4 * n + 1] += rbs * v4.y;
          acc[4 * n + 2] += rbs * v4.z;
          acc[4 * n + 3] += rbs * v4.w;
        }
        r *= s_al[t];
        t = s_ppos[t];
      }
    }
    // a_i x~_i and the value accumulators move from the quad layout to the
    // MFMA layout (same node and channel group, different lane)
#pragma unroll
    for (int c = 0; c < KPL; ++c) x[c] = lane_gather(x[c] * r, src_lane);
#pragma unroll
    for (int c = 0; c < 4 * NT; ++c) acc[c] = lane_gather(acc[c], src_lane);
    __syncthreads();  // v~ consumed

    // 2d: S0 of this head -> LDS as bf16 hi/lo planes [DVS][KAPPA + kSPad].
    //     The MFMA k index kappa = 32 kb + 8 lg + 4 h + e holds key channel
    //     32 kb + 16 h + 4 lg + e, the channel that MFMA lane group lg holds
    //     in register 8 kb + 4 h + e of the pulled-back query.
    {
      uint16_t* s_hi = reinterpret_cast<uint16_t*>(s_rv);
      uint16_t* s_lo = s_hi + DVS * (KAPPA + kSPad);
#pragma unroll
      for (int j = 0; j < NS0; ++j) {
        const int idx = j * kVT + tid;
        if (NS0 * kVT == DVS * DK / 4 || idx < DVS * DK / 4) {
          const int row = idx / (DK / 4), mch = idx % (DK / 4);  // physical chunk m
          const int kch = 8 * (mch / 8) + 2 * (mch % 4) + (mch / 4) % 2;
          uint2 hi, lo;
          split4(s0pf[j], hi, lo);
          *reinterpret_cast<uint2*>(s_hi + row * (KAPPA + kSPad) + 4 * kch) = hi;
          *reinterpret_cast<uint2*>(s_lo + row * (KAPPA + kSPad) + 4 * kch) = lo;
        }
      }
      if (DK < 32) {  // odd kappa chunks carry no channel: zero them
        for (int i = tid; i < DVS * 4; i += kVT) {
          const int row = i / 4, kch = 2 * (i % 4) + 1;
          *reinterpret_cast<uint2*>(s_hi + row * (KAPPA + kSPad) + 4 * kch) = make_uint2(0, 0);
          *reinterpret_cast<uint2*>(s_lo + row * (KAPPA + kSPad) + 4 * kch) = make_uint2(0, 0);
        }
      }
    }
    if (hh + 1 < p.hpw)
      prefetch_s0<DK, DVS>(p.S0 + (size_t(b) * Hv + h + 1) * DV * DK + size_t(c0) * DK, tid, s0pf);
    __syncthreads();

    // 2e: O^T = S0 X~^T + ACC^T on MFMA (MFMA layout); store
    if (wave * 16 < TP) {
      bf16x8 xh[KB], xl[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        float x8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x8[e] = (8 * kb + e < KPL) ? x[(8 * kb + e) % KPL] : 0.0f;
        split8(x8, xh[kb], xl[kb]);
      }
      const uint16_t* s_hi = reinterpret_cast<const uint16_t*>(s_rv);
      const uint16_t* s_lo = s_hi + DVS * (KAPPA + kSPad);
      const int node = mpos < T ? s_ord[mpos] : 0;
      float* orow_p = p.out + (size_t(b) * T + node) * orow + size_t(h) * DV + c0;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        {
          f32x4 d = {acc[4 * n], acc[4 * n + 1], acc[4 * n + 2], acc[4 * n + 3]};
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            const int off = (16 * n + l16) * (KAPPA + kSPad) + 32 * kb + 8 * mlg;
            const bf16x8 ah = *reinterpret_cast<const bf16x8*>(s_hi + off);
            const bf16x8 al = *reinterpret_cast<const bf16x8*>(s_lo + off);
            d = mfma3(ah, al, xh[kb], xl[kb], d);
          }
          if (mpos < T)
            *reinterpret_cast<float4*>(orow_p + 16 * n + 4 * mlg) =
                make_float4(d[0] * p.scale, d[1] * p.scale, d[2] * p.scale, d[3] * p.scale);
        }
      }
    }
    __syncthreads();  // S0 planes consumed before the next head reuses the region
  }
}

template <int DK, int DVS, typename TIn>
static int launch_verify_t(const VerifyArgs& a, int hpw, int ns, hipStream_t stream) {
  VerifyParams p;
  p.B = a.B;
  p.T = a.T;
  p.Hk = a.Hk;
  p.Hv = a.Hv;
  p.DV = a.dv;
  p.hpw = hpw;
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
  const size_t smem = verify_smem(a.T, DK, DVS).total;
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&verify_kernel<DK, DVS, TIn>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(verify_smem(kVMaxT, DK, DVS).total));
    if (e != hipSuccess)
      return set_error(GDN_EHIP, "verify: LDS attribute: %s", hipGetErrorString(e));
    attr_done = true;
  }
  const int G = a.Hv / a.Hk;
  hipLaunchKernelGGL((verify_kernel<DK, DVS, TIn>), dim3(ns, a.Hk * (G / hpw), a.B), dim3(kVT), smem,
                     stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "verify launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

template <int DK, typename TIn>
static int dispatch_dvs(const VerifyArgs& a, hipStream_t s) {
  // Work split: all value heads of a key head share one workgroup (one q/k
  // conv) when that still gives >= 256 workgroups; otherwise one value head
  // per workgroup and, for small batches, the value dim split into slices.
  const int G = a.Hv / a.Hk;
  int hpw = G, ns = 1;
  if (size_t(a.B) * a.Hk < 256) {
    hpw = 1;
    while (size_t(a.B) * a.Hv * ns < 256 && a.dv / (2 * ns) >= 32) ns *= 2;
  }
  switch (a.dv / ns) {
    case 16: return launch_verify_t<DK, 16, TIn>(a, hpw, ns, s);
    case 32: return launch_verify_t<DK, 32, TIn>(a, hpw, ns, s);
    case 64: return launch_verify_t<DK, 64, TIn>(a, hpw, ns, s);
    case 128: return launch_verify_t<DK, 128, TIn>(a, hpw, ns, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify: dv=%d unsupported", a.dv);
}

template <typename TIn>
static int dispatch_dk(const VerifyArgs& a, hipStream_t s) {
  switch (a.dk) {
    case 16: return dispatch_dvs<16, TIn>(a, s);
    case 32: return dispatch_dvs<32, TIn>(a, s);
    case 64: return dispatch_dvs<64, TIn>(a, s);
    case 128: return dispatch_dvs<128, TIn>(a, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify: dk=%d unsupported", a.dk);
}

int launch_verify(const VerifyArgs& a, hipStream_t stream) {
  if (a.T > kVMaxT) return set_error(GDN_EUNSUPPORTED, "verify: T=%d exceeds %d", a.T, kVMaxT);
  if (a.in_dtype == GDN_BF16) return dispatch_dk<BF16>(a, stream);
  return dispatch_dk<float>(a, stream);
}

}  // namespace gdn
