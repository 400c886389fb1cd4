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
  int B, T, Hk, Hv, nslices, hpw;
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

// LDS regions (bytes) for a tree of T slots, key dim DK and value slice DVS
struct VerifySmem {
  size_t rk, rv, meta, total;
};
__host__ __device__ inline VerifySmem verify_smem(int T, int DK, int DVS) {
  const int TP = (T + 15) & ~15;
  VerifySmem s;
  const size_t k_tile = size_t(TP) * (DK + kKPad) * 4;    // k~ (fp32)
  const size_t k_stage = size_t(T + 3) * DK * 4;           // raw q or k rows + 3 conv-state rows
  s.rk = k_tile > k_stage ? k_tile : k_stage;
  const size_t v_tile = size_t(TP) * (DVS + kKPad) * 4;   // v~ (fp32)
  const size_t v_stage = size_t(T + 3) * DVS * 4;          // raw v rows + 3 conv-state rows
  const size_t s_tile = size_t(DVS) * (DK + kSPad) * 2 * 2;  // S0 bf16 hi + lo planes
  s.rv = v_tile > v_stage ? v_tile : v_stage;
  s.rv = s.rv > s_tile ? s.rv : s_tile;
  s.meta = size_t(3 * kVMaxT) * 4                          // order, parent pos, depth
           + size_t(2 * kVMaxT) * 4                        // alpha, beta of the current head
           + size_t(8 * DK) * 4 + size_t(4 * DVS) * 4;     // q/k and v conv weights
  s.total = s.rk + s.rv + s.meta;
  return s;
}

// Issue the loads of this thread's share of S0[b][h][c0 .. c0+DVS][0 .. DK).
template <int DK, int NS0>
__device__ __forceinline__ void prefetch_s0(const float* S0bh, int DVS, int tid, float4 (&pf)[NS0]) {
  const int n4 = DVS * DK / 4;
#pragma unroll
  for (int j = 0; j < NS0; ++j) {
    const int idx = j * kVT + tid;
    pf[j] = idx < n4 ? reinterpret_cast<const float4*>(S0bh)[idx] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// Issue the loads of this thread's share of the raw values v[b][.][h][c0 .. c0+DVS)
// for the T nodes (16-byte chunks, node-major).
template <typename TIn, int NVC>
__device__ __forceinline__ void prefetch_v(const TIn* vin, size_t node_stride, const int* s_ord,
                                           int T, int DVS, int tid, uint4 (&pf)[NVC]) {
  constexpr int EPC = 16 / sizeof(TIn);  // elements per 16-byte chunk
  const int sh = __builtin_ctz(DVS / EPC);  // log2 of the chunks per node row (a power of two)
#pragma unroll
  for (int j = 0; j < NVC; ++j) {
    const int idx = j * kVT + tid;
    const int p = idx >> sh, c = idx & ((1 << sh) - 1);
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

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(kVT) void verify_kernel(VerifyParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int KB = DK >= 32 ? DK / 32 : 1;  // 32-wide key blocks (dk = 16 is zero-padded)
  constexpr int KPL = 8 * KB;                 // key channels per lane (padding included)
  constexpr int KROW = DK + kKPad;            // k~ row stride (floats)
  constexpr int NT_MAX = DV / 16;             // 16-row value tiles
  constexpr int EPC = 16 / sizeof(TIn);
  constexpr int NS0 = (DV * DK / 4 + kVT - 1) / kVT;                   // S0 float4 per thread
  constexpr int NVC = (kVMaxT * DV / EPC + kVT - 1) / kVT;             // raw-v chunks per thread

  const int T = p.T;
  const int TP = (T + 15) & ~15;
  const int Hk = p.Hk, Hv = p.Hv;
  const int G = Hv / Hk;
  const int nhg = G / p.hpw;
  const int b = blockIdx.z;
  const int g = blockIdx.y / nhg;
  const int h0 = g * G + (blockIdx.y % nhg) * p.hpw;
  const int DVS = DV / p.nslices;
  const int c0 = blockIdx.x * DVS;   // first value channel of this slice
  const int NT = DVS / 16;
  const int C = 2 * Hk * DK + Hv * DV;
  const size_t orow = size_t(Hv) * DV;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int pos = wave * 16 + l16;   // tree position owned by this lane

  const VerifySmem L = verify_smem(T, DK, DVS);
  float* s_k = reinterpret_cast<float*>(smem);                 // [TP][KROW]
  unsigned char* s_rv = smem + L.rk;                           // raw v / v~ / S0 planes
  float* s_v = reinterpret_cast<float*>(s_rv);                 // [TP][DVS + kKPad]
  int* s_ord = reinterpret_cast<int*>(smem + L.rk + L.rv);
  int* s_ppos = s_ord + kVMaxT;
  int* s_dep = s_ppos + kVMaxT;
  float* s_al = reinterpret_cast<float*>(s_dep + kVMaxT);
  float* s_be = s_al + kVMaxT;
  float* s_wqk = s_be + kVMaxT;                                // [2][DK][4]
  float* s_wv = s_wqk + 8 * DK;                                // [DVS][4]
  const int VROW = DVS + kKPad;

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

  // ---------------- phase 0 ----------------
  if (tid < T) {
    int node = m.order[b * T + tid];
    node = (node >= 0 && node < T) ? node : 0;  // prepare writes a permutation
    const bool real = tid < nv;
    s_ord[tid] = node;
    s_dep[tid] = real ? m.depth[b * T + node] : -1;
    const int par = m.parent[b * T + node];
    s_ppos[tid] = (real && par >= 0 && par < T) ? m.pos[b * T + par] : -1;
  }
  for (int i = tid; i < 8 * DK; i += kVT) {  // tap-major: s_wqk[part][w][c]
    const int part = i / (4 * DK), w = (i / DK) & 3, c = i % DK;
    s_wqk[i] = p.conv_w[size_t(part * Hk * DK + g * DK + c) * 4 + w];
  }
  float4 s0pf[NS0];
  prefetch_s0<DK>(p.S0 + (size_t(b) * Hv + h0) * DV * DK + size_t(c0) * DK, DVS, tid, s0pf);
  __syncthreads();
  const TIn* vin = static_cast<const TIn*>(p.v);
  uint4 vpf[NVC];
  prefetch_v<TIn>(vin + size_t(b) * T * orow + size_t(h0) * DV + c0, orow, s_ord, T, DVS, tid, vpf);

  // ---------------- phase 1: q~ and k~ ----------------
  // Raw rows are staged in LDS as fp32, in canonical order, followed by the
  // three conv-state slots, so that every conv tap is an LDS row: tap w of a
  // node at depth d is row tap[w] if d - 3 + w >= 0, else conv-state row
  // T + d + w (slot d + w; slot 2 is the most recent token).
  const bool active = pos < nv;
  int trow[4] = {0, 0, 0, 0};
  int dep = -1;
  if (active) {
    dep = s_dep[pos];
    int t2 = s_ppos[pos];
    int t1 = t2 >= 0 ? s_ppos[t2] : -1;
    int t0 = t1 >= 0 ? s_ppos[t1] : -1;
    const int tp[4] = {t0, t1, t2, pos};
#pragma unroll
    for (int w = 0; w < 4; ++w) trow[w] = (dep - 3 + w >= 0) ? tp[w] : T + dep + w;
  }
  float qh[KPL];  // q~ of this lane's node, later the start of the pull-back
  float kh[KPL];
  const TIn* qk_src[2] = {static_cast<const TIn*>(p.q), static_cast<const TIn*>(p.k)};
  const size_t qk_row = size_t(Hk) * DK;
  float* s_stage = s_k;  // [T + 3][DK] fp32
#pragma unroll 1
  for (int part = 0; part < 2; ++part) {
    const TIn* src = qk_src[part] + size_t(b) * T * qk_row + size_t(g) * DK;
    const float* cs = p.conv_state + size_t(b) * 3 * C + part * Hk * DK + g * DK;
    constexpr int cpr = DK / 4;  // float4 chunks per row
    for (int idx = tid; idx < (T + 3) * cpr; idx += kVT) {
      const int row = idx / cpr, c = (idx % cpr) * 4;
      const float4 x = row < T ? ld4(src + size_t(s_ord[row]) * qk_row + c)
                               : ld4(cs + size_t(row - T) * C + c);
      *reinterpret_cast<float4*>(s_stage + row * DK + c) = x;
    }
    __syncthreads();
    float y[KPL];
#pragma unroll
    for (int c = 0; c < KPL; ++c) y[c] = 0.0f;
    if (active) {
      const float* wpart = s_wqk + part * 4 * DK;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int c = 32 * kb + 8 * lg;
        if (c < DK) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            float x[8], wt[8];
            ld8(s_stage + trow[w] * DK + c, x);
            ld8(wpart + w * DK + c, wt);
#pragma unroll
            for (int e = 0; e < 8; ++e) y[8 * kb + e] += wt[e] * x[e];
          }
        }
      }
    }
    float ss = 0.0f;
#pragma unroll
    for (int c = 0; c < KPL; ++c) {
      y[c] = silu(y[c]);  // silu(0) = 0 keeps padding channels at zero
      ss += y[c] * y[c];
    }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    const float inv = rsqrt_hw(ss + 1e-6f);
    if (part == 0) {
#pragma unroll
      for (int c = 0; c < KPL; ++c) qh[c] = active ? y[c] * inv : 0.0f;
    } else {
#pragma unroll
      for (int c = 0; c < KPL; ++c) kh[c] = active ? y[c] * inv : 0.0f;
    }
    __syncthreads();  // staged rows consumed
  }
  if (active) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const int c = 32 * kb + 8 * lg;
      if (c < DK) {
        *reinterpret_cast<float4*>(s_k + pos * KROW + c) =
            make_float4(kh[8 * kb], kh[8 * kb + 1], kh[8 * kb + 2], kh[8 * kb + 3]);
        *reinterpret_cast<float4*>(s_k + pos * KROW + c + 4) =
            make_float4(kh[8 * kb + 4], kh[8 * kb + 5], kh[8 * kb + 6], kh[8 * kb + 7]);
      }
    }
  }

  // ---------------- phase 2: one value head at a time ----------------
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  for (int hh = 0; hh < p.hpw; ++hh) {
    const int h = h0 + hh;
    // 2a: raw v rows (prefetched) + 3 conv-state rows -> LDS as fp32
    //     [T + 3][DVS]; gates and v conv weights -> LDS
    const int vch0 = 2 * Hk * DK + h * DV + c0;  // conv channel of v[h][c0]
    {
      float* s_vs = reinterpret_cast<float*>(s_rv);
      const int sh = __builtin_ctz(DVS / EPC);
#pragma unroll
      for (int j = 0; j < NVC; ++j) {
        const int idx = j * kVT + tid;
        if (idx < (T << sh)) {
          const int row = idx >> sh, c = (idx & ((1 << sh) - 1)) * EPC;
          store_chunk_f32(s_vs + row * DVS + c, vpf[j], static_cast<const TIn*>(nullptr));
        }
      }
      const float* cs = p.conv_state + size_t(b) * 3 * C + vch0;
      for (int i = tid; i < 3 * DVS; i += kVT) s_vs[(T + i / DVS) * DVS + i % DVS] = cs[size_t(i / DVS) * C + i % DVS];
    }
    if (tid < T) {
      const size_t ab = (size_t(b) * T + s_ord[tid]) * Hv + h;
      s_al[tid] = ld(alpha, ab);
      s_be[tid] = ld(beta, ab);
    }
    for (int i = tid; i < 4 * DVS; i += kVT)  // tap-major: s_wv[w][c]
      s_wv[i] = p.conv_w[size_t(vch0 + i % DVS) * 4 + i / DVS];
    __syncthreads();
    // 2b: v~ for this lane's node and value channels 16n + 4lg + e
    float vt[4 * NT_MAX];
    {
      const float* s_vs = reinterpret_cast<const float*>(s_rv);
#pragma unroll
      for (int n = 0; n < NT_MAX; ++n) {
#pragma unroll
        for (int e = 0; e < 4; ++e) vt[4 * n + e] = 0.0f;
        if (active && n < NT) {
          const int c = 16 * n + 4 * lg;
          float y[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const float4 x = ld4(s_vs + trow[w] * DVS + c);
            const float4 wt = ld4(s_wv + w * DVS + c);
            y[0] += wt.x * x.x;
            y[1] += wt.y * x.y;
            y[2] += wt.z * x.z;
            y[3] += wt.w * x.w;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) vt[4 * n + e] = silu(y[e]);
        }
      }
    }
    __syncthreads();  // raw v consumed
    if (active) {
#pragma unroll
      for (int n = 0; n < NT_MAX; ++n)
        if (n < NT)
          *reinterpret_cast<float4*>(s_v + pos * VROW + 16 * n + 4 * lg) =
              make_float4(vt[4 * n], vt[4 * n + 1], vt[4 * n + 2], vt[4 * n + 3]);
    }
    if (hh + 1 < p.hpw)
      prefetch_v<TIn>(vin + size_t(b) * T * orow + size_t(h + 1) * DV + c0, orow, s_ord, T, DVS, tid, vpf);
    __syncthreads();

    // 2c: query pull-back along the path, leaf to root
    float x[KPL];
    float acc[4 * NT_MAX];
#pragma unroll
    for (int c = 0; c < KPL; ++c) x[c] = qh[c];
#pragma unroll
    for (int c = 0; c < 4 * NT_MAX; ++c) acc[c] = 0.0f;
    float r = 1.0f;
    {
      int t = active ? pos : -1;
      // a path has at most T nodes; the bound also ends the walk on corrupt metadata
      for (int step = 0; step < T; ++step) {
        if (t < 0) break;
        float kt[KPL];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int c = 32 * kb + 8 * lg;
          float k8[8];
          if (c < DK) {
            ld8(s_k + t * KROW + c, k8);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) k8[e] = 0.0f;
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) kt[8 * kb + e] = k8[e];
        }
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int c = 0; c < KPL; c += 2) {
          s0 += kt[c] * x[c];
          s1 += kt[c + 1] * x[c + 1];
        }
        float s = s0 + s1;
        s += __shfl_xor(s, 16);
        s += __shfl_xor(s, 32);
        const float bs = s_be[t] * s;
        const float rbs = r * bs;
#pragma unroll
        for (int c = 0; c < KPL; ++c) x[c] -= bs * kt[c];
#pragma unroll
        for (int n = 0; n < NT_MAX; ++n) {
          if (n < NT) {
            const float4 v4 = *reinterpret_cast<const float4*>(s_v + t * VROW + 16 * n + 4 * lg);
            acc[4 * n] += rbs * v4.x;
            acc[4 * n + 1] += rbs * v4.y;
            acc[4 * n + 2] += rbs * v4.z;
            acc[4 * n + 3] += rbs * v4.w;
          }
        }
        r *= s_al[t];
        t = s_ppos[t];
      }
    }
#pragma unroll
    for (int c = 0; c < KPL; ++c) x[c] *= r;  // a_i x~_i
    __syncthreads();  // v~ consumed

    // 2d: S0 of this head -> LDS as bf16 hi/lo planes [DVS][DK + kSPad]
    {
      uint16_t* s_hi = reinterpret_cast<uint16_t*>(s_rv);
      uint16_t* s_lo = s_hi + DVS * (DK + kSPad);
#pragma unroll
      for (int j = 0; j < NS0; ++j) {
        const int idx = j * kVT + tid;
        if (idx < DVS * DK / 4) {
          const int row = idx / (DK / 4), col = (idx % (DK / 4)) * 4;
          uint2 hi, lo;
          split4(s0pf[j], hi, lo);
          *reinterpret_cast<uint2*>(s_hi + row * (DK + kSPad) + col) = hi;
          *reinterpret_cast<uint2*>(s_lo + row * (DK + kSPad) + col) = lo;
        }
      }
    }
    if (hh + 1 < p.hpw)
      prefetch_s0<DK>(p.S0 + (size_t(b) * Hv + h + 1) * DV * DK + size_t(c0) * DK, DVS, tid, s0pf);
    __syncthreads();

    // 2e: O^T = S0 X~^T + ACC^T on MFMA; store
    if (wave * 16 < TP) {
      bf16x8 xh[KB], xl[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        float x8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x8[e] = x[8 * kb + e];
        split8(x8, xh[kb], xl[kb]);
      }
      const uint16_t* s_hi = reinterpret_cast<const uint16_t*>(s_rv);
      const uint16_t* s_lo = s_hi + DVS * (DK + kSPad);
      const int node = pos < T ? s_ord[pos] : 0;
      float* orow_p = p.out + (size_t(b) * T + node) * orow + size_t(h) * DV + c0;
#pragma unroll
      for (int n = 0; n < NT_MAX; ++n) {
        if (n < NT) {
          f32x4 d = {acc[4 * n], acc[4 * n + 1], acc[4 * n + 2], acc[4 * n + 3]};
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) {
            const int c = 32 * kb + 8 * lg;
            bf16x8 ah, al;
            if (c < DK) {
              const int off = (16 * n + l16) * (DK + kSPad) + c;
              ah = *reinterpret_cast<const bf16x8*>(s_hi + off);
              al = *reinterpret_cast<const bf16x8*>(s_lo + off);
            } else {
              ah = bf16x8{};
              al = bf16x8{};
            }
            d = mfma3(ah, al, xh[kb], xl[kb], d);
          }
          if (pos < T)
            *reinterpret_cast<float4*>(orow_p + 16 * n + 4 * lg) =
                make_float4(d[0] * p.scale, d[1] * p.scale, d[2] * p.scale, d[3] * p.scale);
        }
      }
    }
    __syncthreads();  // S0 planes consumed before the next head reuses the region
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
  // Work split: all value heads of a key head share one workgroup (one q/k
  // conv) when that still gives >= 256 workgroups; otherwise one value head
  // per workgroup and, for small batches, the value dim split across slices.
  const int G = a.Hv / a.Hk;
  int hpw = G, ns = 1;
  if (size_t(a.B) * a.Hk < 256) {
    hpw = 1;
    while (size_t(a.B) * a.Hv * ns < 256 && DV / (2 * ns) >= 32) ns *= 2;
  }
  p.hpw = hpw;
  p.nslices = ns;
  const size_t smem = verify_smem(a.T, DK, DV / ns).total;
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&verify_kernel<DK, DV, TIn>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(verify_smem(kVMaxT, DK, DV).total));
    if (e != hipSuccess)
      return set_error(GDN_EHIP, "verify: LDS attribute: %s", hipGetErrorString(e));
    attr_done = true;
  }
  hipLaunchKernelGGL((verify_kernel<DK, DV, TIn>), dim3(ns, a.Hk * (G / hpw), a.B), dim3(kVT), smem,
                     stream, p);
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
