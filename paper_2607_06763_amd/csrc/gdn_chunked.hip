// gdn_chunked.hip -- tree verification in the paper's chunked form
// (Sec. 3.4.1, Eq. 9-13) on the MFMA units.
//
// With positions in canonical (topological) order, a_i the product of alpha
// over the path root..i, and q, k, v the post-conv features of one
// (sequence, value head), the outputs of Eq. 7-8 for every node are
//     X_ij = [j strict ancestor of i] beta_i (a_i / a_j) k_i.k_j      (Eq. 9)
//     Y_ij = [j ancestor of i or i]  (a_i / a_j) q_i.k_j
//     (I + X) U~ = beta (V - a K S0^T)                    (Eq. 10, W S0 folded)
//     O = scale (a Q S0^T + Y U~)                          (Eq. 11)
// in the stored orientation (S0 in R^{dv x dk}).  X is strictly lower
// triangular, so U~ follows from a forward substitution over 16-node blocks
// (Eq. 13): U~_b = (I + X_bb)^{-1} (R_b - sum_{c<b} X_bc U~_c).
//
// Workgroup = one (sequence b, value head h), 512 threads = 8 waves; wave w
// owns the 16 positions of block w.  Phases:
//   0  metadata -> LDS: order, depth, parent position, ancestor-or-self
//      masks in position space, log a (sum of log alpha over the mask), beta
//   1  conv + SiLU + L2 norm of q, k for the wave's own 16 nodes straight
//      from the raw rows (tap rows gathered from HBM/L2, conv-state slots from
//      LDS); k~ of all nodes -> LDS as bf16 hi/lo planes
//   2  Gram on MFMA: G_QK, G_KK rows of the own nodes against every earlier
//      block (lower triangle only)
//   3  S0 -> LDS as bf16 hi/lo planes; v~ of the own nodes -> LDS (fp32)
//   4  P = [Q; K]_own S0^T on MFMA
//   5  R = beta (v - a P_K), O = a P_Q; (I + X_bb)^{-1} of the own diagonal
//      block by forward substitution (fp32, 16 lanes)
//   6  block cascade: block c is solved by its wave (Inv x Acc), published to
//      LDS, and every later block subtracts X_bc U~_c and adds Y_bc U~_c to
//      its outputs; one barrier per block
//   7  store O
// All products use a bf16 hi/lo split of both operands (three products,
// fp32 accumulation, ~1e-5 relative): v_mfma_f32_16x16x32_bf16 where the
// contraction runs over head channels, v_mfma_f32_16x16x16_bf16 where it runs
// over the 16 nodes of a block.
#include <math.h>

#include "gdn_internal.h"

namespace gdn {

constexpr int kQT = 512;       // threads per workgroup (8 waves)
constexpr int kQMaxT = 128;    // tree slots = 8 blocks of 16
constexpr int kQPad = 8;       // bf16 row padding of the operand planes
constexpr int kQVPad = 4;      // fp32 row padding of the v~ tile

typedef short s16x4 __attribute__((ext_vector_type(4)));

struct ChunkParams {
  int B, T, Hk, Hv;
  float scale;
  const void* meta;
  const void *q, *k, *v, *alpha, *beta;
  const float *conv_w, *conv_state, *S0;
  float* out;
};

// LDS regions (bytes)
struct ChunkSmem {
  size_t planes, vtile, meta, total;
};
__host__ __device__ inline ChunkSmem chunk_smem(int T, int DK, int DV) {
  const int TP = (T + 15) & ~15;
  const int NB = TP / 16;
  ChunkSmem s;
  const size_t kpl = size_t(TP) * (DK + kQPad) * 2 * 2;      // k~ planes (hi, lo)
  const size_t spl = size_t(DV) * (DK + kQPad) * 2 * 2;      // S0 planes
  const size_t upl = size_t(NB) * (DV / 16) * 64 * 8 * 2;    // published U~ blocks (hi, lo)
  s.planes = kpl > spl ? kpl : spl;
  s.planes = s.planes > upl ? s.planes : upl;
  const size_t vt = size_t(TP) * (DV + kQVPad) * 4;          // v~ tile
  const size_t inv = size_t(8) * 16 * 16 * 4;                 // per-wave 16 x 16 scratch
  s.vtile = vt > inv ? vt : inv;
  s.meta = size_t(kQMaxT) * 8 * 2                             // ancestor words of the node at each position
           + size_t(kQMaxT) * 4 * 6                           // order, depth, ppos, log alpha, log a, beta
           + size_t(kQMaxT) * 4 * 4                           // ancestor-or-self masks (4 words)
           + size_t(3 * 2 * DK + 3 * DV) * 4                  // conv-state slots of q, k, v
           + size_t(4 * 2 * DK + 4 * DV) * 4;                 // conv weights of q, k, v (tap-major)
  s.total = s.planes + s.vtile + s.meta;
  return s;
}

// 4 floats -> bf16 hi / lo (truncation split)
__device__ __forceinline__ void split4s(const float (&x)[4], s16x4& hi, s16x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t u = __float_as_uint(x[e]);
    const uint32_t h = u & 0xffff0000u;
    hi[e] = short(h >> 16);
    lo[e] = short(__float_as_uint(x[e] - __uint_as_float(h)) >> 16);
  }
}

// Three 16x16x16 bf16 products of hi/lo split operands into fp32.
__device__ __forceinline__ f32x4 mfma16x3(const s16x4& ah, const s16x4& al, const s16x4& bh, const s16x4& bl,
                                          f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(al, bh, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ah, bl, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ah, bh, c, 0, 0, 0);
  return c;
}

// 8 raw input channels of one row (16-byte or 2 x 16-byte load), kept raw
// until used so that no wait is forced at the load.
template <typename TIn>
struct Raw8;
template <>
struct Raw8<BF16> {
  uint4 u;
  __device__ __forceinline__ void load(const BF16* p) { u = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void get(float (&x)[8]) const {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <>
struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ void get(float (&x)[8]) const {
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
};

// Width-4 conv + SiLU of one node for the channels 32 g + 8 m + e (g < D/32,
// e < 8) of one head: tap w reads the raw row of node tnode[w] when
// tcs[w] < 0, else conv-state slot tcs[w] (LDS).  load() issues the four
// tap rows; silu_conv() consumes them.
template <int D, typename TIn>
struct ConvTaps {
  static constexpr int G = D / 32;
  Raw8<TIn> raw[4][G];
  __device__ __forceinline__ void load(const TIn* src, size_t rowlen, const int (&tnode)[4], int m) {
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int g = 0; g < G; ++g) raw[w][g].load(src + size_t(tnode[w]) * rowlen + 32 * g + 8 * m);
  }
  __device__ __forceinline__ void silu_conv(const int (&tcs)[4], const float* s_w, const float* s_cs, int m,
                                            float (&y)[G][8]) const {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) y[g][e] = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int sl = tcs[w] < 0 ? 0 : tcs[w];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int c0 = 32 * g + 8 * m;
        float x[8];
        raw[w][g].get(x);
        const float4 wa = *reinterpret_cast<const float4*>(s_w + w * D + c0);
        const float4 wb = *reinterpret_cast<const float4*>(s_w + w * D + c0 + 4);
        const float4 ca = *reinterpret_cast<const float4*>(s_cs + sl * D + c0);
        const float4 cb = *reinterpret_cast<const float4*>(s_cs + sl * D + c0 + 4);
        const float wt[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
        const float cv[8] = {ca.x, ca.y, ca.z, ca.w, cb.x, cb.y, cb.z, cb.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) y[g][e] += wt[e] * (tcs[w] < 0 ? x[e] : cv[e]);
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) y[g][e] = silu(y[g][e]);
  }
};

// L2 normalisation over the node's 4 lanes (lane bits 4 and 5) and bf16
// hi/lo split per 32-channel block
template <int KB>
__device__ __forceinline__ void norm_split(float (&y)[KB][8], bool real, bf16x8 (&hi)[KB], bf16x8 (&lo)[KB]) {
  float ss = 0.0f;
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += y[kb][e] * y[kb][e];
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  const float inv = real ? rsqrt_hw(ss + 1e-6f) : 0.0f;
#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
    for (int e = 0; e < 8; ++e) y[kb][e] *= inv;
    split8(y[kb], hi[kb], lo[kb]);
  }
}

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(kQT) void chunked_verify_kernel(ChunkParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int KB = DK / 32;   // 32-channel k blocks
  constexpr int NTV = DV / 16;  // 16-channel value tiles
  constexpr int VG = DV / 32;   // 32-channel value groups (conv layout)
  constexpr int KROW = DK + kQPad;
  constexpr int VROW = DV + kQVPad;
  constexpr int NBM = kQMaxT / 16;

  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int TP = (T + 15) & ~15;
  const int NB = TP / 16;
  const int h = blockIdx.x, b = blockIdx.y;
  const int g = h * Hk / Hv;
  const int C = 2 * Hk * DK + Hv * DV;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, m = lane >> 4;
  const size_t orow = size_t(Hv) * DV;
  // block of 16 positions owned by this wave: waves w and w + 4 share a SIMD
  // and take blocks w and 7 - w, which evens out the lower-triangular work
  const int blk = wave < 4 ? wave : 11 - wave;
  const bool owner = blk < NB;
  const int pos = 16 * blk + r;

  const ChunkSmem L = chunk_smem(T, DK, DV);
  unsigned char* s_planes = smem;
  float* s_v = reinterpret_cast<float*>(smem + L.planes);  // v~ tile, later the 16 x 16 scratch
  uint64_t* s_anc = reinterpret_cast<uint64_t*>(smem + L.planes + L.vtile);  // [kQMaxT][2]
  int* s_ord = reinterpret_cast<int*>(s_anc + 2 * kQMaxT);
  int* s_dep = s_ord + kQMaxT;
  int* s_ppos = s_dep + kQMaxT;
  float* s_lal = reinterpret_cast<float*>(s_ppos + kQMaxT);  // log alpha by position
  float* s_la = s_lal + kQMaxT;                              // log a by position
  float* s_be = s_la + kQMaxT;                               // beta by position (0 for padding)
  uint32_t* s_pm = reinterpret_cast<uint32_t*>(s_be + kQMaxT);  // [kQMaxT][4]
  float* s_cq = reinterpret_cast<float*>(s_pm + 4 * kQMaxT);   // [3][DK]
  float* s_ck = s_cq + 3 * DK;                                  // [3][DK]
  float* s_cv = s_ck + 3 * DK;                                  // [3][DV]
  float* s_wq = s_cv + 3 * DV;                                  // [4][DK]
  float* s_wk = s_wq + 4 * DK;                                  // [4][DK]
  float* s_wv = s_wk + 4 * DK;                                  // [4][DV]

  const MetaPtrs mp = meta_ptrs(p.meta, p.B, T);
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);

  // ---------------- phase 0: metadata, gates, conv weights and state ----------------
  // The first load wave issues every load that does not depend on the tree
  // (status, order / depth / parent position, conv weights and state, S0);
  // the second the gates and ancestor words of the node at each position
  // together with the raw q / k / v rows of the conv taps.  The status is
  // tested after the first wave (every address is valid whatever the status).
  const int status = mp.status[b];
  const int nv = mp.nvalid[b];
  int node = 0, pdep = -1, pp = -1;
  if (tid < kQMaxT && tid < T) {
    node = mp.order[size_t(b) * T + tid];
    pdep = mp.pdep[size_t(b) * T + tid];
    pp = mp.ppos[size_t(b) * T + tid];
  }
  static_assert(4 * DK <= kQT && 4 * DV <= kQT, "one conv weight / state element per thread");
  float cqv = 0.f, ckv = 0.f, cvv = 0.f, wqv = 0.f, wkv = 0.f, wvv = 0.f;
  {
    const float* cs = p.conv_state + size_t(b) * 3 * C;
    const int iq = tid < 3 * DK ? tid : 0, iv = tid < 3 * DV ? tid : 0;
    const int jq = tid < 4 * DK ? tid : 0, jv = tid < 4 * DV ? tid : 0;
    cqv = cs[size_t(iq / DK) * C + g * DK + iq % DK];
    ckv = cs[size_t(iq / DK) * C + Hk * DK + g * DK + iq % DK];
    cvv = cs[size_t(iv / DV) * C + 2 * Hk * DK + h * DV + iv % DV];
    wqv = p.conv_w[size_t(g * DK + jq % DK) * 4 + jq / DK];
    wkv = p.conv_w[size_t(Hk * DK + g * DK + jq % DK) * 4 + jq / DK];
    wvv = p.conv_w[size_t(2 * Hk * DK + h * DV + jv % DV) * 4 + jv / DV];
  }
  // S0 of this head: issued now, stored as planes after the Gram
  constexpr int NS0 = (DV * DK / 4 + kQT - 1) / kQT;
  float4 s0pf[NS0];
  {
    const float4* S0bh = reinterpret_cast<const float4*>(p.S0 + (size_t(b) * Hv + h) * DV * DK);
#pragma unroll
    for (int j = 0; j < NS0; ++j) {
      const int idx = j * kQT + tid;
      s0pf[j] = S0bh[idx < DV * DK / 4 ? idx : 0];
    }
  }
  if (tid < kQMaxT) {
    node = (node >= 0 && node < T) ? node : 0;
    const bool real = tid < T && tid < nv;
    s_ord[tid] = node;
    s_dep[tid] = real ? pdep : -1;
    s_ppos[tid] = (real && pp >= 0 && pp < T) ? pp : -1;
  }
  if (tid < 3 * DK) {
    s_cq[tid] = cqv;
    s_ck[tid] = ckv;
  }
  if (tid < 3 * DV) s_cv[tid] = cvv;
  if (tid < 4 * DK) {
    s_wq[tid] = wqv;
    s_wk[tid] = wkv;
  }
  if (tid < 4 * DV) s_wv[tid] = wvv;
  // second load wave, part 1: gates and ancestor words of the node at position tid
  TIn g_al = TIn(), g_be = TIn();
  uint64_t g_a0 = 0ull, g_a1 = 0ull;
  if (tid < kQMaxT) {
    const size_t ab = (size_t(b) * T + node) * Hv + h;
    g_al = alpha[ab];
    g_be = beta[ab];
    g_a0 = mp.anc[(size_t(b) * T + node) * mp.W];
    g_a1 = mp.W > 1 ? mp.anc[(size_t(b) * T + node) * mp.W + 1] : 0ull;
  }
  if (status != GDN_TREE_OK) {
    for (int idx = tid; idx < T * DV; idx += kQT)
      p.out[(size_t(b) * T + idx / DV) * orow + size_t(h) * DV + idx % DV] = 0.0f;
    return;
  }
  __syncthreads();  // order, depth, parent positions, conv weights / state in LDS

  // second load wave, part 2: the conv tap rows of the own node (position
  // pos = 16 blk + r, channels 32 g + 8 m + e)
  const bool preal = owner && pos < nv;
  int tnode[4], tcs[4];
  {
    const int pc = preal ? pos : 0;
    const int dep = preal ? s_dep[pc] : 0;
    const int t2 = preal ? s_ppos[pc] : -1;
    const int t1 = t2 >= 0 ? s_ppos[t2] : -1;
    const int t0 = t1 >= 0 ? s_ppos[t1] : -1;
    const int tp[4] = {t0, t1, t2, pc};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const bool fromrow = dep - 3 + w >= 0;
      tnode[w] = (fromrow && tp[w] >= 0) ? s_ord[tp[w]] : 0;
      tcs[w] = fromrow ? -1 : dep + w;
    }
  }
  const size_t qk_row = size_t(Hk) * DK;
  const TIn* qsrc = static_cast<const TIn*>(p.q) + size_t(b) * T * qk_row + size_t(g) * DK;
  const TIn* ksrc = static_cast<const TIn*>(p.k) + size_t(b) * T * qk_row + size_t(g) * DK;
  ConvTaps<DK, TIn> tq, tk;
  tq.load(qsrc, qk_row, tnode, m);

  if (tid < kQMaxT) {
    const bool real = tid < T && tid < nv;
    s_lal[tid] = real ? __logf(to_f32(g_al)) : 0.0f;
    s_be[tid] = real ? to_f32(g_be) : 0.0f;
    s_anc[2 * tid] = g_a0;
    s_anc[2 * tid + 1] = g_a1;
  }
  __syncthreads();
  // ancestor-or-self masks in position space: bit q of word q / 32 of s_pm[p]
  {
    const int pi = tid >> 2, wd = tid & 3;
    uint32_t bits = 0;
    if (pi < nv) {
      const uint64_t a0 = s_anc[2 * pi], a1 = s_anc[2 * pi + 1];
      for (int qq = 0; qq < 32; ++qq) {
        const int q = 32 * wd + qq;
        if (q < nv) {
          const int nq = s_ord[q];
          const uint64_t aw = nq < 64 ? a0 : a1;
          const bool set = q == pi || ((aw >> (nq & 63)) & 1ull);
          bits |= set ? (1u << qq) : 0u;
        }
      }
    }
    s_pm[pi * 4 + wd] = bits;
  }
  __syncthreads();
  // log a_p = sum of log alpha over the ancestors of p and p itself
  if (tid < kQMaxT) {
    float la = 0.0f;
#pragma unroll
    for (int wd = 0; wd < 4; ++wd) {
      uint32_t bits = s_pm[tid * 4 + wd];
      while (bits) {
        const int qq = __builtin_ctz(bits);
        bits &= bits - 1;
        la += s_lal[32 * wd + qq];
      }
    }
    s_la[tid] = la;
  }

  // ---------------- phase 1: q~, k~ of the own nodes ----------------
  bf16x8 qh[KB], ql[KB], kh[KB], kl[KB];
  {
    float y[KB][8];
    tq.silu_conv(tcs, s_wq, s_cq, m, y);
    norm_split<KB>(y, preal, qh, ql);
    tk.load(ksrc, qk_row, tnode, m);
    tk.silu_conv(tcs, s_wk, s_ck, m, y);
    norm_split<KB>(y, preal, kh, kl);
  }
  // the value rows load during the Gram
  ConvTaps<DV, TIn> tv;
  tv.load(static_cast<const TIn*>(p.v) + size_t(b) * T * orow + size_t(h) * DV, orow, tnode, m);
  if (owner) {
    uint16_t* s_kh = reinterpret_cast<uint16_t*>(s_planes);
    uint16_t* s_kl = s_kh + size_t(TP) * KROW;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      *reinterpret_cast<bf16x8*>(s_kh + pos * KROW + 32 * kb + 8 * m) = kh[kb];
      *reinterpret_cast<bf16x8*>(s_kl + pos * KROW + 32 * kb + 8 * m) = kl[kb];
    }
  }
  __syncthreads();  // k~ planes and s_la complete

  // ---------------- phase 2: Gram rows of the own nodes ----------------
  // lane (r, m): GQ[n][e] = q_i.k_j, GK[n][e] = k_i.k_j with i = 16 blk + r,
  // j = 16 n + 4 m + e, for the blocks n <= blk
  f32x4 GQ[NBM], GK[NBM];
#pragma unroll
  for (int n = 0; n < NBM; ++n) {
    GQ[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    GK[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (owner) {
    const uint16_t* s_kh = reinterpret_cast<const uint16_t*>(s_planes);
    const uint16_t* s_kl = s_kh + size_t(TP) * KROW;
#pragma unroll
    for (int n = 0; n < NBM; ++n) {
      if (n <= blk) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int off = (16 * n + r) * KROW + 32 * kb + 8 * m;
          const bf16x8 ah = *reinterpret_cast<const bf16x8*>(s_kh + off);
          const bf16x8 al = *reinterpret_cast<const bf16x8*>(s_kl + off);
          GQ[n] = mfma3(ah, al, qh[kb], ql[kb], GQ[n]);
          GK[n] = mfma3(ah, al, kh[kb], kl[kb], GK[n]);
        }
      }
    }
  }
  __syncthreads();  // k~ planes consumed

  // ---------------- phase 3: S0 planes, v~ of the own nodes ----------------
  {
    uint16_t* s_sh = reinterpret_cast<uint16_t*>(s_planes);
    uint16_t* s_sl = s_sh + size_t(DV) * KROW;
#pragma unroll
    for (int j = 0; j < NS0; ++j) {
      const int idx = j * kQT + tid;
      if (idx < DV * DK / 4) {
        const int row = idx / (DK / 4), kq = idx % (DK / 4);
        const float x4[4] = {s0pf[j].x, s0pf[j].y, s0pf[j].z, s0pf[j].w};
        s16x4 hi, lo;
        split4s(x4, hi, lo);
        *reinterpret_cast<s16x4*>(s_sh + row * KROW + 4 * kq) = hi;
        *reinterpret_cast<s16x4*>(s_sl + row * KROW + 4 * kq) = lo;
      }
    }
  }
  if (owner) {
    float y[VG][8];
    tv.silu_conv(tcs, s_wv, s_cv, m, y);
#pragma unroll
    for (int vg = 0; vg < VG; ++vg) {
      float* dst = s_v + pos * VROW + 32 * vg + 8 * m;
      *reinterpret_cast<float4*>(dst) =
          preal ? make_float4(y[vg][0], y[vg][1], y[vg][2], y[vg][3]) : make_float4(0.f, 0.f, 0.f, 0.f);
      *reinterpret_cast<float4*>(dst + 4) =
          preal ? make_float4(y[vg][4], y[vg][5], y[vg][6], y[vg][7]) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  __syncthreads();

  // ---------------- phase 4: P = [Q; K]_own S0^T; R and a P_Q ----------------
  // lane (r, m): O[t][e] = a_i (S0 q_i)[16 t + r], Acc[t][e] = R[i][16 t + r]
  // with i = 16 blk + 4 m + e
  f32x4 O[NTV], Acc[NTV];
#pragma unroll
  for (int t = 0; t < NTV; ++t) {
    O[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    Acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  if (owner) {
    const uint16_t* s_sh = reinterpret_cast<const uint16_t*>(s_planes);
    const uint16_t* s_sl = s_sh + size_t(DV) * KROW;
#pragma unroll
    for (int t = 0; t < NTV; ++t) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int off = (16 * t + r) * KROW + 32 * kb + 8 * m;
        const bf16x8 bh = *reinterpret_cast<const bf16x8*>(s_sh + off);
        const bf16x8 bl = *reinterpret_cast<const bf16x8*>(s_sl + off);
        O[t] = mfma3(qh[kb], ql[kb], bh, bl, O[t]);
        Acc[t] = mfma3(kh[kb], kl[kb], bh, bl, Acc[t]);
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int pe = 16 * blk + 4 * m + e;
      const bool re = pe < nv;
      const float a = re ? __expf(s_la[pe]) : 0.0f;
      const float be = re ? s_be[pe] : 0.0f;
#pragma unroll
      for (int t = 0; t < NTV; ++t) {
        const float vv = s_v[pe * VROW + 16 * t + r];
        O[t][e] = a * O[t][e];
        Acc[t][e] = be * (vv - a * Acc[t][e]);
      }
    }
  }
  __syncthreads();  // S0 planes and v~ tile consumed

  // ---------------- phase 5: coefficients, diagonal-block inverse ----------------
  // lane (r, m), block n: xs = -X_ij, ys = Y_ij with i = 16 blk + r,
  // j = 16 n + 4 m + e, as bf16 hi/lo A operands of the 16x16x16 products
  s16x4 xh[NBM], xl[NBM], yh[NBM], yl[NBM];
  float* sx = s_v + wave * 256;  // [16][16] row-major scratch of this wave
  {
    uint32_t pm[4];
#pragma unroll
    for (int wd = 0; wd < 4; ++wd) pm[wd] = owner ? s_pm[pos * 4 + wd] : 0u;
    const float la_i = owner ? s_la[pos] : 0.0f;
    const float be_i = preal ? s_be[pos] : 0.0f;
#pragma unroll
    for (int n = 0; n < NBM; ++n) {
      float x[4] = {0.f, 0.f, 0.f, 0.f}, y[4] = {0.f, 0.f, 0.f, 0.f};
      if (owner && n <= blk) {
        const uint32_t word = pm[n >> 1];  // j < 32 (n / 2 + 1) for every lane
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = 16 * n + 4 * m + e;
          const bool anc = (word >> (j & 31)) & 1u;  // j ancestor of i, or i
          const float dec = anc ? __expf(la_i - s_la[j]) : 0.0f;
          x[e] = (anc && j != pos) ? -be_i * dec * GK[n][e] : 0.0f;
          y[e] = dec * GQ[n][e];
        }
        if (n == blk)
          *reinterpret_cast<float4*>(sx + r * 16 + 4 * m) = make_float4(-x[0], -x[1], -x[2], -x[3]);
      }
      split4s(x, xh[n], xl[n]);
      split4s(y, yh[n], yl[n]);
    }
  }
  // (I + X_bb)^{-1}: forward substitution by the 16 lanes of column c
  s16x4 ivh = {0, 0, 0, 0}, ivl = {0, 0, 0, 0};
  if (owner) {
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the tile is complete for the whole wave
    __builtin_amdgcn_wave_barrier();
    if (m == 0) {
      float inv[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float xr[16];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 v4 = *reinterpret_cast<const float4*>(sx + i * 16 + 4 * q4);
          xr[4 * q4] = v4.x;
          xr[4 * q4 + 1] = v4.y;
          xr[4 * q4 + 2] = v4.z;
          xr[4 * q4 + 3] = v4.w;
        }
        float s = i == r ? 1.0f : 0.0f;
#pragma unroll
        for (int mm = 0; mm < i; ++mm) s -= xr[mm] * inv[mm];
        inv[i] = s;
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) sx[i * 16 + r] = inv[i];
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    const float4 iv = *reinterpret_cast<const float4*>(sx + r * 16 + 4 * m);
    const float ivx[4] = {iv.x, iv.y, iv.z, iv.w};
    split4s(ivx, ivh, ivl);
  }

  // ---------------- phase 6: block cascade (Eq. 13) ----------------
  // block c: U~_c = Inv_cc Acc_c by its wave, published to LDS; after one
  // barrier every later block subtracts X_bc U~_c from its Acc
  uint2* s_uh = reinterpret_cast<uint2*>(s_planes);
  uint2* s_ul = s_uh + size_t(NB) * NTV * 64;
#pragma unroll
  for (int c = 0; c < NBM; ++c) {
    if (c < NB) {
      if (blk == c) {
        // all tiles split first, then the products tile-interleaved, so that
        // no product waits for the previous one's result
        s16x4 bh[NTV], bl[NTV];
#pragma unroll
        for (int t = 0; t < NTV; ++t) {
          const float a4[4] = {Acc[t][0], Acc[t][1], Acc[t][2], Acc[t][3]};
          split4s(a4, bh[t], bl[t]);
        }
        f32x4 u[NTV];
#pragma unroll
        for (int t = 0; t < NTV; ++t)
          u[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ivl, bh[t], f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
#pragma unroll
        for (int t = 0; t < NTV; ++t) u[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ivh, bl[t], u[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < NTV; ++t) u[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ivh, bh[t], u[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < NTV; ++t) {
          const float u4[4] = {u[t][0], u[t][1], u[t][2], u[t][3]};
          s16x4 uh, ul;
          split4s(u4, uh, ul);
          s_uh[(c * NTV + t) * 64 + lane] = __builtin_bit_cast(uint2, uh);
          s_ul[(c * NTV + t) * 64 + lane] = __builtin_bit_cast(uint2, ul);
        }
      }
      __syncthreads();
      if (owner && blk > c) {
        s16x4 uh[NTV], ul[NTV];
#pragma unroll
        for (int t = 0; t < NTV; ++t) {
          uh[t] = __builtin_bit_cast(s16x4, s_uh[(c * NTV + t) * 64 + lane]);
          ul[t] = __builtin_bit_cast(s16x4, s_ul[(c * NTV + t) * 64 + lane]);
        }
#pragma unroll
        for (int t = 0; t < NTV; ++t) Acc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(xl[c], uh[t], Acc[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < NTV; ++t) Acc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(xh[c], ul[t], Acc[t], 0, 0, 0);
#pragma unroll
        for (int t = 0; t < NTV; ++t) Acc[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(xh[c], uh[t], Acc[t], 0, 0, 0);
      }
    }
  }

  // ---------------- phase 7: O += Y U~ (every published block), store ----------------
  if (owner) {
#pragma unroll
    for (int c = 0; c < NBM; ++c) {
      if (c <= blk) {
#pragma unroll
        for (int t = 0; t < NTV; ++t) {
          const s16x4 uh = __builtin_bit_cast(s16x4, s_uh[(c * NTV + t) * 64 + lane]);
          const s16x4 ul = __builtin_bit_cast(s16x4, s_ul[(c * NTV + t) * 64 + lane]);
          O[t] = mfma16x3(yh[c], yl[c], uh, ul, O[t]);
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int pe = 16 * blk + 4 * m + e;
      if (pe < T) {
        float* dst = p.out + (size_t(b) * T + s_ord[pe]) * orow + size_t(h) * DV + r;
#pragma unroll
        for (int t = 0; t < NTV; ++t) dst[16 * t] = p.scale * O[t][e];
      }
    }
  }
}

template <int DK, int DV, typename TIn>
static int launch_chunked_t(const VerifyArgs& a, hipStream_t stream) {
  ChunkParams p;
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
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&chunked_verify_kernel<DK, DV, TIn>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(chunk_smem(kQMaxT, DK, DV).total));
    if (e != hipSuccess) return set_error(GDN_EHIP, "verify_chunked: LDS attribute: %s", hipGetErrorString(e));
    attr_done = true;
  }
  hipLaunchKernelGGL((chunked_verify_kernel<DK, DV, TIn>), dim3(a.Hv, a.B), dim3(kQT),
                     chunk_smem(a.T, DK, DV).total, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "verify_chunked launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

template <int DK, typename TIn>
static int chunked_dv(const VerifyArgs& a, hipStream_t s) {
  switch (a.dv) {
    case 32: return launch_chunked_t<DK, 32, TIn>(a, s);
    case 64: return launch_chunked_t<DK, 64, TIn>(a, s);
    case 128: return launch_chunked_t<DK, 128, TIn>(a, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify_chunked: dv=%d unsupported (32, 64, 128)", a.dv);
}

template <typename TIn>
static int chunked_dk(const VerifyArgs& a, hipStream_t s) {
  switch (a.dk) {
    case 32: return chunked_dv<32, TIn>(a, s);
    case 64: return chunked_dv<64, TIn>(a, s);
    case 128: return chunked_dv<128, TIn>(a, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify_chunked: dk=%d unsupported (32, 64, 128)", a.dk);
}

int launch_verify_chunked(const VerifyArgs& a, hipStream_t stream) {
  if (a.T > kQMaxT) return set_error(GDN_EUNSUPPORTED, "verify_chunked: T=%d exceeds %d", a.T, kQMaxT);
  if (a.in_dtype == GDN_BF16) return chunked_dk<BF16>(a, stream);
  return chunked_dk<float>(a, stream);
}

}  // namespace gdn
