// gdn_coef.hip -- tree verification, commit and the fused decode step through
// one GDN layer, with every dense product on the MFMA units.
//
// The output of node i is Eq. 7 applied along i's path from the cached state
// S0 and read out with q_i (Eq. 8).  Walking the path from the leaf to the
// root, Eq. 7 in the stored orientation (S in R^{dv x dk}) gives, for any x,
//     S_t x = alpha_t S_{t-1} (x - beta_t (k_t . x) k_t) + beta_t (k_t . x) v_t,
// so with path nodes t_0 = i, t_1 = parent(i), ..., t_d = root,
//     s_m = k_{t_m} . x_m,   x_{m+1} = x_m - beta s_m k_{t_m},   x_0 = q_i,
// every s_m is a scalar recurrence over Gram entries:
//     s_m = (q_i . k_{t_m}) - sum_{m' < m} c_{m'} (k_{t_m'} . k_{t_m}),
//     c_m = beta_{t_m} s_m,
// and the node's output is
//     o_i = scale ( a_i S0 (q_i - sum_m c_m k_{t_m}) + sum_m r_m c_m v_{t_m} ),
// r_m = prod_{m' < m} alpha_{t_m'}, a_i = product of alpha over the path
// (Sec. 3.4.1: cumulative decay).  Per (sequence, value head) the vector work
// is then three dense products,
//     X~^T = (a Q)^T - K^T C'^T      (C'[i][t] = a_i c, the node's path only)
//     O^T  = S0 X~^T + V^T D^T       (D[i][t]  = r c)
// on v_mfma_f32_16x16x32_f16 (fp16 operands, fp32 accumulation), and the
// per-node scalar recurrences need only the ancestor entries of the Gram
// products Q K^T and K K^T, themselves MFMA products per key head.  This is
// the paper's ancestor-masked chunk form (Eq. 9-11) solved per node instead
// of with a block forward substitution: the triangular system of node i has
// only its depth + 1 unknowns.
//
// The commit (Sec. 3.4.2: the one state write, after the accepted node is
// known) uses the same algebra in its WY form: along the path p_0..p_{L-1},
// S_L = A S0 + sum_j u~_j k_j^T with u_j = beta_j (v_j - alpha_j S_j k_j),
// where S_j k_j = (prod) S0 k_j + sum_{m<j} (...) (k_m . k_j) u_m is updated
// as a recurrence over the dv-vectors u (32 path nodes at a time):
//     P = S0 Kp^T  and  S_L^T = A S0^T + Kp^T U~^T
// run as bf16 hi/lo three-product MFMAs (round-to-nearest splits, about
// 2^-16 relative error).
//
// Workgroup: 512 threads (8 waves) for one key head g of one sequence b and
// hpw of its value heads (GQA, Sec. 3.4.2 "for all heads").  The head dims
// are padded to 128 (zero channels).  Wave w owns state rows (value
// channels) 16w..16w+15 and key channels 16w..16w+15.  The state of a value
// head stays in registers in the accumulator layout of S^T (lane (lg, l16)
// holds S[16w + l16][16t + 4lg + i]); the same registers, with the key index
// permuted inside each 32-block, are the A operand of the verify product.
//
// Per key head: raw q, k staged in LDS by canonical position -> width-4
// conv along each node's path + SiLU + L2 norm (16 lanes per node) -> Q~, K~
// (fp16 rows) -> Gram tiles -> ragged tables QK[p][depth] (ancestors and
// self) and G[p][depth] (proper ancestors) in fp16 -> K~^T MFMA operand and
// Q~ accumulator init in registers.
// Per value head: raw v staged -> conv + SiLU in the MFMA operand layout;
// (step / commit) commit of the previous accepted path into the state
// registers, stored; row scales; coefficient recurrences (4 or 16 lanes per
// node) -> C', D as MFMA operand tiles in LDS; X~ product -> LDS; output
// product -> out.
#include <utility>

#include "gdn_internal.h"

namespace gdn {

constexpr int kCT = 512;          // threads per workgroup
constexpr int kCD = 128;          // padded head dim
constexpr int kCMaxT = 128;       // tree slots (the LDS tiles hold all nodes)
constexpr int kQRow = kCD + 8;    // fp16 row stride of the Q~ / K~ tiles (272 B)
constexpr int kPC = 32;           // commit path nodes per chunk
constexpr int kKpRow = kCD + 4;   // fp32 row stride of the path-key tile
constexpr int kGpRow = kPC + 1;   // fp32 row stride of the path Gram tile
constexpr int kFrag = 1024;       // bytes of one 16x32 fp16 MFMA operand tile (64 lanes x 16 B)

enum { kModeVerify = 0, kModeStep = 1, kModeCommit = 2 };

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));

struct CoefParams {
  int B, T, Hk, Hv, DK, DV, hpw;
  float scale;
  // verify side (verify / step): the current tree and its raw inputs
  const void* meta;
  const void *q, *k, *v, *alpha, *beta;
  const float* conv_w;
  const float* conv_state;  // before the commit
  const float* S0;          // verify: read-only state
  float* out;
  // commit side (step / commit): the tree whose accepted node is committed
  const void* pmeta;
  const int32_t* paccepted;
  const void *pq, *pk, *pv, *palpha, *pbeta;
  float* conv_state_out;  // step: conv state after the commit
  float* S;               // step / commit: state, in place
  int32_t* commit_status;
};

// Fixed-size per-workgroup tables at the start of LDS.
struct CoefMeta {
  int ord[kCMaxT];     // node at canonical position p
  int ppos[kCMaxT];    // position of the parent (-1 root / padding)
  int pdep[kCMaxT];    // depth (-1 padding)
  uint32_t tap[kCMaxT];  // staged rows of the 4 conv taps (8 bits each)
  int qoff[kCMaxT + 4];  // start of position p's row in the ragged tables
  uint64_t ancp[kCMaxT][2];  // proper ancestors in position space
  float a[kCMaxT];     // path decay product of the node at p (this head)
  float al[kCMaxT], be[kCMaxT];  // gates by position (this head)
  float wv[4][kCD];    // v conv weights of this head, tap-major
  float rs[kCD];       // inverse power-of-two scale of each state row
  float rsv[kCD];      // inverse power-of-two scale of each v~ channel
  float4 gt[kCMaxT];   // per position: beta, alpha, start of its G-table row
  int ppath[kCMaxT];   // committed path, root first (slots of the commit tree)
  float pal[kCMaxT], pbe[kCMaxT], psuf[kCMaxT];  // its gates; suffix products
  float cso[3][kCD];   // conv-state slots before the commit (v channels of this head)
  int misc[16];
};

struct CoefSmem {
  size_t tab, kp, big, total;
  int TR;  // rows of the Q~ / K~ tiles: T rounded up to 32
};

__host__ __device__ inline int coef_nfrag(int NT) { return ((NT + 1) * (NT + 1)) / 4; }

__host__ __device__ inline CoefSmem coef_smem(int T, int mode, int in_bytes) {
  CoefSmem s;
  const int NT = (T + 15) / 16;
  s.TR = 32 * ((T + 31) / 32);
  const size_t meta = (sizeof(CoefMeta) + 255) & ~size_t(255);
  // ragged tables (T^2 entries at most) or fixed rows (2 x kDRow T)
  const size_t tab_entries = size_t(T) * T > 2 * 66 * size_t(T) ? size_t(T) * T : 2 * 66 * size_t(T);
  const size_t tab = mode == kModeCommit ? 0 : ((2 * tab_entries + 255) & ~size_t(255));
  // path keys, path Gram, U~ transposes (8 waves x [kPC][16])
  const size_t kp = mode == kModeVerify ? 0
                                        : ((size_t(kPC) * kKpRow * 4 + size_t(kPC) * kGpRow * 4 +
                                            8 * size_t(kPC) * 16 * 4 + 255) & ~size_t(255));
  const size_t stage = size_t(T + 3) * (kCD + 4) * 4;
  const size_t qk = 2 * size_t(s.TR) * kQRow * 2;
  const size_t frags = 2 * size_t(coef_nfrag(NT)) * kFrag + 4 * size_t(NT) * kFrag;
  size_t big = 0;
  if (mode != kModeCommit) {
    big = stage > qk ? stage : qk;
    big = big > frags ? big : frags;
  }
  s.tab = meta;
  s.kp = s.tab + tab;
  s.big = s.kp + kp;
  s.total = s.big + ((big + 255) & ~size_t(255));
  return s;
}

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ f32x4 mma16(const h8& a, const h8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// bf16 hi/lo split with round-to-nearest: x = hi + lo + O(2^-17 |x|)
__device__ __forceinline__ void split_rne8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = (__bf16)x[e];
    hi[e] = h;
    lo[e] = (__bf16)(x[e] - (float)h);
  }
}

// Workgroup barrier that orders LDS accesses only: global loads and stores
// issued before it stay in flight (a full __syncthreads would wait for all
// of them, which exposes the latency of every load issued ahead of use).  No
// thread of these kernels reads global memory that another thread writes.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// LDS ordering among the lanes of one wave
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// Broadcast of lane SRC of every group of NL lanes (NL = 4: quads, 16: rows)
template <int NL, int SRC>
__device__ __forceinline__ float bcast(float x) {
  static_assert((NL == 4 && SRC < 4) || (NL == 16 && SRC < 16), "broadcast group");
  if constexpr (NL == 4)
    return dpp_f<SRC * 0x55>(x);  // quad_perm [SRC, SRC, SRC, SRC]
  else
    return dpp_f<0x150 + SRC>(x);  // row_newbcast:SRC
}

// The thread index as a value the compiler cannot see through: addresses
// derived from it inside the head loop are computed where they are used
// instead of being hoisted out of the loop and kept in registers across it.
__device__ __forceinline__ int opaque_i(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// f(integral_constant<int, I>) for I = 0 .. N-1, unrolled at compile time
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ float hmax4(float v) {  // max over lanes l, l^16, l^32, l^48
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

__device__ __forceinline__ int wave_max_i(int v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v = max(v, __shfl_xor(v, o));
  return v;
}

// Power-of-two scale that brings a row's largest magnitude m into [1, 2)
// (exact; inv = 1 / scale).  Zero or subnormal rows keep scale 1.
__device__ __forceinline__ void pow2_scale(float m, float& scale, float& inv) {
  int ex = int((__float_as_uint(m) >> 23) & 0xffu);
  if (ex == 0) {
    scale = inv = 1.0f;
    return;
  }
  ex = ex > 253 ? 253 : ex;
  scale = __uint_as_float(uint32_t(254 - ex) << 23);
  inv = __uint_as_float(uint32_t(ex) << 23);
}

// 8 raw inputs starting at element e0 of a row (16-byte aligned), as fp32
__device__ __forceinline__ void load8(const BF16* src, float (&x)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(src);
  x[0] = __uint_as_float(u.x << 16);
  x[1] = __uint_as_float(u.x & 0xffff0000u);
  x[2] = __uint_as_float(u.y << 16);
  x[3] = __uint_as_float(u.y & 0xffff0000u);
  x[4] = __uint_as_float(u.z << 16);
  x[5] = __uint_as_float(u.z & 0xffff0000u);
  x[6] = __uint_as_float(u.w << 16);
  x[7] = __uint_as_float(u.w & 0xffff0000u);
}
__device__ __forceinline__ void load8(const float* src, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(src);
  const float4 c = *reinterpret_cast<const float4*>(src + 4);
  x[0] = a.x;
  x[1] = a.y;
  x[2] = a.z;
  x[3] = a.w;
  x[4] = c.x;
  x[5] = c.y;
  x[6] = c.z;
  x[7] = c.w;
}

// Byte offset of element (position pos, node column n) in the fragment
// array of a coefficient matrix: block (kb = pos / 32, nt = n / 16) of the
// lower block triangle (kb <= nt / 2), lane ((pos % 32) / 8, n % 16),
// element pos % 8: the B operand of a 16x16x32 MFMA.
__device__ __forceinline__ int cfrag_off(int pos, int n) {
  const int nt = n >> 4;
  const int blk = ((nt + 1) * (nt + 1)) / 4 + (pos >> 5);
  return blk * kFrag + ((((pos & 31) >> 3) << 4) + (n & 15)) * 16 + (pos & 7) * 2;
}

// Conv-state slot s seen after the commit of a path of L nodes: old slot
// L + s while that is below 3, else the raw input of path node L - 3 + s.
template <typename TIn>
__device__ __forceinline__ float conv_slot(const CoefParams& p, const CoefMeta& s, int b, int L, int sl,
                                           int ch, const TIn* prev, size_t node_stride, int col) {
  const int C = 2 * p.Hk * p.DK + p.Hv * p.DV;
  if (L + sl < 3) return p.conv_state[(size_t(b) * 3 + L + sl) * C + ch];
  return to_f32(prev[(size_t(b) * p.T + s.ppath[L - 3 + sl]) * node_stride + col]);
}

// ---------------------------------------------------------------------------
// Staging of raw rows (node-major by canonical position) and the width-4
// conv + SiLU (+ L2 norm) of 8 channels per lane, 16 lanes per node.
// ---------------------------------------------------------------------------
constexpr int kSRow = kCD + 4;  // fp32 row stride of the staging tile (528 B)

// rows p < T of the staging tile <- raw src rows of the nodes at positions p,
// widened to fp32 (rows T .. T + 2 hold the conv-state slots)
template <typename TIn>
__device__ __forceinline__ void stage_rows(float* stage, const TIn* src, size_t node_stride, int ncols,
                                           const CoefMeta& s, int T, int tid) {
  constexpr int EPC = 16 / sizeof(TIn);
  const int cpr = ncols / EPC;
  for (int idx = tid; idx < T * cpr; idx += kCT) {
    const int r = idx / cpr, c = idx % cpr;
    const TIn* from = src + size_t(s.ord[r]) * node_stride + c * EPC;
    float* to = stage + r * kSRow + c * EPC;
    if constexpr (sizeof(TIn) == 2) {
      float x[8];
      load8(reinterpret_cast<const BF16*>(from), x);
      *reinterpret_cast<float4*>(to) = make_float4(x[0], x[1], x[2], x[3]);
      *reinterpret_cast<float4*>(to + 4) = make_float4(x[4], x[5], x[6], x[7]);
    } else {
      *reinterpret_cast<float4*>(to) = *reinterpret_cast<const float4*>(from);
    }
  }
}

// SiLU(conv) of channels 8 cg .. 8 cg + 7 of the node at position pos (taps
// from the staged rows); w = weights [channel][tap].  Channels >= ncols
// give 0.
__device__ __forceinline__ void conv8(const float* stage, const CoefMeta& s, int pos, int cg, int ncols,
                                      const float (&w)[8][4], float (&y)[8]) {
  const uint32_t taps = s.tap[pos];
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = 0.0f;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int row = (taps >> (8 * t)) & 255;
    float x[8];
    load8(stage + row * kSRow + 8 * cg, x);
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = fmaf(w[e][t], x[e], y[e]);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = 8 * cg + e < ncols ? silu(y[e]) : 0.0f;
}

__device__ __forceinline__ uint4 pack_h8(const float (&y)[8], float sc) {
  h8 h;
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (_Float16)(y[e] * sc);
  return __builtin_bit_cast(uint4, h);
}

// ---------------------------------------------------------------------------
// Coefficient recurrences of all nodes, one group of NL lanes per node.  The
// path slots rho = 0 (the node itself), 1 (its parent), ..., d (the root) are
// taken in order; lane q of a group holds the pending sums of the slots
// rho = rho0 + NL k + q (k < 8) of the current round rho0, as a shift
// register that moves down by one entry per round, so the slot being
// resolved is always entry 0 of lane rho % NL.  Writes D[t][i] = r c and
// C'[t][i] = -c into the fragment arrays (the decay a_i of C' is applied to
// the X~ product) and a_i into s.a.  s.gt[p] = (beta, alpha, G-row start).
// ---------------------------------------------------------------------------

// next path position: the node itself for slot 0, then the ancestors from the
// deepest up (highest set position bit first)
__device__ __forceinline__ int next_pos(int rho, int p, uint64_t& lo, uint64_t& hi) {
  if (rho == 0) return p;
  const bool useh = hi != 0;
  const int bit = 63 - __builtin_clzll((useh ? hi : lo) | 1ull);
  const uint64_t clr = ~(1ull << bit);
  hi = useh ? (hi & clr) : hi;
  lo = useh ? lo : (lo & clr);
  return useh ? 64 + bit : bit;
}

// 4 lanes per node (depth < 32).  The tables then have fixed rows of kDRow
// entries per position in reversed depth order: entry 31 - delta of row p
// holds the product with p's ancestor (or p itself) at depth delta, every
// other entry is zero.  The pending sum of slot rho2 of a node at depth d
// (ancestor depth d - rho2) is then entry 31 - d + rho2 of the row: a fixed
// offset from a per-round base for each of the lane's 8 slots, and slots
// already resolved (rho2 <= rho) or beyond the root (rho2 > d) read zeros, so
// the update needs no masking.  One LDS round trip per step.
constexpr int kDRow = 66;  // 64 entries + 2 of padding (rows 33 banks apart)
// K pending sums per lane: slots up to 4 K - 1, i.e. trees of depth < 4 K.
template <int K>
__device__ __forceinline__ void coef_recurrence4(CoefMeta& s, const _Float16* tabQ, const _Float16* tabG,
                                                 unsigned char* cfr, unsigned char* dfr, int nval, int tid) {
  constexpr int NL = 4;
  const int q = tid & 3;
  for (int base = 0; base < nval; base += kCT / NL) {
    const int p = base + tid / NL;
    const bool active = p < nval;
    const int d = active ? s.pdep[p] : -1;
    const int dmax = wave_max_i(d);
    float w[K];
    {
      const _Float16* row = tabQ + (active ? p : 0) * kDRow + 31 - (active ? d : 0) + q;
#pragma unroll
      for (int k = 0; k < K; ++k) w[k] = (float)row[4 * k];
    }
    uint64_t lo = active ? s.ancp[p][0] : 0, hi = active ? s.ancp[p][1] : 0;
    float r = 1.0f;
    for (int rho0 = 0; rho0 <= dmax; rho0 += NL) {
      // entry of slot rho0 + q in any row (clamped for lanes past their root,
      // whose reads are not used)
      int e0 = 31 - d + rho0 + q;
      e0 = e0 < 35 ? e0 : 35;
      static_for<NL>([&](auto jc) __attribute__((always_inline)) {
        constexpr int j = decltype(jc)::value;
        const int rho = rho0 + j;
        const bool act = active && rho <= d;
        const int pos = next_pos(rho, p, lo, hi);
        const int ps = act ? pos : 0;
        const float2 gba = *reinterpret_cast<const float2*>(&s.gt[ps]);
        const _Float16* row = tabG + ps * kDRow + e0;
        float gv[K];
#pragma unroll
        for (int k2 = 0; k2 < K; ++k2) gv[k2] = (float)row[4 * k2];
        const float c = gba.x * bcast<NL, j>(w[0]);
        if (act && q == j) {
          *reinterpret_cast<_Float16*>(dfr + cfrag_off(ps, p)) = (_Float16)(r * c);
          *reinterpret_cast<_Float16*>(cfr + cfrag_off(ps, p)) = (_Float16)(-c);
        }
        r *= act ? gba.y : 1.0f;
#pragma unroll
        for (int k2 = 0; k2 < K; ++k2) w[k2] = fmaf(-c, gv[k2], w[k2]);
        __builtin_amdgcn_sched_barrier(0);  // one step's loads live at a time
      });
#pragma unroll
      for (int k = 0; k < K - 1; ++k) w[k] = w[k + 1];
      w[K - 1] = 0.0f;
    }
    if (active && q == 0) s.a[p] = r;
  }
}

// 16 lanes per node (any depth up to 127): the general case, one step at a
// time with the pending sum broadcast through ds_bpermute.
__device__ __forceinline__ void coef_recurrence16(CoefMeta& s, const _Float16* tabQ, const _Float16* tabG,
                                                  unsigned char* cfr, unsigned char* dfr, int nval, int tid) {
  constexpr int NL = 16;
  const int q = tid & 15;
  for (int base = 0; base < nval; base += kCT / NL) {
    const int p = base + tid / NL;
    const bool active = p < nval;
    const int d = active ? s.pdep[p] : -1;
    const int dmax = wave_max_i(d);
    const int qo = active ? s.qoff[p] : 0;
    float w[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int rho = NL * k + q;
      w[k] = (active && rho <= d) ? (float)tabQ[qo + d - rho] : 0.0f;
    }
    uint64_t lo = active ? s.ancp[p][0] : 0, hi = active ? s.ancp[p][1] : 0;
    float r = 1.0f;
    const int gbase = (tid & 63) & ~(NL - 1);
    for (int rho0 = 0; rho0 <= dmax; rho0 += NL) {
      for (int j = 0; j < NL; ++j) {
        const int rho = rho0 + j;
        const bool act = active && rho <= d;
        const int pos = next_pos(rho, p, lo, hi);
        const int ps = act ? pos : 0;
        const float4 gt = s.gt[ps];
        const float c = gt.x * __shfl(w[0], gbase + j);
        if (act && q == j) {
          *reinterpret_cast<_Float16*>(dfr + cfrag_off(ps, p)) = (_Float16)(r * c);
          *reinterpret_cast<_Float16*>(cfr + cfrag_off(ps, p)) = (_Float16)(-c);
        }
        r *= act ? gt.y : 1.0f;
        const int go = __float_as_int(gt.z);
        float gv[8];
#pragma unroll
        for (int k2 = 0; k2 < 8; ++k2) {
          const int rho2 = rho0 + NL * k2 + q;
          const bool u = act && rho2 > rho && rho2 <= d;
          gv[k2] = (float)tabG[u ? go + d - rho2 : 0];
        }
#pragma unroll
        for (int k2 = 0; k2 < 8; ++k2) {
          const int rho2 = rho0 + NL * k2 + q;
          const bool u = act && rho2 > rho && rho2 <= d;
          w[k2] = fmaf(u ? -c : 0.0f, gv[k2], w[k2]);
        }
      }
#pragma unroll
      for (int k = 0; k < 7; ++k) w[k] = w[k + 1];
      w[7] = 0.0f;
    }
    if (active && q == 0) s.a[p] = r;
  }
}

// ---------------------------------------------------------------------------
// Path-key features of one commit chunk (path slots m0 .. m0 + cnt - 1): conv
// along the path (conv state before the commit above the root) + SiLU + L2
// norm -> s_kp (fp32 rows), then the chunk's Gram matrix -> s_gp (bf16x3
// MFMA on waves 0..3).  Ends with a barrier.
// ---------------------------------------------------------------------------
template <typename TIn>
__device__ __forceinline__ void kp_features(const CoefParams& p, const CoefMeta& s, float* s_kp, float* s_gp,
                                            int b, int g, int m0, int cnt, int tid) {
  const int T = p.T, Hk = p.Hk, DK = p.DK;
  const int C = 2 * Hk * DK + p.Hv * p.DV;
  const int kch0 = Hk * DK + g * DK;
  const int cg = tid & 15, j = tid >> 4;  // 8 channels of path slot m0 + j
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, lg = lane >> 4;
  const TIn* pk = static_cast<const TIn*>(p.pk);
  float x[4][8], wk[8][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int mm = m0 + j - 3 + t;
    if (j < cnt && mm >= 0 && 8 * cg < DK) {
      load8(pk + (size_t(b) * T + s.ppath[mm]) * Hk * DK + size_t(g) * DK + 8 * cg, x[t]);
    } else if (j < cnt && mm < 0 && 8 * cg < DK) {
      load8(p.conv_state + (size_t(b) * 3 + mm + 3) * C + kch0 + 8 * cg, x[t]);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[t][e] = 0.0f;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int c = 8 * cg + e;
    const float4 w4 = c < DK ? *reinterpret_cast<const float4*>(p.conv_w + size_t(kch0 + c) * 4)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
    wk[e][0] = w4.x;
    wk[e][1] = w4.y;
    wk[e][2] = w4.z;
    wk[e][3] = w4.w;
  }
  float y[8];
  float ss = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float v = fmaf(wk[e][3], x[3][e], fmaf(wk[e][2], x[2][e], fmaf(wk[e][1], x[1][e], wk[e][0] * x[0][e])));
    y[e] = (j < cnt && 8 * cg + e < DK) ? silu(v) : 0.0f;
    ss = fmaf(y[e], y[e], ss);
  }
  ss = group_sum<16>(ss);
  const float inv = rsqrt_hw(ss + 1e-6f);
  float* dst = s_kp + j * kKpRow + 8 * cg;
  *reinterpret_cast<float4*>(dst) = make_float4(y[0] * inv, y[1] * inv, y[2] * inv, y[3] * inv);
  *reinterpret_cast<float4*>(dst + 4) = make_float4(y[4] * inv, y[5] * inv, y[6] * inv, y[7] * inv);
  lds_sync();
  if (wave < 4) {  // path Gram Kp Kp^T (32 x 32)
    const int ti = wave >> 1, tj = wave & 1;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      float xa[8], xb[8];
      load8(s_kp + (16 * ti + l16) * kKpRow + 32 * kb + 8 * lg, xa);
      load8(s_kp + (16 * tj + l16) * kKpRow + 32 * kb + 8 * lg, xb);
      bf16x8 ah, al, bh, bl;
      split_rne8(xa, ah, al);
      split_rne8(xb, bh, bl);
      acc = mfma3(ah, al, bh, bl, acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) s_gp[(16 * ti + 4 * lg + i) * kGpRow + 16 * tj + l16] = acc[i];
  }
  lds_sync();
}

// Streaming load of 16 bytes (raw rows, read once): the non-temporal hint
// keeps them from displacing the state rows in the caches.
__device__ __forceinline__ uint4 load_stream16(const void* src) {
  typedef unsigned u32v4 __attribute__((ext_vector_type(4)));
  const u32v4 v = __builtin_nontemporal_load(reinterpret_cast<const u32v4*>(src));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// ---------------------------------------------------------------------------
// Inputs of one value head, loaded into registers one head ahead (the
// loads are issued before the previous head's outputs are stored, so that
// waiting for them does not wait for those stores) and written to LDS at
// the head's start.
// ---------------------------------------------------------------------------
template <typename TIn>
struct Raw4T;
template <>
struct Raw4T<BF16> {
  typedef uint2 type;
};
template <>
struct Raw4T<float> {
  typedef uint4 type;
};
__device__ __forceinline__ float4 raw4_f32(const uint2& u) {
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xffff0000u));
}
__device__ __forceinline__ float4 raw4_f32(const uint4& u) {
  return make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z), __uint_as_float(u.w));
}

template <typename TIn, int MODE>
struct HeadIn {
  static constexpr int EPC = 16 / sizeof(TIn);
  static constexpr int NVC = kCMaxT * kCD / EPC / kCT;  // 16-byte raw-v chunks per thread
  static constexpr bool kStep = MODE == kModeStep;
  typedef typename Raw4T<TIn>::type Raw4;
  uint4 raw[NVC];
  TIn al, be;   // gates of position tid
  float wv;     // v conv weight: tap tid / 128, channel tid % 128
  float cs;     // conv-state slot tid / 128, channel tid % 128 seen by this step
  float cso;    // the same slot before the commit (path features of the commit)
  TIn pal, pbe;  // gates of path slot tid
  Raw4 pt[2][4];  // raw path values: slot 16 u + l16, channels 16 wave + 4 lg .. + 3, tap t

  __device__ __forceinline__ void load(const CoefParams& p, const CoefMeta& s, int b, int h, int Lp, bool vok,
                                       int tid) {
    const int T = p.T, Hk = p.Hk, Hv = p.Hv, DK = p.DK, DV = p.DV;
    const int C = 2 * Hk * DK + Hv * DV;
    const int vch0 = 2 * Hk * DK + h * DV;
    const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, lg = lane >> 4;
    if (vok) {
      const TIn* src = static_cast<const TIn*>(p.v) + size_t(b) * T * Hv * DV + size_t(h) * DV;
      const int cpr = DV / EPC;
#pragma unroll
      for (int jj = 0; jj < NVC; ++jj) {
        const int idx = jj * kCT + tid;
        const int ok = idx < T * cpr;
        const int r = ok ? idx / cpr : 0, c = ok ? idx % cpr : 0;
        raw[jj] = load_stream16(src + size_t(s.ord[r]) * Hv * DV + c * EPC);
      }
      const size_t ai = (size_t(b) * T + s.ord[tid < T ? tid : 0]) * Hv + h;
      al = static_cast<const TIn*>(p.alpha)[ai];
      be = static_cast<const TIn*>(p.beta)[ai];
      {
        const int i = tid < 3 * kCD ? tid : 0;
        const int sl = i / kCD, c = i % kCD;
        cs = c < DV ? conv_slot<TIn>(p, s, b, kStep ? Lp : 0, sl, vch0 + c, static_cast<const TIn*>(p.pv),
                                     size_t(Hv) * DV, h * DV + c)
                    : 0.0f;
      }
    }
    if (vok || (MODE != kModeVerify && Lp > 0)) {  // v conv weights (verify and path values)
      const int c = tid % kCD, t = tid / kCD;
      wv = c < DV ? p.conv_w[size_t(vch0 + c) * 4 + t] : 0.0f;
    }
    if constexpr (MODE != kModeVerify) {
      if (Lp > 0) {
        const int i = tid < 3 * kCD ? tid : 0;
        const int sl = i / kCD, c = i % kCD;
        cso = c < DV ? p.conv_state[(size_t(b) * 3 + sl) * C + vch0 + c] : 0.0f;
        const size_t ai = (size_t(b) * T + s.ppath[tid < Lp ? tid : 0]) * Hv + h;
        pal = static_cast<const TIn*>(p.palpha)[ai];
        pbe = static_cast<const TIn*>(p.pbeta)[ai];
        const int cl = 16 * wave + 4 * lg;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int mm = 16 * u + l16 - 3 + t;
            const int node = s.ppath[(mm >= 0 && mm < Lp) ? mm : 0];
            pt[u][t] = *reinterpret_cast<const Raw4*>(static_cast<const TIn*>(p.pv) +
                                                      (size_t(b) * T + node) * Hv * DV + size_t(h) * DV +
                                                      (cl < DV ? cl : 0));
          }
      }
    }
  }

  __device__ __forceinline__ void store(const CoefParams& p, CoefMeta& s, float* stage, int Lp, bool vok,
                                        int tid) const {
    const int T = p.T, DV = p.DV;
    if (vok) {
      const int cpr = DV / EPC;
#pragma unroll
      for (int jj = 0; jj < NVC; ++jj) {
        const int idx = jj * kCT + tid;
        if (idx < T * cpr) {
          const int r = idx / cpr, c = idx % cpr;
          float* to = stage + r * kSRow + c * EPC;
          if constexpr (sizeof(TIn) == 2) {
            const uint4 u = raw[jj];
            *reinterpret_cast<float4*>(to) = raw4_f32(make_uint2(u.x, u.y));
            *reinterpret_cast<float4*>(to + 4) = raw4_f32(make_uint2(u.z, u.w));
          } else {
            *reinterpret_cast<uint4*>(to) = raw[jj];
          }
        }
      }
      if (tid < 3 * kCD) stage[(T + tid / kCD) * kSRow + tid % kCD] = cs;
      if (tid < T) {
        const int go = s.qoff[tid] - tid;
        s.gt[tid] = make_float4(to_f32(be), to_f32(al), __int_as_float(go), 0.0f);
      }
    }
    if (vok || (MODE != kModeVerify && Lp > 0)) s.wv[tid / kCD][tid % kCD] = wv;
    if constexpr (MODE != kModeVerify) {
      if (Lp > 0) {
        if (tid < 3 * kCD) s.cso[tid / kCD][tid % kCD] = cso;
        if (tid < Lp) {
          s.pal[tid] = to_f32(pal);
          s.pbe[tid] = to_f32(pbe);
        }
      }
    }
  }
};

// state rows of head h in the S^T accumulator layout (16 dk columns ...)
__device__ __forceinline__ void load_state(const float* S, int b, int Hv, int DV, int DK, int h, int wave, int l16,
                                           int lg, float (&sf)[8][4]) {
  const float* Sb = S + (size_t(b) * Hv + h) * size_t(DV) * DK;
  const int dv = 16 * wave + l16;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const int dk = 16 * t + 4 * lg;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (dv < DV && dk < DK) v = *reinterpret_cast<const float4*>(Sb + size_t(dv) * DK + dk);
    sf[t][0] = v.x;
    sf[t][1] = v.y;
    sf[t][2] = v.z;
    sf[t][3] = v.w;
  }
}

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
template <typename TIn, int MODE>
__global__ __launch_bounds__(kCT) void coef_kernel(CoefParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr bool kVerify = MODE != kModeCommit;
  constexpr bool kCommit = MODE != kModeVerify;
  constexpr int EPC = 16 / sizeof(TIn);
  constexpr int NVC = HeadIn<TIn, MODE>::NVC;
  CoefMeta& s = *reinterpret_cast<CoefMeta*>(smem);
  const int T = p.T, Hk = p.Hk, Hv = p.Hv, DK = p.DK, DV = p.DV;
  const CoefSmem L_ = coef_smem(T, MODE, sizeof(TIn));
  const int TR = L_.TR;
  _Float16* tabQ = reinterpret_cast<_Float16*>(smem + L_.tab);
  _Float16* tabG = tabQ;  // set once the tree's depth is known
  float* s_kp = reinterpret_cast<float*>(smem + L_.kp);  // [kPC][kKpRow] path keys
  float* s_gp = s_kp + kPC * kKpRow;                      // [kPC][kGpRow] path Gram
  float* s_ut0 = s_gp + kPC * kGpRow;                     // 8 x [kPC][16] U~ transposes
  unsigned char* big = smem + L_.big;
  float* stage = reinterpret_cast<float*>(big);

  const int G = Hv / Hk;
  const int nhg = G / p.hpw;
  const int b = blockIdx.y;
  const int g = blockIdx.x / nhg;
  const int h0 = g * G + (blockIdx.x % nhg) * p.hpw;
  const int C = 2 * Hk * DK + Hv * DV;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, lg = lane >> 4;
  const int NT = (T + 15) / 16;
  const int KBP = (T + 31) / 32;


  // ---- commit path (step / commit): the accepted node's path, root first
  int Lp = 0;
  if constexpr (kCommit) {
    const MetaPtrs pm = meta_ptrs(p.pmeta, p.B, T);
    const int acc = p.paccepted[b];
    const int pst = pm.status[b];
    int cst = pst;
    if (cst == GDN_TREE_OK && acc != -1) {
      if (acc < -1 || acc >= T || pm.depth[size_t(b) * T + acc] < 0) cst = GDN_TREE_BAD_ACCEPTED;
    }
    Lp = (cst == GDN_TREE_OK && acc >= 0) ? pm.depth[size_t(b) * T + acc] + 1 : 0;
    if (blockIdx.x == 0 && tid == 0 && p.commit_status) p.commit_status[b] = cst;
    if (Lp > 0 && tid < T) {
      const uint64_t word = pm.anc[(size_t(b) * T + acc) * pm.W + (tid >> 6)];
      if (tid == acc || ((word >> (tid & 63)) & 1ull)) s.ppath[pm.depth[size_t(b) * T + tid]] = tid;
    }
  }

  // ---- tree metadata of the verified tree
  int tstat = GDN_TREE_OK, nval = 0;
  if constexpr (kVerify) {
    const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
    tstat = m.status[b];
    nval = m.nvalid[b];
    if (tid < kCMaxT) {
      const bool in = tid < T;
      const size_t bi = size_t(b) * T + tid;
      s.ord[tid] = in ? m.order[bi] : 0;
      s.ppos[tid] = in ? m.ppos[bi] : -1;
      s.pdep[tid] = in ? m.pdep[bi] : -1;
      s.ancp[tid][0] = in ? m.ancp[bi * m.W] : 0;
      s.ancp[tid][1] = (in && m.W > 1) ? m.ancp[bi * m.W + 1] : 0;
    }
    if (tid <= T) s.qoff[tid] = m.qoff[size_t(b) * (T + 1) + tid];
  }
  lds_sync();
  if constexpr (kVerify) {
    if (tid >= T && tid < kCMaxT) s.tap[tid] = 0;  // positions past the tree read row 0
    if (tid < T) {  // staged rows of the 4 conv taps of position tid
      const int d = s.pdep[tid];
      const int t2 = s.ppos[tid];
      const int t1 = t2 >= 0 ? s.ppos[t2] : -1;
      const int t0 = t1 >= 0 ? s.ppos[t1] : -1;
      const int tp[4] = {t0, t1, t2, tid};
      uint32_t taps = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int row = d < 0 ? 0 : (d - 3 + w >= 0 ? tp[w] : T + d + w);
        taps |= uint32_t(row) << (8 * w);
      }
      s.tap[tid] = taps;
    }
  }
  const bool vok = kVerify && tstat == GDN_TREE_OK;
  // trees of depth < 32: fixed-row tables and 4 lanes per node in the
  // recurrence; deeper trees: ragged rows (offsets qoff) and 16 lanes
  const bool shallow = (nval > 0 ? s.pdep[nval - 1] : 0) < 32;
  tabG = tabQ + (shallow ? T * kDRow : (T * (T + 1)) / 2);


  // ---- per key head: Q~, K~, Gram tables, K~^T operand and Q~ init
  h8 kta[4];   // A operand of X~^T: K~^T rows 16 wave + l16, positions 32 kb + 8 lg ..
  h4 qin[8];   // Q~[16 nt + l16][16 wave + 4 lg + i]
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) kta[kb] = h8{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) qin[nt] = h4{0, 0, 0, 0};
  if (vok) {
    const TIn* pqs = static_cast<const TIn*>(p.pq);
    const TIn* pks = static_cast<const TIn*>(p.pk);
    const int cg = tid & 15, nj = tid >> 4;
    const int cpr = DK / EPC;
    // raw q and k rows and the conv-state rows of both, issued together
    uint4 rq[2][NVC];
    float csq[2];
#pragma unroll
    for (int part = 0; part < 2; ++part) {
      const TIn* src = static_cast<const TIn*>(part ? p.k : p.q) + size_t(b) * T * Hk * DK + size_t(g) * DK;
#pragma unroll
      for (int jj = 0; jj < NVC; ++jj) {
        const int idx = jj * kCT + tid;
        const int ok = idx < T * cpr;
        const int r = ok ? idx / cpr : 0, c = ok ? idx % cpr : 0;
        rq[part][jj] = load_stream16(src + size_t(s.ord[r]) * Hk * DK + c * EPC);
      }
      const int i = tid < 3 * kCD ? tid : 0;
      const int sl = i / kCD, c = i % kCD;
      csq[part] = c < DK ? conv_slot<TIn>(p, s, b, MODE == kModeStep ? Lp : 0, sl, part * Hk * DK + g * DK + c,
                                          part ? pks : pqs, size_t(Hk) * DK, g * DK + c)
                         : 0.0f;
    }
    uint4 qk_out[2][4];
#pragma unroll
    for (int part = 0; part < 2; ++part) {
      const int ch0 = part * Hk * DK + g * DK;
      if (part) lds_sync();  // q staging consumed
#pragma unroll
      for (int jj = 0; jj < NVC; ++jj) {
        const int idx = jj * kCT + tid;
        if (idx < T * cpr) {
          const int r = idx / cpr, c = idx % cpr;
          float* to = stage + r * kSRow + c * EPC;
          if constexpr (sizeof(TIn) == 2) {
            const uint4 u = rq[part][jj];
            *reinterpret_cast<float4*>(to) = raw4_f32(make_uint2(u.x, u.y));
            *reinterpret_cast<float4*>(to + 4) = raw4_f32(make_uint2(u.z, u.w));
          } else {
            *reinterpret_cast<uint4*>(to) = rq[part][jj];
          }
        }
      }
      if (tid < 3 * kCD) stage[(T + tid / kCD) * kSRow + tid % kCD] = csq[part];
      float wq[8][4];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int c = 8 * cg + e;
        const float4 w4 = c < DK ? *reinterpret_cast<const float4*>(p.conv_w + size_t(ch0 + c) * 4)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
        wq[e][0] = w4.x;
        wq[e][1] = w4.y;
        wq[e][2] = w4.z;
        wq[e][3] = w4.w;
      }
      lds_sync();
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int pos = 32 * r + nj;
        float y[8];
        if (pos < nval) {
          conv8(stage, s, pos, cg, DK, wq, y);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) y[e] = 0.0f;
        }
        float ss = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) ss = fmaf(y[e], y[e], ss);
        ss = group_sum<16>(ss);
        qk_out[part][r] = pack_h8(y, rsqrt_hw(ss + 1e-6f));
      }
    }
    if (shallow) {  // the fixed-row tables are zero outside the entries written below
      const int n16 = (2 * T * kDRow * 2 + 15) / 16;
      for (int i = tid; i < n16; i += kCT) reinterpret_cast<uint4*>(tabQ)[i] = make_uint4(0, 0, 0, 0);
    }
    lds_sync();  // staging consumed: Q~, K~ rows go to the same region
    _Float16* s_q = reinterpret_cast<_Float16*>(big);
    _Float16* s_k = s_q + TR * kQRow;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int pos = 32 * r + nj;
      if (pos < TR) {
        *reinterpret_cast<uint4*>(s_q + pos * kQRow + 8 * cg) = qk_out[0][r];
        *reinterpret_cast<uint4*>(s_k + pos * kQRow + 8 * cg) = qk_out[1][r];
      }
    }
    lds_sync();
    // Gram tiles (pt, pt2), pt2 <= pt: Q K^T (ancestors and self) and K K^T
    // (proper ancestors) scattered into the ragged tables
    const int ntile = NT * (NT + 1) / 2;
    for (int t = wave; t < ntile; t += 8) {
      int pt = 0;
      while ((pt + 1) * (pt + 2) / 2 <= t) ++pt;
      const int pt2 = t - pt * (pt + 1) / 2;
      f32x4 aq = {0.f, 0.f, 0.f, 0.f}, ag = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const h8 a1 = *reinterpret_cast<const h8*>(s_q + (16 * pt + l16) * kQRow + 32 * kb + 8 * lg);
        const h8 a2 = *reinterpret_cast<const h8*>(s_k + (16 * pt + l16) * kQRow + 32 * kb + 8 * lg);
        const h8 bk = *reinterpret_cast<const h8*>(s_k + (16 * pt2 + l16) * kQRow + 32 * kb + 8 * lg);
        aq = mma16(a1, bk, aq);
        ag = mma16(a2, bk, ag);
      }
      const int pc = 16 * pt2 + l16;
      const int dc = s.pdep[pc];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int pr = 16 * pt + 4 * lg + i;
        if (pr < nval && pc <= pr) {
          const bool anc = (s.ancp[pr][pc >> 6] >> (pc & 63)) & 1ull;
          // shallow trees: reversed fixed rows; deep trees: ragged rows
          const int iq = shallow ? pr * kDRow + 31 - dc : s.qoff[pr] + dc;
          const int ig = shallow ? pr * kDRow + 31 - dc : s.qoff[pr] - pr + dc;
          if (anc || pc == pr) tabQ[iq] = (_Float16)aq[i];
          if (anc) tabG[ig] = (_Float16)ag[i];
        }
      }
    }
    // operands kept in registers for all value heads of the key head
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if (kb < KBP) {
        h8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = s_k[(32 * kb + 8 * lg + e) * kQRow + 16 * wave + l16];
        kta[kb] = v;
      }
    }
#pragma unroll
    for (int nt = 0; nt < 8; ++nt)
      if (nt < NT) qin[nt] = *reinterpret_cast<const h4*>(s_q + (16 * nt + l16) * kQRow + 16 * wave + 4 * lg);
    lds_sync();  // Q~ / K~ tiles consumed
  }

  // inputs and state of the first value head
  HeadIn<TIn, MODE> hin;
  hin.load(p, s, b, h0, Lp, vok, tid);
  float sf[8][4];
  load_state(kCommit ? p.S : p.S0, b, Hv, DV, DK, h0, wave, l16, lg, sf);

  // ---- commit: path-key features of the first chunk (shared by the heads)
  const int nchunks = (Lp + kPC - 1) / kPC;
  if constexpr (kCommit) {
    if (Lp > 0) kp_features<TIn>(p, s, s_kp, s_gp, b, g, 0, Lp < kPC ? Lp : kPC, tid);
  }

  // ---- value heads
  for (int hh = 0; hh < p.hpw; ++hh) {
    const int h = h0 + hh;
    const bool more = hh + 1 < p.hpw;
    // per-lane indices re-derived inside the loop (see opaque_i)
    const int tid = opaque_i(threadIdx.x), lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    // this head's inputs -> LDS (staged raw v + conv rows, gates, weights)
    hin.store(p, s, stage, Lp, vok, tid);
    lds_sync();

    // ---- commit of the previous accepted path into sf (step / commit)
    if constexpr (kCommit) {
      if (Lp > 0) {
        for (int ch = 0; ch < nchunks; ++ch) {
          const int tid = opaque_i(threadIdx.x), lane = tid & 63, wave = tid >> 6;
          const int l16 = lane & 15, lg = lane >> 4;
          float* s_ut = s_ut0 + wave * (kPC * 16);  // this wave's U~^T scratch [slot][16]
          const int cl = 16 * wave + 4 * lg;        // value channels of this lane's rows
          const int m0 = ch * kPC;
          const int cnt = Lp - m0 < kPC ? Lp - m0 : kPC;
          if (ch > 0) kp_features<TIn>(p, s, s_kp, s_gp, b, g, m0, cnt, tid);
          // path values of the chunk in the P accumulator layout: slot
          // 16 u + l16, channels cl .. cl + 3 (conv along the path + SiLU)
          float vp[2][4];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            float4 x[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int mm = m0 + 16 * u + l16 - 3 + t;
              if (mm >= 0) {
                if (ch == 0) {
                  x[t] = raw4_f32(hin.pt[u][t]);
                } else {
                  const int node = s.ppath[mm < Lp ? mm : 0];
                  x[t] = raw4_f32(*reinterpret_cast<const typename Raw4T<TIn>::type*>(
                      static_cast<const TIn*>(p.pv) + (size_t(b) * T + node) * Hv * DV + size_t(h) * DV +
                      (cl < DV ? cl : 0)));
                }
              } else {
                x[t] = *reinterpret_cast<const float4*>(&s.cso[mm + 3][cl]);
              }
            }
            const bool okv = m0 + 16 * u + l16 < Lp && cl < DV;
            const float* xs = reinterpret_cast<const float*>(x);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float y = fmaf(s.wv[3][cl + i], xs[12 + i],
                                   fmaf(s.wv[2][cl + i], xs[8 + i],
                                        fmaf(s.wv[1][cl + i], xs[4 + i], s.wv[0][cl + i] * xs[i])));
              vp[u][i] = okv ? silu(y) : 0.0f;
            }
          }
          if (tid < kPC) {  // alpha products after slot m0 + tid within the chunk
            float sp = 1.0f;
            for (int m = tid + 1; m < cnt; ++m) sp *= s.pal[m0 + m];
            s.psuf[m0 + tid] = tid < cnt ? sp : 0.0f;
          }
          lds_sync();
          float Ac = 1.0f;  // alpha product over the chunk
          for (int m = 0; m < cnt; ++m) Ac *= s.pal[m0 + m];
          // P = S Kp^T (rows cl + i, path slot 16 u + l16)
          f32x4 P[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) {
            const float xa[8] = {sf[2 * kb][0],     sf[2 * kb][1],     sf[2 * kb][2],     sf[2 * kb][3],
                                 sf[2 * kb + 1][0], sf[2 * kb + 1][1], sf[2 * kb + 1][2], sf[2 * kb + 1][3]};
            bf16x8 ah, al;
            split_rne8(xa, ah, al);
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const float* kr = s_kp + (16 * u + l16) * kKpRow + 32 * kb + 4 * lg;
              const float4 k0 = *reinterpret_cast<const float4*>(kr);
              const float4 k1 = *reinterpret_cast<const float4*>(kr + 16);
              const float xb[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
              bf16x8 bh, bl;
              split_rne8(xb, bh, bl);
              P[u] = mfma3(ah, al, bh, bl, P[u]);
            }
          }
          // recurrence over the chunk's path nodes: u_j = beta_j (v_j - alpha_j T_j),
          // T_m <- alpha_j T_m + u_j (k_j . k_m) for the later slots m; T_j and v_j
          // of this lane group's rows are in lane j of tile j / 16 (row broadcast)
          f32x4 U[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
          static_for<2>([&](auto utc) __attribute__((always_inline)) {
            constexpr int ut = decltype(utc)::value;
            if (16 * ut >= cnt) return;
            static_for<16>([&](auto jc) __attribute__((always_inline)) {
              constexpr int j = decltype(jc)::value;
              const int jj = 16 * ut + j;
              if (jj >= cnt) return;
              const float aj = s.pal[m0 + jj], bj = s.pbe[m0 + jj];
              float uj[4];
#pragma unroll
              for (int i = 0; i < 4; ++i)
                uj[i] = bj * (bcast<16, j>(vp[ut][i]) - aj * bcast<16, j>(P[ut][i]));
              const bool own = l16 == j;
#pragma unroll
              for (int i = 0; i < 4; ++i) U[ut][i] = own ? uj[i] : U[ut][i];
              static_for<2>([&](auto uc) __attribute__((always_inline)) {
                constexpr int u = decltype(uc)::value;
                if constexpr (u >= ut) {
                  const float gg = s_gp[jj * kGpRow + 16 * u + l16];
#pragma unroll
                  for (int i = 0; i < 4; ++i) P[u][i] = fmaf(aj, P[u][i], uj[i] * gg);
                }
              });
              __builtin_amdgcn_sched_barrier(0);  // one step's loads at a time
            });
          });
          // u~_m = u_m times the alpha product of the later slots of the chunk;
          // U~^T through this wave's scratch: row slot, 16 value rows
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const float f = s.psuf[m0 + 16 * u + l16];
            *reinterpret_cast<float4*>(s_ut + (16 * u + l16) * 16 + 4 * lg) =
                make_float4(U[u][0] * f, U[u][1] * f, U[u][2] * f, U[u][3] * f);
          }
          wave_lds_sync();
          bf16x8 bh, bl;
          {
            float xb[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) xb[e] = s_ut[(8 * lg + e) * 16 + l16];
            split_rne8(xb, bh, bl);
          }
          // S^T <- Ac S^T + Kp^T U~^T
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            float xa[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) xa[e] = s_kp[(8 * lg + e) * kKpRow + 16 * t + l16];
            bf16x8 ah, al;
            split_rne8(xa, ah, al);
            f32x4 acc = {Ac * sf[t][0], Ac * sf[t][1], Ac * sf[t][2], Ac * sf[t][3]};
            acc = mfma3(ah, al, bh, bl, acc);
            sf[t][0] = acc[0];
            sf[t][1] = acc[1];
            sf[t][2] = acc[2];
            sf[t][3] = acc[3];
            __builtin_amdgcn_sched_barrier(0);
          }
          if (nchunks > 1) lds_sync();  // chunk features consumed before the next chunk's
        }
        // the committed state
        float* Sb = p.S + (size_t(b) * Hv + h) * size_t(DV) * DK;
        const int dv = 16 * wave + l16;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int dk = 16 * t + 4 * lg;
          if (dv < DV && dk < DK)
            *reinterpret_cast<float4*>(Sb + size_t(dv) * DK + dk) = make_float4(sf[t][0], sf[t][1], sf[t][2], sf[t][3]);
        }
      }
    }

    if (!vok) {
      if constexpr (kVerify) {  // invalid tree: zero outputs for this head
        for (int i = tid; i < T * DV / 4; i += kCT) {
          const int node = i / (DV / 4), c4 = i % (DV / 4);
          *reinterpret_cast<float4*>(p.out + (size_t(b) * T + node) * size_t(Hv) * DV + size_t(h) * DV + 4 * c4) =
              make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      if (more) {
        lds_sync();  // this head's path tables consumed
        hin.load(p, s, b, h + 1, Lp, vok, tid);
        load_state(kCommit ? p.S : p.S0, b, Hv, DV, DK, h + 1, wave, l16, lg, sf);
      }
      continue;
    }

    // ---- v conv in the MFMA operand layout: channel 16 wave + l16,
    //      positions 32 kb + 8 lg + e; fp16 with a power-of-two scale per channel
    h8 va[4];
    {
      const int c = 16 * wave + l16;
      const float w0 = s.wv[0][c], w1 = s.wv[1][c], w2 = s.wv[2][c], w3 = s.wv[3][c];
      float vt[4][8];
      float mx = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if (kb < KBP) {
          // the taps of 8 consecutive positions, then all 32 staged values
          const uint4 ta = *reinterpret_cast<const uint4*>(&s.tap[32 * kb + 8 * lg]);
          const uint4 tb = *reinterpret_cast<const uint4*>(&s.tap[32 * kb + 8 * lg + 4]);
          const uint32_t taps[8] = {ta.x, ta.y, ta.z, ta.w, tb.x, tb.y, tb.z, tb.w};
          float x[8][4];
#pragma unroll
          for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int t = 0; t < 4; ++t) x[e][t] = stage[((taps[e] >> (8 * t)) & 255) * kSRow + c];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int pos = 32 * kb + 8 * lg + e;
            const float y = silu(fmaf(w3, x[e][3], fmaf(w2, x[e][2], fmaf(w1, x[e][1], w0 * x[e][0]))));
            vt[kb][e] = (pos < nval && c < DV) ? y : 0.0f;
            mx = fmaxf(mx, fabsf(vt[kb][e]));
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) vt[kb][e] = 0.0f;
        }
      }
      mx = hmax4(mx);
      float sc, inv;
      pow2_scale(mx, sc, inv);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 8; ++e) va[kb][e] = (_Float16)(vt[kb][e] * sc);
      if (lg == 0) s.rsv[c] = inv;
    }
    lds_sync();  // staging consumed

    // ---- state rows -> fp16 operand with a power-of-two scale per row
    h8 sa[4];
    {
      float mx = 0.0f;
#pragma unroll
      for (int t = 0; t < 8; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = fmaxf(mx, fabsf(sf[t][i]));
      mx = hmax4(mx);
      float sc, inv;
      pow2_scale(mx, sc, inv);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sa[kb][i] = (_Float16)(sf[2 * kb][i] * sc);
          sa[kb][4 + i] = (_Float16)(sf[2 * kb + 1][i] * sc);
        }
      if (lg == 0) s.rs[16 * wave + l16] = inv;
    }

    // ---- coefficient recurrences -> C', D fragment arrays
    unsigned char* cfr = big;
    unsigned char* dfr = big + coef_nfrag(NT) * kFrag;
    unsigned char* xfr = big + 2 * coef_nfrag(NT) * kFrag;  // X~^T operand tiles [kb][nt]
    for (int i = tid; i < 2 * coef_nfrag(NT) * (kFrag / 16); i += kCT)
      reinterpret_cast<uint4*>(cfr)[i] = make_uint4(0, 0, 0, 0);
    if (tid < kCMaxT) s.a[tid] = 0.0f;
    lds_sync();
    // the next head's inputs and state load during the recurrence (LDS and
    // VALU bound, the memory pipe is otherwise idle), ahead of this head's
    // output stores
    if (more) {
      hin.load(p, s, b, h + 1, Lp, vok, tid);
      load_state(kCommit ? p.S : p.S0, b, Hv, DV, DK, h + 1, wave, l16, lg, sf);
    }
    {
      const int dmax = nval > 0 ? s.pdep[nval - 1] : 0;
      if (dmax < 12)
        coef_recurrence4<3>(s, tabQ, tabG, cfr, dfr, nval, tid);
      else if (dmax < 20)
        coef_recurrence4<5>(s, tabQ, tabG, cfr, dfr, nval, tid);
      else if (shallow)
        coef_recurrence4<8>(s, tabQ, tabG, cfr, dfr, nval, tid);
      else
        coef_recurrence16(s, tabQ, tabG, cfr, dfr, nval, tid);
    }
    lds_sync();

    // ---- X~^T = a (Q~^T - K~^T C^T)  (rows: key channels of this wave)
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) {
      if (nt >= NT) break;
      const float an = s.a[16 * nt + l16];
      f32x4 acc = {(float)qin[nt][0], (float)qin[nt][1], (float)qin[nt][2], (float)qin[nt][3]};
      const int base = coef_nfrag(nt);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        if (kb > nt / 2) break;
        const h8 bf = *reinterpret_cast<const h8*>(cfr + (base + kb) * kFrag + lane * 16);
        acc = mma16(kta[kb], bf, acc);
      }
      h4 hx;
#pragma unroll
      for (int i = 0; i < 4; ++i) hx[i] = (_Float16)(an * acc[i]);
      *reinterpret_cast<h4*>(xfr + ((wave >> 1) * NT + nt) * kFrag + lane * 16 + (wave & 1) * 8) = hx;
    }
    lds_sync();

    // ---- O^T = S X~^T + V~^T D^T  (rows: value channels of this wave)
    {
      const float4 is4 = *reinterpret_cast<const float4*>(&s.rs[16 * wave + 4 * lg]);
      const float4 iv4 = *reinterpret_cast<const float4*>(&s.rsv[16 * wave + 4 * lg]);
      const int dvr = 16 * wave + 4 * lg;
#pragma unroll
      for (int nt = 0; nt < 8; ++nt) {
        if (nt >= NT) break;
        f32x4 accs = {0.f, 0.f, 0.f, 0.f}, accv = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          const h8 bx = *reinterpret_cast<const h8*>(xfr + (kb * NT + nt) * kFrag + lane * 16);
          accs = mma16(sa[kb], bx, accs);
        }
        const int base = coef_nfrag(nt);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          if (kb > nt / 2) break;
          const h8 bd = *reinterpret_cast<const h8*>(dfr + (base + kb) * kFrag + lane * 16);
          accv = mma16(va[kb], bd, accv);
        }
        const int pp = 16 * nt + l16;
        if (pp < T && dvr < DV) {
          const int node = s.ord[pp];
          float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
          if (pp < nval)
            o = make_float4(p.scale * fmaf(accs[0], is4.x, accv[0] * iv4.x),
                            p.scale * fmaf(accs[1], is4.y, accv[1] * iv4.y),
                            p.scale * fmaf(accs[2], is4.z, accv[2] * iv4.z),
                            p.scale * fmaf(accs[3], is4.w, accv[3] * iv4.w));
          *reinterpret_cast<float4*>(p.out + (size_t(b) * T + node) * size_t(Hv) * DV + size_t(h) * DV + dvr) = o;
        }
      }
    }
    lds_sync();  // fragment tiles consumed before the next head
  }

  // ---- fused step: conv state after the commit for this workgroup's channels
  if constexpr (MODE == kModeStep) {
    const float* cs = p.conv_state + size_t(b) * 3 * C;
    float* co = p.conv_state_out + size_t(b) * 3 * C;
    if (blockIdx.x % nhg == 0) {
      for (int i = tid; i < 3 * 2 * DK; i += kCT) {
        const int sl = i / (2 * DK), part = (i / DK) & 1, c = i % DK;
        const int ch = part * Hk * DK + g * DK + c;
        const TIn* src = static_cast<const TIn*>(part ? p.pk : p.pq);
        co[size_t(sl) * C + ch] = Lp + sl < 3 ? cs[size_t(Lp + sl) * C + ch]
                                              : to_f32(src[(size_t(b) * T + s.ppath[Lp - 3 + sl]) * Hk * DK +
                                                           size_t(g) * DK + c]);
      }
    }
    const int nv = p.hpw * DV;
    for (int i = tid; i < 3 * nv; i += kCT) {
      const int sl = i / nv, j = i % nv;
      const int col = h0 * DV + j;
      const int ch = 2 * Hk * DK + col;
      co[size_t(sl) * C + ch] = Lp + sl < 3 ? cs[size_t(Lp + sl) * C + ch]
                                            : to_f32(static_cast<const TIn*>(p.pv)[(size_t(b) * T + s.ppath[Lp - 3 + sl]) *
                                                                                    Hv * DV + col]);
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename TIn, int MODE>
static int launch_coef_t(const CoefParams& p, hipStream_t stream) {
  const size_t smem = coef_smem(p.T, MODE, sizeof(TIn)).total;
  static bool attr_done = false;
  if (!attr_done) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&coef_kernel<TIn, MODE>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(coef_smem(kCMaxT, MODE, sizeof(TIn)).total));
    if (e != hipSuccess) return set_error(GDN_EHIP, "LDS attribute: %s", hipGetErrorString(e));
    attr_done = true;
  }
  const int G = p.Hv / p.Hk;
  hipLaunchKernelGGL((coef_kernel<TIn, MODE>), dim3(p.Hk * (G / p.hpw), p.B), dim3(kCT), smem, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

template <int MODE>
static int launch_coef_mode(const CoefParams& p, int in_dtype, hipStream_t stream) {
  if (in_dtype == GDN_BF16) return launch_coef_t<BF16, MODE>(p, stream);
  return launch_coef_t<float, MODE>(p, stream);
}

static CoefParams coef_params(const VerifyArgs& a) {
  CoefParams p;
  p.B = a.B;
  p.T = a.T;
  p.Hk = a.Hk;
  p.Hv = a.Hv;
  p.DK = a.dk;
  p.DV = a.dv;
  const int G = a.Hv / a.Hk;
  // one value head per workgroup when the grouped grid would leave CUs idle
  p.hpw = a.B * a.Hk >= 256 ? G : 1;
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
  p.pmeta = a.pmeta;
  p.paccepted = a.paccepted;
  p.pq = a.pq;
  p.pk = a.pk;
  p.pv = a.pv;
  p.palpha = a.palpha;
  p.pbeta = a.pbeta;
  p.conv_state_out = a.conv_state_out;
  p.S = a.S;
  p.commit_status = a.commit_status;
  return p;
}

int launch_coef_verify(const VerifyArgs& a, hipStream_t stream) {
  if (a.T > kCMaxT) return set_error(GDN_EUNSUPPORTED, "verify: T=%d exceeds %d", a.T, kCMaxT);
  const CoefParams p = coef_params(a);
  if (a.fused) return launch_coef_mode<kModeStep>(p, a.in_dtype, stream);
  return launch_coef_mode<kModeVerify>(p, a.in_dtype, stream);
}

// commit only: the state kernel in commit mode (the conv-state shift runs
// after it, see launch_commit)
int launch_coef_commit(const CommitArgs& a, hipStream_t stream) {
  if (a.T > kCMaxT) return set_error(GDN_EUNSUPPORTED, "commit: T=%d exceeds %d", a.T, kCMaxT);
  CoefParams p = {};
  p.B = a.B;
  p.T = a.T;
  p.Hk = a.Hk;
  p.Hv = a.Hv;
  p.DK = a.dk;
  p.DV = a.dv;
  const int G = a.Hv / a.Hk;
  p.hpw = a.B * a.Hk >= 256 ? G : 1;
  p.conv_w = a.conv_w;
  p.conv_state = a.conv_state;
  p.pmeta = a.meta;
  p.paccepted = a.accepted;
  p.pq = a.q;
  p.pk = a.k;
  p.pv = a.v;
  p.palpha = a.alpha;
  p.pbeta = a.beta;
  p.S = a.S;
  p.commit_status = a.commit_status;
  return launch_coef_mode<kModeCommit>(p, a.in_dtype, stream);
}

}  // namespace gdn
