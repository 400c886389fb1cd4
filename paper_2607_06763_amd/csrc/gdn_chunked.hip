// gdn_chunked.hip -- tree verification in the paper's chunked form
// (Sec. 3.4.1-3.4.2, Eq. 9-13), for trees of up to 512 slots.
//
// With positions in canonical (topological) order, a_i the product of alpha
// over the path root..i, and q~, k~, v~ the post-conv features of one
// (sequence, value head), Eq. 7-8 give for every node, in the stored
// orientation (S0 in R^{dv x dk}):
//     X_ij = [j strict ancestor of i] beta_i (a_i / a_j) k~_i.k~_j      (Eq. 9)
//     Y_ij = [j ancestor of i or i]  (a_i / a_j) q~_i.k~_j
//     (I + X) U = beta (V - a K S0^T)           (Eq. 10 with W S0 folded in)
//     O = scale (a Q S0^T + Y U)                 (Eq. 11)
// X is strictly lower triangular (ancestors come first), so U follows from a
// forward substitution over sub-blocks of B_c = 32 positions (Eq. 13):
//     U_j = (I + X_jj)^-1 (R_j - sum_{c<j} X_jc U_c),
// where the inverse of each unit lower-triangular diagonal block is the
// product (I - N)(I + N^2)(I + N^4)(I + N^8)(I + N^16), N = X_jj (N^32 = 0),
// formed by repeated squaring.
//
// The features come from the feature kernel (gdn_large.hip) in a workspace
// F[B][T][C]; U[B][Hv][T][dv] is a second workspace.  One workgroup per
// (value head, sequence), 512 threads = 8 waves; products are 16 x 16 MFMA
// tiles with operands in LDS.  The large ones (the S0 products, the Gram
// blocks and the block updates) take both operands as bf16 hi/lo planes and
// three v_mfma_f32_16x16x32_bf16 (hi*hi + hi*lo + lo*hi, fp32 accumulation,
// ~1e-5 relative); the diagonal-block inverse and its two products stay on
// v_mfma_f32_16x16x4f32 (fp32 operands):
//   phase A  S0 staged once; for each block: a Q S0^T -> out (node order),
//            beta (V - a K S0^T) -> U (padding rows zero)
//   phase B  for each block j in order: R_j, O_j in registers; for every
//            earlier block c holding an ancestor of a node of j: the decayed,
//            masked Gram blocks X_jc, Y_jc, then R_j -= X_jc U_c and
//            O_j += Y_jc U_c; the diagonal block: X_jj, Y_jj, the inverse by
//            five rounds of squaring (the powers of A = -N on waves 0-3, the
//            partial products on waves 4-7), U_j = (I + X_jj)^-1 R_j -> U,
//            O_j += Y_jj U_j, scaled and stored.
#include <math.h>

#include "gdn_internal.h"

namespace gdn {

constexpr int kHT = 512;      // threads per workgroup (8 waves)
constexpr int kBc = 32;       // positions per sub-block (B_c)
constexpr int kHMaxT = 512;   // tree slots supported
constexpr int kHW = 8;        // ancestor words per node (512 / 64)
constexpr int kLs = 36;       // row stride of the 32 x 32 matrices (floats)

struct ChunkParams {
  int B, T, Hk, Hv;
  float scale;
  const void* meta;
  const void *alpha, *beta;
  const float* S0;
  float* out;
  const float* F;  // features [B][T][C]
  float* U;        // [B][Hv][T][DV]: right-hand sides, then the solved rows
};

template <int DK, int DV>
struct ChunkSmem {
  static constexpr int KP = DK < 32 ? 32 : DK;  // contraction extent of the key products (zero padded)
  static constexpr int LKH = KP + 8;            // bf16 plane row (halves)
  static constexpr int LV = DV + 4;             // fp32 row of a 32 x DV block
  static constexpr int UL = kBc + 8;            // bf16 row of a 32-column plane (X, Y, transposed U)
  static constexpr size_t pk = size_t(kBc) * LKH * 2;  // one 32-row key plane
  static constexpr size_t head = 4 * pk;               // block q and k planes (hi, lo)
  static constexpr size_t uni_a = size_t(2) * DV * LKH * 2;  // phase A: S0 planes
  static constexpr size_t uni_b = 2 * pk                     // keys of block c
                                  + size_t(2) * DV * UL * 2  // U of block c, transposed
                                  + size_t(4) * kBc * UL * 2  // -X and Y blocks
                                  + size_t(5) * kBc * kLs * 4  // Y_jj, powers, partial products
                                  + size_t(2) * kBc * LV * 4;  // R_j, U_j
  static constexpr size_t uni = uni_a > uni_b ? uni_a : uni_b;
  static constexpr size_t anc = size_t(kBc) * kHW * 8;
  static constexpr size_t meta = size_t(kHMaxT) * (2 + 2 + 4 + 4 + 4);
  static constexpr size_t total = head + uni + anc + meta;
};

size_t chunked_workspace_bytes(int B, int T, int Hk, int Hv, int dk, int dv) {
  return features_f32_bytes(B, T, Hk, Hv, dk, dv) + size_t(B) * Hv * size_t(T) * dv * sizeof(float);
}

// acc += A (16 x K) B (K x 16) for one 16 x 16 tile on v_mfma_f32_16x16x4f32.
// A[i][k] = a[i * lda + k]; B[k][j] = b[j * ldb + k] (BT) or b[k * ldb + j].
// Result layout: acc[r] = D[4 (lane / 16) + r][lane % 16].
template <int K, bool BT>
__device__ __forceinline__ f32x4 mm16(const float* a, int lda, const float* b, int ldb, f32x4 acc, int lane) {
  const int i = lane & 15, kk = lane >> 4;
#pragma unroll 8
  for (int k0 = 0; k0 < K; k0 += 4) {
    const float av = a[i * lda + k0 + kk];
    const float bv = BT ? b[i * ldb + k0 + kk] : b[(k0 + kk) * ldb + i];
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
  }
  return acc;
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// 16 x 16 tile of a 32 x 32 matrix in LDS as an accumulator
__device__ __forceinline__ f32x4 ld_tile(const float* m, int ti, int tj, int lane) {
  f32x4 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = m[(16 * ti + 4 * (lane >> 4) + r) * kLs + 16 * tj + (lane & 15)];
  return v;
}
__device__ __forceinline__ void st_tile(float* m, int ti, int tj, int lane, f32x4 v) {
#pragma unroll
  for (int r = 0; r < 4; ++r) m[(16 * ti + 4 * (lane >> 4) + r) * kLs + 16 * tj + (lane & 15)] = v[r];
}

// x -> bf16 hi (truncation) + bf16 lo (truncation of the remainder)
__device__ __forceinline__ uint32_t hi16(float x) { return __float_as_uint(x) >> 16; }
__device__ __forceinline__ uint32_t lo16(float x) {
  return __float_as_uint(x - __uint_as_float(__float_as_uint(x) & 0xffff0000u)) >> 16;
}
// 4 consecutive floats -> hi / lo planes (8 bytes each)
__device__ __forceinline__ void st_split4(uint16_t* hi, uint16_t* lo, float4 v) {
  *reinterpret_cast<uint2*>(hi) = make_uint2(hi16(v.x) | (hi16(v.y) << 16), hi16(v.z) | (hi16(v.w) << 16));
  *reinterpret_cast<uint2*>(lo) = make_uint2(lo16(v.x) | (lo16(v.y) << 16), lo16(v.z) | (lo16(v.w) << 16));
}
__device__ __forceinline__ void st_split1(uint16_t* hi, uint16_t* lo, float x) {
  *hi = uint16_t(hi16(x));
  *lo = uint16_t(lo16(x));
}

// acc += A (16 x K) B (K x 16) for one 16 x 16 tile from bf16 hi/lo planes:
// A[i][k] = a[i * lda + k], B[k][j] = b[j * ldb + k] (k contiguous in both);
// three v_mfma_f32_16x16x32_bf16 per 32 k.
template <int K>
__device__ __forceinline__ f32x4 mm16x3(const uint16_t* ah, const uint16_t* al, int lda, const uint16_t* bh,
                                        const uint16_t* bl, int ldb, f32x4 acc, int lane) {
  const int i = lane & 15, kk = 8 * (lane >> 4);
#pragma unroll
  for (int k0 = 0; k0 < K; k0 += 32) {
    const bf16x8 xah = *reinterpret_cast<const bf16x8*>(ah + i * lda + k0 + kk);
    const bf16x8 xal = *reinterpret_cast<const bf16x8*>(al + i * lda + k0 + kk);
    const bf16x8 xbh = *reinterpret_cast<const bf16x8*>(bh + i * ldb + k0 + kk);
    const bf16x8 xbl = *reinterpret_cast<const bf16x8*>(bl + i * ldb + k0 + kk);
    acc = mfma3(xah, xal, xbh, xbl, acc);
  }
  return acc;
}

template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(kHT) void chunk_kernel(ChunkParams p) {
  using SM = ChunkSmem<DK, DV>;
  constexpr int KP = SM::KP, LKH = SM::LKH, LV = SM::LV, UL = SM::UL;
  constexpr int NTV = DV / 16;    // tiles across dv
  constexpr int NTILE = 2 * NTV;  // tiles of a 32 x DV block matrix
  constexpr int NKP = (kBc * DK / 4 + kHT - 1) / kHT;  // float4 of a block's keys per thread
  constexpr int NUP = (kBc * DV / 4 + kHT - 1) / kHT;  // float4 of a block's U rows per thread
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ uint32_t s_need;  // earlier blocks holding ancestors of the current block's nodes
  uint16_t* s_qh = reinterpret_cast<uint16_t*>(smem);  // block q~ planes [32][LKH]
  uint16_t* s_ql = s_qh + kBc * LKH;
  uint16_t* s_kh = s_ql + kBc * LKH;                    // block k~ planes
  uint16_t* s_kl = s_kh + kBc * LKH;
  uint16_t* s_s0h = reinterpret_cast<uint16_t*>(smem + SM::head);  // phase A: S0 planes [DV][LKH]
  uint16_t* s_s0l = s_s0h + DV * LKH;
  uint16_t* s_kch = reinterpret_cast<uint16_t*>(smem + SM::head);  // phase B: keys of block c
  uint16_t* s_kcl = s_kch + kBc * LKH;
  uint16_t* s_uth = s_kcl + kBc * LKH;  // U of block c, transposed [DV][UL]
  uint16_t* s_utl = s_uth + DV * UL;
  uint16_t* s_xh = s_utl + DV * UL;     // -X_jc [32][UL]
  uint16_t* s_xl = s_xh + kBc * UL;
  uint16_t* s_yh = s_xl + kBc * UL;     // Y_jc
  uint16_t* s_yl = s_yh + kBc * UL;
  float* s_y = reinterpret_cast<float*>(s_yl + kBc * UL);  // Y_jj [32][kLs] (fp32)
  float* s_pa = s_y + kBc * kLs;                            // powers of A
  float* s_pb = s_pa + kBc * kLs;
  float* s_ma = s_pb + kBc * kLs;                           // partial products of the inverse
  float* s_mb = s_ma + kBc * kLs;
  float* s_rt = s_mb + kBc * kLs;                           // R_j [32][LV]
  float* s_uj = s_rt + kBc * LV;                            // U_j [32][LV]
  uint64_t* s_anc = reinterpret_cast<uint64_t*>(smem + SM::head + SM::uni);  // [32][kHW]
  int16_t* s_ord = reinterpret_cast<int16_t*>(s_anc + kBc * kHW);
  int16_t* s_ppos = s_ord + kHMaxT;
  float* s_lal = reinterpret_cast<float*>(s_ppos + kHMaxT);
  float* s_la = s_lal + kHMaxT;
  float* s_be = s_la + kHMaxT;

  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int g = h * Hk / Hv;
  const int nq = Hk * DK;
  const size_t C = size_t(2 * nq + Hv * DV);
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int W = m.W;
  const size_t bt = size_t(b) * T;
  const int nval = m.status[b] == GDN_TREE_OK ? m.nvalid[b] : 0;
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  const float* Fb = p.F + bt * C;
  float* Ub = p.U + (size_t(b) * Hv + h) * size_t(T) * DV;
  float* outb = p.out + bt * size_t(Hv) * DV + size_t(h) * DV;

  // ---- metadata by position: node, parent position, log alpha, beta
  for (int j = tid; j < T; j += kHT) {
    const int nd = m.order[bt + j];
    const bool real = j < nval;
    s_ord[j] = int16_t(nd);
    s_ppos[j] = int16_t(real ? m.ppos[bt + j] : -1);
    // log alpha, floored at the smallest normal float so that alpha = 0
    // still gives finite ratios a_i / a_j
    s_lal[j] = real ? fmaxf(logf(ld(alpha, (bt + nd) * Hv + h)), -87.0f) : 0.0f;
    s_be[j] = real ? ld(beta, (bt + nd) * Hv + h) : 0.0f;
  }
  __syncthreads();
  // log a_p: sum of log alpha over the path root..p, by pointer jumping
  // (ceil(log2 T) rounds instead of a walk of depth(p) steps per position;
  // s_lal and s_ppos are rewritten to partial sums and 2^r-th ancestors)
  static_assert(kHT >= kHMaxT, "one position per thread");
  {
    float sl = tid < T ? s_lal[tid] : 0.0f;
    int nx = tid < T ? s_ppos[tid] : -1;
    for (int span = 1; span < T; span <<= 1) {
      if (nx >= 0) {
        sl += s_lal[nx];
        nx = s_ppos[nx];
      }
      __syncthreads();
      if (tid < T) {
        s_lal[tid] = sl;
        s_ppos[tid] = int16_t(nx);
      }
      __syncthreads();
    }
    if (tid < T) s_la[tid] = sl;
  }
  if (nval > 0) {
    const float* S0 = p.S0 + (size_t(b) * Hv + h) * size_t(DV) * DK;
    constexpr int NS4 = (DV * DK / 4 + kHT - 1) / kHT;  // float4 per thread, all in flight
    float4 sv[NS4];
#pragma unroll
    for (int j = 0; j < NS4; ++j) {
      const int i = j * kHT + tid < DV * DK / 4 ? j * kHT + tid : 0;
      sv[j] = *reinterpret_cast<const float4*>(S0 + size_t(i / (DK / 4)) * DK + 4 * (i % (DK / 4)));
    }
#pragma unroll
    for (int j = 0; j < NS4; ++j) {
      const int i = j * kHT + tid;
      if (i < DV * DK / 4) {
        const int r = i / (DK / 4), c4 = i % (DK / 4);
        st_split4(s_s0h + r * LKH + 4 * c4, s_s0l + r * LKH + 4 * c4, sv[j]);
      }
    }
    if constexpr (DK < KP) {  // zero padding of the contraction
      for (int i = tid; i < DV * (KP - DK); i += kHT) {
        const int r = i / (KP - DK), c = DK + i % (KP - DK);
        s_s0h[r * LKH + c] = 0;
        s_s0l[r * LKH + c] = 0;
      }
      for (int i = tid; i < 4 * kBc * (KP - DK); i += kHT) {
        const int r = i / (KP - DK), c = DK + i % (KP - DK);
        s_qh[r * LKH + c] = 0;  // q and k planes are contiguous: rows 0 .. 4 kBc - 1
      }
    }
  }
  __syncthreads();

  const int NB = (T + kBc - 1) / kBc, NBv = (nval + kBc - 1) / kBc;
  // block rows of q~ and k~ (zero past the tree) -> hi / lo planes: the
  // loads of a block go to registers first (all in flight together, issued
  // a block ahead where the planes are still in use), then to the planes
  constexpr int NQK = (2 * kBc * (DK / 4) + kHT - 1) / kHT;
  float4 qkv[NQK];
  auto fetch_qk = [&](int jb) {
#pragma unroll
    for (int j = 0; j < NQK; ++j) {
      const int i = j * kHT + tid;
      const int part = i / (kBc * (DK / 4)), rem = i % (kBc * (DK / 4));
      const int r = rem / (DK / 4), c4 = rem % (DK / 4);
      const int pos = kBc * jb + r;
      // clamped rows: every load is unconditional; rows past the tree are
      // zeroed at the store
      const int pc = pos < nval ? pos : 0;
      qkv[j] = *reinterpret_cast<const float4*>(Fb + pc * C + (part ? nq : 0) + g * DK + 4 * c4);
    }
  };
  auto store_qk = [&](int jb) {
#pragma unroll
    for (int j = 0; j < NQK; ++j) {
      const int i = j * kHT + tid;
      if (i < 2 * kBc * (DK / 4)) {
        const int part = i / (kBc * (DK / 4)), rem = i % (kBc * (DK / 4));
        const int r = rem / (DK / 4), c4 = rem % (DK / 4);
        const float4 v = kBc * jb + r < nval ? qkv[j] : make_float4(0.f, 0.f, 0.f, 0.f);
        st_split4((part ? s_kh : s_qh) + r * LKH + 4 * c4, (part ? s_kl : s_ql) + r * LKH + 4 * c4, v);
      }
    }
  };

  // ---- phase A: a Q S0^T -> out, beta (V - a K S0^T) -> U
  constexpr int NTA = (2 * NTILE + kHT / 64 - 1) / (kHT / 64);  // tasks per wave
  if (NBv > 0) fetch_qk(0);
  for (int jb = 0; jb < NB; ++jb) {
    if (jb < NBv) {
      store_qk(jb);
      if (jb + 1 < NBv) fetch_qk(jb + 1);  // in flight during this block's products
      // the value operands of this wave's K S0^T tasks, loaded ahead
      float vop[NTA][4];
#pragma unroll
      for (int ta = 0; ta < NTA; ++ta) {
        const int task = wave + ta * (kHT / 64);
        const int t = task % NTILE, ti = t / NTV, tj = t % NTV, col = 16 * tj + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pos = kBc * jb + 16 * ti + 4 * (lane >> 4) + r;
          vop[ta][r] = Fb[(pos < nval ? pos : 0) * C + 2 * nq + h * DV + col];
        }
      }
      __syncthreads();
#pragma unroll
      for (int ta = 0; ta < NTA; ++ta) {
        const int task = wave + ta * (kHT / 64);
        if (task >= 2 * NTILE) continue;  // uniform per wave
        const int kind = task / NTILE, t = task % NTILE;
        const int ti = t / NTV, tj = t % NTV;
        const f32x4 acc = mm16x3<KP>((kind ? s_kh : s_qh) + 16 * ti * LKH, (kind ? s_kl : s_ql) + 16 * ti * LKH,
                                     LKH, s_s0h + 16 * tj * LKH, s_s0l + 16 * tj * LKH, LKH, zero4(), lane);
        const int col = 16 * tj + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pos = kBc * jb + 16 * ti + 4 * (lane >> 4) + r;
          if (pos >= T) continue;
          const bool real = pos < nval;
          const float a = real ? expf(s_la[pos]) : 0.0f;
          if (kind == 0) {
            outb[size_t(s_ord[pos]) * Hv * DV + col] = real ? a * acc[r] : 0.0f;
          } else {
            Ub[size_t(pos) * DV + col] = real ? s_be[pos] * (vop[ta][r] - a * acc[r]) : 0.0f;
          }
        }
      }
      __syncthreads();
    } else {  // all padding
      for (int i = tid; i < kBc * DV; i += kHT) {
        const int pos = kBc * jb + i / DV;
        if (pos < T) outb[size_t(s_ord[pos]) * Hv * DV + i % DV] = 0.0f;
      }
    }
  }
  __syncthreads();  // S0 region reused below
  if constexpr (DK < KP) {
    for (int i = tid; i < 2 * kBc * (KP - DK); i += kHT) {
      const int r = i / (KP - DK), c = DK + i % (KP - DK);
      s_kch[r * LKH + c] = 0;  // hi and lo planes are contiguous
    }
  }

  // ---- phase B: forward substitution over the blocks
  // block-top inputs of block jb (the ancestor words of its rows, R_j and
  // the a Q S0^T part of O_j from phase A), loaded a block ahead: every load
  // is unconditional (clamped rows), padding is zeroed when they are used
  constexpr int NAW = (kBc * kHW + kHT - 1) / kHT;
  uint64_t awpf[NAW];
  f32x4 rrpf[2], oopf[2];
  auto fetch_top = [&](int jb) {
#pragma unroll
    for (int j = 0; j < NAW; ++j) {
      const int i = j * kHT + tid;
      const int r = (i / kHW) % kBc, w = i % kHW;
      const int pos = kBc * jb + r;
      awpf[j] = m.anc[(bt + s_ord[pos < nval ? pos : 0]) * W + (w < W ? w : 0)];
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = (wave + 8 * u) % NTILE;
      const int ti = t / NTV, tj = t % NTV, col = 16 * tj + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int pos = kBc * jb + 16 * ti + 4 * (lane >> 4) + r;
        const int pc = pos < nval ? pos : 0;
        rrpf[u][r] = Ub[size_t(pc) * DV + col];
        oopf[u][r] = outb[size_t(s_ord[pc]) * Hv * DV + col];
      }
    }
  };
  if (NBv > 0) {
    fetch_qk(0);
    fetch_top(0);
  }
  for (int jb = 0; jb < NBv; ++jb) {
    store_qk(jb);
#pragma unroll
    for (int j = 0; j < NAW; ++j) {
      const int i = j * kHT + tid;
      if (i < kBc * kHW) {
        const int r = i / kHW, w = i % kHW;
        s_anc[i] = (kBc * jb + r < nval && w < W) ? awpf[j] : 0ull;
      }
    }
    f32x4 rr[2], oo[2];  // R_j and O_j tiles of this wave: t = wave, wave + 8
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = wave + 8 * u;
      const int ti = (t % NTILE) / NTV;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool live = t < NTILE && kBc * jb + 16 * ti + 4 * (lane >> 4) + r < nval;
        rr[u][r] = live ? rrpf[u][r] : 0.0f;
        oo[u][r] = live ? oopf[u][r] : 0.0f;
      }
    }
    __syncthreads();
    // the earlier blocks that hold an ancestor of a node of this block (one
    // bit per block); their keys and U rows are loaded one block ahead
    if (tid == 0) s_need = 0u;
    __syncthreads();
    {
      uint32_t mask = 0u;
      for (int pr = tid; pr < kBc * kBc * jb; pr += kHT) {
        const int i = pr % kBc, pc = pr / kBc;
        if (kBc * jb + i < nval && pc < nval) {
          const int nd = s_ord[pc];
          if ((s_anc[i * kHW + (nd >> 6)] >> (nd & 63)) & 1ull) mask |= 1u << (pc / kBc);
        }
      }
      if (mask) atomicOr(&s_need, mask);
    }
    __syncthreads();
    uint32_t need = s_need;
    float4 kpf[NKP], upf[NUP];
    auto fetch = [&](int cb) {
#pragma unroll
      for (int j = 0; j < NKP; ++j) {
        const int i = j * kHT + tid;
        const int r = i < kBc * (DK / 4) ? i / (DK / 4) : 0, c4 = i < kBc * (DK / 4) ? i % (DK / 4) : 0;
        kpf[j] = *reinterpret_cast<const float4*>(Fb + (kBc * cb + r) * C + nq + g * DK + 4 * c4);
      }
#pragma unroll
      for (int j = 0; j < NUP; ++j) {
        const int i = j * kHT + tid;
        const int r = i < kBc * (DV / 4) ? i % kBc : 0, c4 = i < kBc * (DV / 4) ? i / kBc : 0;
        upf[j] = *reinterpret_cast<const float4*>(Ub + size_t(kBc * cb + r) * DV + 4 * c4);
      }
    };
    int cb = need ? __ffs(int(need)) - 1 : -1;
    if (cb >= 0) fetch(cb);
    while (cb >= 0) {
#pragma unroll
      for (int j = 0; j < NKP; ++j) {
        const int i = j * kHT + tid;
        if (i < kBc * (DK / 4)) {
          const int r = i / (DK / 4), c4 = i % (DK / 4);
          st_split4(s_kch + r * LKH + 4 * c4, s_kcl + r * LKH + 4 * c4, kpf[j]);
        }
      }
#pragma unroll
      for (int j = 0; j < NUP; ++j) {  // U_c transposed: [dv][node]
        const int i = j * kHT + tid;
        if (i < kBc * (DV / 4)) {
          const int r = i % kBc, c4 = i / kBc;
          const float4 u = upf[j];
          st_split1(s_uth + (4 * c4) * UL + r, s_utl + (4 * c4) * UL + r, u.x);
          st_split1(s_uth + (4 * c4 + 1) * UL + r, s_utl + (4 * c4 + 1) * UL + r, u.y);
          st_split1(s_uth + (4 * c4 + 2) * UL + r, s_utl + (4 * c4 + 2) * UL + r, u.z);
          st_split1(s_uth + (4 * c4 + 3) * UL + r, s_utl + (4 * c4 + 3) * UL + r, u.w);
        }
      }
      need &= need - 1u;
      const int nb = need ? __ffs(int(need)) - 1 : -1;
      if (nb >= 0) fetch(nb);  // the next block's loads fly during this one
      __syncthreads();
      {  // -X_jc (waves 0-3) and Y_jc (waves 4-7), one 16 x 16 tile each
        const int kind = wave >> 2, ti = (wave >> 1) & 1, tc = wave & 1;
        const f32x4 acc = mm16x3<KP>((kind ? s_qh : s_kh) + 16 * ti * LKH, (kind ? s_ql : s_kl) + 16 * ti * LKH,
                                     LKH, s_kch + 16 * tc * LKH, s_kcl + 16 * tc * LKH, LKH, zero4(), lane);
        const int c = 16 * tc + (lane & 15), pc = kBc * cb + c;
        const int nd = s_ord[pc];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = 16 * ti + 4 * (lane >> 4) + r, pi = kBc * jb + i;
          float val = 0.0f;
          if (pi < nval && pc < nval && ((s_anc[i * kHW + (nd >> 6)] >> (nd & 63)) & 1ull))
            val = expf(s_la[pi] - s_la[pc]) * acc[r];
          if (kind == 0)
            st_split1(s_xh + i * UL + c, s_xl + i * UL + c, -(pi < nval ? s_be[pi] : 0.0f) * val);
          else
            st_split1(s_yh + i * UL + c, s_yl + i * UL + c, val);
        }
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = wave + 8 * u;
        if (t < NTILE) {
          const int ti = t / NTV, tj = t % NTV;
          rr[u] = mm16x3<kBc>(s_xh + 16 * ti * UL, s_xl + 16 * ti * UL, UL, s_uth + 16 * tj * UL,
                              s_utl + 16 * tj * UL, UL, rr[u], lane);
          oo[u] = mm16x3<kBc>(s_yh + 16 * ti * UL, s_yl + 16 * ti * UL, UL, s_uth + 16 * tj * UL,
                              s_utl + 16 * tj * UL, UL, oo[u], lane);
        }
      }
      __syncthreads();
      cb = nb;
    }
    // ---- diagonal block: A = -X_jj, M0 = I + A, Y_jj; R_j -> LDS
    {
      const int kind = wave >> 2, ti = (wave >> 1) & 1, tc = wave & 1;
      const f32x4 acc = mm16x3<KP>((kind ? s_qh : s_kh) + 16 * ti * LKH, (kind ? s_ql : s_kl) + 16 * ti * LKH,
                                   LKH, s_kh + 16 * tc * LKH, s_kl + 16 * tc * LKH, LKH, zero4(), lane);
      const int c = 16 * tc + (lane & 15), pc = kBc * jb + c;
      const int nd = s_ord[pc];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 16 * ti + 4 * (lane >> 4) + r, pi = kBc * jb + i;
        const bool anc = pi < nval && pc < nval && ((s_anc[i * kHW + (nd >> 6)] >> (nd & 63)) & 1ull);
        if (kind == 0) {
          const float av = anc ? -s_be[pi] * expf(s_la[pi] - s_la[pc]) * acc[r] : 0.0f;
          s_pa[i * kLs + c] = av;
          s_ma[i * kLs + c] = av + (i == c ? 1.0f : 0.0f);
        } else {
          s_y[i * kLs + c] = (anc || (i == c && pi < nval)) ? expf(s_la[pi] - s_la[pc]) * acc[r] : 0.0f;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = wave + 8 * u;
      if (t < NTILE) {
        const int ti = t / NTV, tj = t % NTV, col = 16 * tj + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) s_rt[(16 * ti + 4 * (lane >> 4) + r) * LV + col] = rr[u][r];
      }
    }
    __syncthreads();
    // this block's q / k planes are read for the last time above: the next
    // block's rows and block-top inputs load during the inverse
    if (jb + 1 < NBv) {
      fetch_qk(jb + 1);
      fetch_top(jb + 1);
    }
    // ---- (I + X_jj)^-1 = (I + A)(I + A^2)(I + A^4)(I + A^8)(I + A^16):
    //      round s: waves 0-3 square the power of A, waves 4-7 multiply the
    //      partial product by (I + the power formed in round s - 1)
    {
      const int ti = (wave >> 1) & 1, tj = wave & 1;
      float* pw[2] = {s_pa, s_pb};
      float* mp[2] = {s_ma, s_mb};
#pragma unroll
      for (int s = 1; s <= 5; ++s) {
        if (wave < 4) {
          if (s <= 4) {
            const float* src = pw[(s - 1) & 1];
            const f32x4 d = mm16<kBc, false>(src + 16 * ti * kLs, kLs, src + 16 * tj, kLs, zero4(), lane);
            st_tile(pw[s & 1], ti, tj, lane, d);
          }
        } else if (s >= 2) {
          const float* msrc = mp[s & 1];          // M_{s-2}
          const float* psrc = pw[(s - 1) & 1];    // A^(2^(s-1))
          f32x4 d = ld_tile(msrc, ti, tj, lane);
          d = mm16<kBc, false>(msrc + 16 * ti * kLs, kLs, psrc + 16 * tj, kLs, d, lane);
          st_tile(mp[(s + 1) & 1], ti, tj, lane, d);
        }
        __syncthreads();
      }
    }
    // the inverse is in s_ma (M_4); U_j = M_4 R_j -> LDS and the workspace
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = wave + 8 * u;
      if (t < NTILE) {
        const int ti = t / NTV, tj = t % NTV, col = 16 * tj + (lane & 15);
        const f32x4 d = mm16<kBc, false>(s_ma + 16 * ti * kLs, kLs, s_rt + 16 * tj, LV, zero4(), lane);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 16 * ti + 4 * (lane >> 4) + r, pos = kBc * jb + row;
          s_uj[row * LV + col] = d[r];
          if (pos < T) Ub[size_t(pos) * DV + col] = d[r];
        }
      }
    }
    __syncthreads();
    // ---- O_j += Y_jj U_j, scaled and stored
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = wave + 8 * u;
      if (t < NTILE) {
        const int ti = t / NTV, tj = t % NTV, col = 16 * tj + (lane & 15);
        const f32x4 d = mm16<kBc, false>(s_y + 16 * ti * kLs, kLs, s_uj + 16 * tj, LV, oo[u], lane);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int pos = kBc * jb + 16 * ti + 4 * (lane >> 4) + r;
          if (pos < nval) outb[size_t(s_ord[pos]) * Hv * DV + col] = p.scale * d[r];
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Launch: features, then the chunked kernel
// ---------------------------------------------------------------------------
template <int DK, int DV, typename TIn>
static int launch_chunk_t(const ChunkParams& p, hipStream_t stream) {
  using SM = ChunkSmem<DK, DV>;
  const int rc = ensure_dynamic_lds(reinterpret_cast<const void*>(&chunk_kernel<DK, DV, TIn>), int(SM::total),
                                    "verify_chunked");
  if (rc != GDN_OK) return rc;
  hipLaunchKernelGGL((chunk_kernel<DK, DV, TIn>), dim3(p.Hv, p.B), dim3(kHT), SM::total, stream, p);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "verify_chunked launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

template <int DK, typename TIn>
static int chunk_dv(int dv, const ChunkParams& p, hipStream_t s) {
  switch (dv) {
    case 16: return launch_chunk_t<DK, 16, TIn>(p, s);
    case 32: return launch_chunk_t<DK, 32, TIn>(p, s);
    case 64: return launch_chunk_t<DK, 64, TIn>(p, s);
    case 128: return launch_chunk_t<DK, 128, TIn>(p, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify_chunked: dv=%d unsupported", dv);
}

template <typename TIn>
static int chunk_dk(int dk, int dv, const ChunkParams& p, hipStream_t s) {
  switch (dk) {
    case 16: return chunk_dv<16, TIn>(dv, p, s);
    case 32: return chunk_dv<32, TIn>(dv, p, s);
    case 64: return chunk_dv<64, TIn>(dv, p, s);
    case 128: return chunk_dv<128, TIn>(dv, p, s);
  }
  return set_error(GDN_EUNSUPPORTED, "verify_chunked: dk=%d unsupported", dk);
}

int launch_verify_chunked(const VerifyArgs& a, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (a.T > kHMaxT) return set_error(GDN_EUNSUPPORTED, "verify_chunked: T=%d exceeds %d", a.T, kHMaxT);
  if (ws_bytes < chunked_workspace_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv))
    return set_error(GDN_EINVAL, "verify_chunked: workspace of %zu bytes is too small", ws_bytes);
  float* F = static_cast<float*>(ws);
  int rc = launch_features(a, F, stream);
  if (rc != GDN_OK) return rc;
  ChunkParams p;
  p.B = a.B;
  p.T = a.T;
  p.Hk = a.Hk;
  p.Hv = a.Hv;
  p.scale = a.scale;
  p.meta = a.meta;
  p.alpha = a.alpha;
  p.beta = a.beta;
  p.S0 = a.S0;
  p.out = a.out;
  p.F = F;
  p.U = F + features_f32_bytes(a.B, a.T, a.Hk, a.Hv, a.dk, a.dv) / sizeof(float);
  if (a.in_dtype == GDN_BF16) return chunk_dk<BF16>(a.dk, a.dv, p, stream);
  return chunk_dk<float>(a.dk, a.dv, p, stream);
}

}  // namespace gdn
