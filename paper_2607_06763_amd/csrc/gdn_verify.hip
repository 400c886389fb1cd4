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
// per (sequence, value head), which runs on the MFMA units in fp16 with fp32
// accumulation: each row of S0 is first scaled by a power of two that brings
// its largest magnitude into [1, 2) (exact, undone on the output row), so any
// finite state fits the fp16 range; x~ is bounded by |q~| = 1.  The rounding
// of both operands to 11 significant bits puts the error of this product at
// ~1e-4 of max|o| on the named workloads.
//
// Workgroup = (dv slice, key head g with HPW of its value heads, sequence b),
// 512 threads.  Wave w owns 16 tree positions of the canonical (depth,
// index) order: 8 from a shallow block of 16 and 8 from a deep one, so that
// all waves walk about equally long paths.  Two layouts are used:
//   * conv / pull-back: 8 lanes per node, lane (n, o) = (lane / 8, lane % 8)
//     carries shallow node n and deep node n of the wave (walked one after
//     the other) and the channels lane_chan(o, r); a node's 8 lanes read 128
//     contiguous bytes of an LDS row per access, which keeps bank conflicts
//     low when the 8 nodes of a wave read 8 unrelated ancestor rows;
//   * MFMA: node column l16 = lane % 16, lane group mlg = lane / 16, the
//     B-operand layout of X~^T and the accumulator layout of O^T for
//     v_mfma_f32_16x16x32_f16.  The halves of each 8-lane group first trade
//     registers by DPP so that every ds_bpermute that moves the pulled-back
//     queries (fp16 pairs) and value accumulators across carries only values
//     its destination needs.
//   phase 0  tree metadata in canonical order -> LDS
//   phase 1  conv + SiLU + L2-norm of q and k along each node's path (raw
//            rows staged in LDS); q~ stays in registers, k~ -> LDS (fp32);
//            the first head's raw v and gates load meanwhile
//   per value head:
//     2a/b   raw v (prefetched) -> LDS, conv + SiLU -> v~ in LDS (fp32);
//            this head's S0 loads
//     2c     pull-back with k~, v~ gathered from LDS (8 lanes per node),
//            move to the MFMA layout
//     2d     S0 -> LDS as one fp16 plane of row-scaled values; the next
//            head's raw v and gates load (ahead of this head's stores)
//     2e     MFMA P^T = (D S0) X~^T, O^T = D^-1 P^T + ACC^T, store
// The fused step (FUSED) first commits the previous step's accepted path
// into each head's state rows, which then stand in for S0 (see
// fused_commit).
#include "gdn_internal.h"

namespace gdn {


constexpr int kVT = 512;        // threads per workgroup (8 waves)
constexpr int kVMaxT = 128;     // tree slots supported = 8 waves x 16 nodes
constexpr int kKPad = 4;        // fp32 row padding of the k~ and v~ tiles
constexpr int kSPad = 8;        // fp16 row padding of the S0 plane
constexpr int kLPN = 8;         // lanes per node in the conv / pull-back layout

struct VerifyParams {
  int B, T, Hk, Hv, DV, hpw;
  float scale;
  const void* meta;
  const void *q, *k, *v, *alpha, *beta;
  const float *conv_w, *conv_state, *S0;
  float* out;
  // fused step only: the previous step's accepted path is committed into S
  // (in place; S0 == S) and into conv_state_out before the verification
  const void* pmeta;
  const int32_t* paccepted;
  const void *pq, *pk, *pv, *palpha, *pbeta;
  float* conv_state_out;
  float* S;
  int32_t* commit_status;
};

// LDS rows of the conv / pull-back tiles: D floats, unpadded, for D >= 64;
// D + 4 floats otherwise.  With unpadded rows of 512 or 256 bytes the 128-byte
// chunk c of any row sits in bank half c % 2 (64 banks of 4 bytes), so when
// the odd lane groups of a wave read the chunks of their rows in the order
// c ^ 1 (chunk swap sw = 1) the two lane groups of every 16-lane quarter of a
// ds_read_b128 hit disjoint bank halves whatever rows they read.
template <int D>
__device__ __forceinline__ constexpr int row_floats() {
  return D >= 64 ? D : D + kKPad;
}
// chunk swap of the lane group ln for rows of D floats
template <int D>
__device__ __forceinline__ constexpr int chunk_swap(int ln) {
  return D >= 64 ? (ln & 1) : 0;
}

// Channel carried in register r (r < D / 8) by lane o (o < 8) of a node with
// chunk swap sw: groups of 4 consecutive channels, lane o taking group o of
// every 32-channel chunk, chunks in the order c ^ sw.
template <int D>
__device__ __forceinline__ constexpr int lane_chan(int o, int r, int sw) {
  return D >= 32 ? 32 * ((r / 4) ^ sw) + 4 * o + (r % 4) : 2 * o + r;
}

// This lane's D / 8 channels of an fp32 LDS row (16-byte or 8-byte pieces).
template <int D>
__device__ __forceinline__ void ld_lane(const float* row, int o, int sw, float (&x)[D / kLPN]) {
  if constexpr (D >= 32) {
#pragma unroll
    for (int c = 0; c < D / 32; ++c) {
      const float4 v = *reinterpret_cast<const float4*>(row + 32 * (c ^ sw) + 4 * o);
      x[4 * c] = v.x;
      x[4 * c + 1] = v.y;
      x[4 * c + 2] = v.z;
      x[4 * c + 3] = v.w;
    }
  } else {
    const float2 v = *reinterpret_cast<const float2*>(row + 2 * o);
    x[0] = v.x;
    x[1] = v.y;
  }
}
template <int D>
__device__ __forceinline__ void st_lane(float* row, int o, int sw, const float (&x)[D / kLPN]) {
  if constexpr (D >= 32) {
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
      *reinterpret_cast<float4*>(row + 32 * (c ^ sw) + 4 * o) =
          make_float4(x[4 * c], x[4 * c + 1], x[4 * c + 2], x[4 * c + 3]);
  } else {
    *reinterpret_cast<float2*>(row + 2 * o) = make_float2(x[0], x[1]);
  }
}

// Staged rows read by the four conv taps of the nodes at positions pos[u]:
// tap w of a node at depth d is its path node at depth d - 3 + w, or
// conv-state row T + d + w (slot d + w) above the root.  Inactive -> row 0.
__device__ __forceinline__ void conv_rows(const int* s_dep, const int* s_ppos, int T, const int (&pos)[2],
                                          const bool (&act)[2], int (&trow)[2][4]) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int w = 0; w < 4; ++w) trow[u][w] = 0;
    if (act[u]) {
      const int dep = s_dep[pos[u]];
      const int t2 = s_ppos[pos[u]];
      const int t1 = t2 >= 0 ? s_ppos[t2] : -1;
      const int t0 = t1 >= 0 ? s_ppos[t1] : -1;
      const int tp[4] = {t0, t1, t2, pos[u]};
#pragma unroll
      for (int w = 0; w < 4; ++w) trow[u][w] = (dep - 3 + w >= 0) ? tp[w] : T + dep + w;
    }
  }
}

// Offset (floats) of row t of a conv / pull-back tile.
template <int D>
__device__ __forceinline__ int row_off(int t) {
  static_assert((D & (D - 1)) == 0 && kKPad == 4, "power-of-two rows (plus 4)");
  return D >= 64 ? (t << __builtin_ctz(D)) : (t << __builtin_ctz(D)) + (t << 2);
}

// Workgroup barrier that orders LDS accesses only: global loads and stores
// issued before it stay in flight (a full __syncthreads waits for all of
// them).  No thread here reads global memory another thread writes.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Streaming load of 16 bytes (the raw q, k, v rows, read once per launch):
// the non-temporal hint keeps them from displacing the state rows in the
// caches.
__device__ __forceinline__ uint4 load_stream(const void* src) {
  typedef unsigned u32v4 __attribute__((ext_vector_type(4)));
  const u32v4 v = __builtin_nontemporal_load(reinterpret_cast<const u32v4*>(src));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Pins x to a register at this point: keeps the compiler from sinking the
// arithmetic that produces it past a later barrier (which would keep every
// operand it reads alive across the barrier).
__device__ __forceinline__ void pin(float& x) { asm volatile("" : "+v"(x)); }

// The thread index as a value the compiler cannot see through: addresses
// derived from it are computed where they are used instead of being hoisted
// out of the head loop and held in registers across it (which spills, and a
// spill reload waits for every vector memory operation issued before it).
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Value of v held by lane src of this wave (ds_bpermute).
__device__ __forceinline__ float lane_gather(float v, int src) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(v)));
}

// LDS regions (bytes) for a tree of T slots, key dim DK and value slice DVS
struct VerifySmem {
  size_t rk, rv, meta, p0, total;
};
__host__ __device__ inline VerifySmem verify_smem(int T, int DK, int DVS, bool fused) {
  const int TP = (T + 15) & ~15;
  const int kappa = DK >= 32 ? DK : 32;
  const size_t rows = size_t(TP > T + 3 ? TP : T + 3);
  VerifySmem s;
  const int krow = DK >= 64 ? DK : DK + kKPad, vrow = DVS >= 64 ? DVS : DVS + kKPad;
  s.rk = rows * krow * 4;                                   // q staging [T+3][krow], then k~ [TP][krow]
  const size_t k_stage = rows * krow * 4;                   // k staging [T+3][krow]
  const size_t v_tile = rows * vrow * 4;                    // v staging [T+3][vrow], then v~
  const size_t s_tile = size_t(DVS) * (kappa + kSPad) * 2;  // S0 fp16 plane
  s.rv = k_stage > v_tile ? k_stage : v_tile;
  s.rv = s.rv > s_tile ? s.rv : s_tile;
  const size_t c_tile = size_t(kMC) * (DK + DVS) * 4 + kMC * 4 + 2 * kVMaxT * 4;  // fused commit
  s.rv = s.rv > c_tile ? s.rv : c_tile;
  s.meta = size_t(3 * kVMaxT) * 4                           // order, parent pos, depth
           + size_t(2 * kVMaxT) * 4                         // alpha, beta of the current head
           + size_t(8 * DK) * 4 + size_t(4 * DVS) * 4       // q/k and v conv weights
           + size_t(kVMaxT) * 4                             // previous path (fused step)
           + size_t(kVMaxT) * 4;                            // S0 row scales
  // fused step with two row pieces per thread: the first half of the fp16
  // plane, written right after the commit, so that its registers can take
  // the next head's rows during the pull-back
  const bool split = fused && DVS * DK / kVT >= 16;
  s.p0 = split ? size_t(DVS / 2) * (kappa + kSPad) * 2 : 0;
  s.total = s.rk + s.rv + s.meta + s.p0;
  return s;
}

// Issue the loads of this thread's share of S0[b][h][c0 .. c0+DVS][0 .. DK).
// Only the loads j with j % PARTS == part are issued, so that a prefetch can
// be spread over the steps of a compute phase (a burst of loads holds the
// issuing wave until most of its data has arrived).
// When the slice has at least one float4 per thread, each thread takes NS0
// consecutive float4 of one row (S0 rows of TPR threads), so that a row's
// scale needs one max over TPR lanes; otherwise thread tid takes float4
// j kVT + tid.
template <int DK, int DVS>
struct S0Split {
  static constexpr int N4 = DVS * DK / 4;        // float4 of the slice
  static constexpr bool kRows = N4 >= kVT;       // the row-wise split applies
  static constexpr int NS0 = kRows ? N4 / kVT : 1;
  static constexpr int TPR = kRows ? DK / 4 / NS0 : 1;  // threads per row
  static_assert(!kRows || (TPR >= 1 && TPR <= 32 && NS0 * TPR == DK / 4), "S0 split");
};
template <int DK, int DVS, int NS0, int PARTS = 1>
__device__ __forceinline__ void prefetch_s0(const float* S0bh, int tid, float4 (&pf)[NS0], int part = 0) {
  using SP = S0Split<DK, DVS>;
  static_assert(SP::NS0 == NS0, "S0 split");
#pragma unroll
  for (int j = 0; j < NS0; ++j) {
    if (j % PARTS != part) continue;
    if constexpr (SP::kRows) {
      const int idx = (tid / SP::TPR) * (DK / 4) + (tid % SP::TPR) * NS0 + j;
      pf[j] = reinterpret_cast<const float4*>(S0bh)[idx];
    } else {
      const int idx = j * kVT + tid;
      pf[j] = idx < SP::N4 ? reinterpret_cast<const float4*>(S0bh)[idx] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
}

// Issue the loads of this thread's share of the raw values v[b][.][h][c0 .. c0+DVS)
// for the T nodes (16-byte chunks, node-major).
template <typename TIn, int DVS, int NVC, int PARTS = 1>
__device__ __forceinline__ void prefetch_v(const TIn* vin, size_t node_stride, const int* s_ord,
                                           int T, int tid, uint4 (&pf)[NVC], int part = 0) {
  constexpr int EPC = 16 / sizeof(TIn);  // elements per 16-byte chunk
  constexpr int CPR = DVS / EPC;         // chunks per node row
#pragma unroll
  for (int j = 0; j < NVC; ++j) {
    if (j % PARTS != part) continue;
    const int idx = j * kVT + tid;
    const int p = idx / CPR < T ? idx / CPR : T - 1, c = idx % CPR;  // rows >= T are never stored
    pf[j] = load_stream(vin + size_t(s_ord[p]) * node_stride + c * EPC);
  }
}

// Conv-state slot s seen by a step after the commit of a path of L nodes
// (L = 0: nothing committed): the last three raw inputs of (old slots 0..2,
// path p_0 .. p_{L-1}), i.e. the old slot L + s while L + s < 3, else the
// raw input of path node L - 3 + s.
__device__ __forceinline__ int slot_old(int L, int s) { return L + s < 3 ? L + s : 2; }
__device__ __forceinline__ bool slot_from_path(int L, int s) { return L + s >= 3; }

// Gates (alpha, beta of the T positions), v conv weights ([4][DVS],
// tap-major) and v conv-state rows ([3][DVS]) of one value head, loaded
// into registers ahead of their use.  Every load is unconditional (indices
// are clamped) so that nothing waits for it before the store.  In the fused
// step the conv-state rows are those after the commit of the previous path
// (Lp nodes, path positions in s_ppath, raw values pv of the previous step).
template <int DVS, typename TIn, bool FUSED>
struct HeadGates {
  static constexpr int NW = (4 * DVS + kVT - 1) / kVT;
  static constexpr int NC = (3 * DVS + kVT - 1) / kVT;
  TIn al, be;
  float w[NW], cs[NC];
  TIn cr[FUSED ? NC : 1];  // raw inputs of the committed path (fused step)
  int Lp = 0;
  __device__ __forceinline__ void load(const TIn* alpha, const TIn* beta, const float* conv_w,
                                       const float* conv_state, const int* s_ord, int b, int T, int Hv,
                                       int C, int h, int vch0, int tid, const TIn* pv = nullptr,
                                       size_t vrow = 0, int vcol0 = 0, const int* s_ppath = nullptr, int L = 0) {
    const size_t ab = (size_t(b) * T + s_ord[tid < T ? tid : 0]) * Hv + h;
    al = alpha[ab];
    be = beta[ab];
    Lp = L;
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      const int i = j * kVT + tid < 4 * DVS ? j * kVT + tid : 4 * DVS - 1;
      w[j] = conv_w[size_t(vch0 + i % DVS) * 4 + i / DVS];
    }
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int i = j * kVT + tid < 3 * DVS ? j * kVT + tid : 3 * DVS - 1;
      const int sl = i / DVS;
      cs[j] = conv_state[(size_t(b) * 3 + slot_old(L, sl)) * C + vch0 + i % DVS];
      if constexpr (FUSED) {
        const int node = slot_from_path(L, sl) ? s_ppath[L - 3 + sl] : 0;
        cr[j] = pv[(size_t(b) * T + node) * vrow + vcol0 + i % DVS];
      }
    }
  }
  // gates -> s_al, s_be; weights -> s_wv; conv-state rows -> rows T..T+2 of
  // the v staging tile
  __device__ __forceinline__ void store(float* s_al, float* s_be, float* s_wv, float* s_v, int vrow, int T,
                                        int tid) const {
    if (tid < T) {
      s_al[tid] = to_f32(al);
      s_be[tid] = to_f32(be);
    }
#pragma unroll
    for (int j = 0; j < NW; ++j)
      if (j * kVT + tid < 4 * DVS) s_wv[j * kVT + tid] = w[j];
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      const int i = j * kVT + tid;
      if (i < 3 * DVS) {
        float x = cs[j];
        if constexpr (FUSED) x = slot_from_path(Lp, i / DVS) ? to_f32(cr[j]) : x;
        s_v[(T + i / DVS) * vrow + i % DVS] = x;
      }
    }
  }
};

// Split of a DVS x DK state slice over the workgroup for the fused commit:
// each thread holds R rows (q + i RS, i < R, RS = DVS / R) times CPT
// consecutive columns; LPR lanes share a row.  Two rows per thread halve the
// LDS reads of the key slices in the replay (every row of a step reads the
// same key).  The first DVS DK / EPT threads own elements (all of them
// unless DVS DK < kVT).  Element e of a thread is row row(tid, e / CPT),
// column col0(tid) + e % CPT.
template <int DK, int DVS>
struct FusedSplit {
  static constexpr int EPT = DVS * DK >= kVT ? DVS * DK / kVT : 1;
  static constexpr int R = EPT >= 16 ? 2 : 1;
  static constexpr int CPT = EPT / R;
  static constexpr int LPR = DK / CPT;
  static constexpr int RS = DVS / R;
  static_assert(CPT >= 1 && LPR >= 1 && LPR <= 64 && (LPR & (LPR - 1)) == 0 && DVS % R == 0, "fused state split");
  __device__ static __forceinline__ bool owns(int tid) { return tid < RS * LPR; }
  __device__ static __forceinline__ int row(int tid, int i) { return (owns(tid) ? tid / LPR : RS - 1) + i * RS; }
  __device__ static __forceinline__ int col0(int tid) { return (tid % LPR) * CPT; }
};

// State rows c0 .. c0 + DVS of head h (before the fused commit) in the
// commit layout, part `part` of PARTS: the run of 16-byte groups (4
// consecutive elements of one row piece) [part G / PARTS, (part + 1) G /
// PARTS) of the thread's G groups, or all elements when a row piece is not a
// multiple of 4 wide (part 0 only).  With PARTS <= R a part is whole row
// pieces, so the threads of a row still cover whole cache lines.  Threads
// that own no elements load rows of thread 0 (never stored).
template <int DK, int DVS, int PARTS = 1>
__device__ __forceinline__ void load_state_rows(const float* S, int b, int Hv, int DV, int h, int c0, int tid,
                                                float (&sr)[FusedSplit<DK, DVS>::EPT], int part = 0) {
  using FS = FusedSplit<DK, DVS>;
  const int t = FS::owns(tid) ? tid : 0;
  const float* base = S + ((size_t(b) * Hv + h) * DV + c0 + FS::row(t, 0)) * DK + FS::col0(t);
  if constexpr (FS::CPT % 4 == 0) {
#pragma unroll
    for (int gi = 0; gi < FS::EPT / 4; ++gi) {
      if (gi * PARTS / (FS::EPT / 4) != part) continue;
      const int i = gi / (FS::CPT / 4), e = 4 * (gi % (FS::CPT / 4));
      const float4 v = *reinterpret_cast<const float4*>(base + size_t(i) * FS::RS * DK + e);
      sr[i * FS::CPT + e] = v.x;
      sr[i * FS::CPT + e + 1] = v.y;
      sr[i * FS::CPT + e + 2] = v.z;
      sr[i * FS::CPT + e + 3] = v.w;
    }
  } else {
    if (part != 0) return;
#pragma unroll
    for (int i = 0; i < FS::R; ++i)
#pragma unroll
      for (int e = 0; e < FS::CPT; ++e) sr[i * FS::CPT + e] = base[size_t(i) * FS::RS * DK + e];
  }
}

// Stores part `part` of PARTS of this thread's state elements to the rows of
// head h (the grouping of load_state_rows).
template <int DK, int DVS, int PARTS = 1>
__device__ __forceinline__ void store_state_rows(float* S, int b, int Hv, int DV, int h, int c0, int tid,
                                                 const float (&sr)[FusedSplit<DK, DVS>::EPT], int part = 0) {
  using FS = FusedSplit<DK, DVS>;
  if (!FS::owns(tid)) return;
  float* base = S + ((size_t(b) * Hv + h) * DV + c0 + FS::row(tid, 0)) * DK + FS::col0(tid);
  if constexpr (FS::CPT % 4 == 0) {
#pragma unroll
    for (int gi = 0; gi < FS::EPT / 4; ++gi) {
      if (gi * PARTS / (FS::EPT / 4) != part) continue;
      const int i = gi / (FS::CPT / 4), e = 4 * (gi % (FS::CPT / 4));
      *reinterpret_cast<float4*>(base + size_t(i) * FS::RS * DK + e) =
          make_float4(sr[i * FS::CPT + e], sr[i * FS::CPT + e + 1], sr[i * FS::CPT + e + 2], sr[i * FS::CPT + e + 3]);
    }
  } else {
    if (part != 0) return;
#pragma unroll
    for (int i = 0; i < FS::R; ++i)
#pragma unroll
      for (int e = 0; e < FS::CPT; ++e) base[size_t(i) * FS::RS * DK + e] = sr[i * FS::CPT + e];
  }
}

// Fused step: row piece i of this thread's state elements -> the fp16 plane
// at base (rows in natural order, stride KS halves), each row scaled by the
// power of two of row_scale; the inverse scales -> s_rs.
template <int DK, int DVS, int KS>
__device__ __forceinline__ void plane_piece(const float (&sr)[FusedSplit<DK, DVS>::EPT], int i, _Float16* base,
                                            float* s_rs, int tid) {
  using FS = FusedSplit<DK, DVS>;
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < FS::CPT; ++e) m = fmaxf(m, fabsf(sr[i * FS::CPT + e]));
  m = group_max<FS::LPR>(m);
  float sc, inv;
  row_scale(m, sc, inv);
  if (FS::owns(tid)) {
    const int off = FS::row(tid, i) * KS + FS::col0(tid);
    if constexpr (FS::CPT % 4 == 0) {
#pragma unroll
      for (int e = 0; e < FS::CPT; e += 4)
        *reinterpret_cast<uint2*>(base + off + e) = to_f16x4(
            make_float4(sr[i * FS::CPT + e], sr[i * FS::CPT + e + 1], sr[i * FS::CPT + e + 2], sr[i * FS::CPT + e + 3]),
            sc);
    } else {
#pragma unroll
      for (int e = 0; e < FS::CPT; ++e) base[off + e] = (_Float16)(sr[i * FS::CPT + e] * sc);
    }
    if (FS::col0(tid) == 0) s_rs[FS::row(tid, i)] = inv;
  }
}

// Commit (fused step) of the previous step's accepted path (L nodes, slots
// s_ppath) into the state rows c0 .. c0 + DVS of value head h: features of
// the path (previous step's raw inputs, conv state before the commit), then
// one rank-1 step per path node on this thread's elements of the rows
// (Eq. 7, see replay_rows).  sr holds the elements before the commit on
// entry (load_state_rows) and after it on return; the caller stores them
// (store_state_rows).  Uses lds (the value-tile region) and ends with a
// barrier; a uniform no-op when L = 0.
template <int DK, int DVS, typename TIn>
__device__ __forceinline__ void fused_commit(const VerifyParams& p, unsigned char* lds, const int* s_ppath, int L,
                                             int b, int g, int h, int c0, int tid,
                                             float (&sr)[FusedSplit<DK, DVS>::EPT]) {
  using FS = FusedSplit<DK, DVS>;
  constexpr int EPT = FS::EPT, LPR = FS::LPR, R = FS::R, CPT = FS::CPT;
  constexpr int FP = 4 * (DK + DVS) <= kVT ? 4 : 2;  // feature parts per chunk
  constexpr int FN = kMC / FP;                       // path nodes per feature task
  static_assert(FP * (DK + DVS) <= kVT, "one feature task per thread");
  if (L == 0) return;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv, DV = p.DV;
  const int C = 2 * Hk * DK + Hv * DV;
  float* s_fk = reinterpret_cast<float*>(lds);  // [kMC][DK] keys (unnormalised)
  float* s_fv = s_fk + kMC * DK;                // [kMC][DVS] values of the slice
  float* s_inv = s_fv + kMC * DVS;              // [kMC] 1 / ||k||
  float* s_al = s_inv + kMC;                    // [kVMaxT] gates by path index
  float* s_be = s_al + kVMaxT;
  // gates of path node tid (tid < L): loaded with the first chunk's window
  // and stored with its features, so that one wait covers both
  const size_t gab = (size_t(b) * T + s_ppath[tid < L ? tid : 0]) * Hv + h;
  // feature task of this thread: value channel of the slice (tid < FP DVS)
  // or key channel (FP DVS <= tid < FP (DVS + DK)); fpart picks the part
  const bool vtask = tid < FP * DVS;
  const bool ktask = !vtask && tid < FP * (DVS + DK);
  const int tt = vtask ? tid : tid - FP * DVS;
  const int fc = vtask ? tt % DVS : tt % DK;
  const int fpart = vtask ? tt / DVS : tt / DK;
  const int fch = vtask ? 2 * Hk * DK + h * DV + c0 + fc : Hk * DK + g * DK + fc;  // conv channel
  const TIn* fsrc = vtask ? static_cast<const TIn*>(p.pv) + size_t(b) * T * Hv * DV + size_t(h) * DV + c0 + fc
                          : static_cast<const TIn*>(p.pk) + size_t(b) * T * Hk * DK + size_t(g) * DK + fc;
  const size_t fstride = vtask ? size_t(Hv) * DV : size_t(Hk) * DK;
  const float* fcs = p.conv_state + size_t(b) * 3 * C + fch;
  const int row0 = FS::row(tid, 0), col0 = FS::col0(tid);
  float gamma = 1.0f;
  for (int base = 0; base < L; base += kMC) {
    FeatWindow<TIn, FN> win;
    if (vtask || ktask) win.load(fsrc, fstride, fcs, C, p.conv_w + size_t(fch) * 4, s_ppath, base + fpart * FN, L);
    TIn gal, gbe;
    if (base == 0) {  // clamped loads, issued after the window's
      gal = static_cast<const TIn*>(p.palpha)[gab];
      gbe = static_cast<const TIn*>(p.pbeta)[gab];
    }
    if (vtask || ktask) {
      const int m0 = base + fpart * FN;
#pragma unroll
      for (int mr = 0; mr < FN; ++mr) {
        const float y = silu(win.w.x * win.x(mr, m0, L) + win.w.y * win.x(mr + 1, m0, L) +
                             win.w.z * win.x(mr + 2, m0, L) + win.w.w * win.x(mr + 3, m0, L));
        if (vtask)
          s_fv[(fpart * FN + mr) * DVS + fc] = y;
        else
          s_fk[(fpart * FN + mr) * DK + fc] = y;
      }
    }
    if (base == 0 && tid < L) {
      s_al[tid] = to_f32(gal);
      s_be[tid] = to_f32(gbe);
    }
    __syncthreads();
    // key norms: 16 lanes per path node, DK / 16 channels per lane
    {
      constexpr int CPL = DK / 16;
      const int nd = tid >> 4, ln = tid & 15;
      float ss = 0.0f;
      if (nd < kMC) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const float y = s_fk[nd * DK + ln * CPL + c];
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
      ld_slice<CPT>(s_fk + mr * DK + col0, kk);
#pragma unroll
      for (int i = 0; i < R; ++i) vr[i] = s_fv[mr * DVS + row0 + i * FS::RS];
      gamma = replay_rows<R, CPT, LPR>(sr, kk, vr, s_al[base + mr], s_be[base + mr], s_inv[mr], gamma);
    }
    __syncthreads();  // chunk features consumed
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) sr[e] *= gamma;
}

// Conv state after the fused commit for the channels a workgroup owns:
// q and k of key head g (if owns_qk) and v of heads h0 .. h0 + hpw - 1,
// channels c0 .. c0 + DVS.  Slot s is the old slot Lp + s while that is
// below 3, else the raw input of path node Lp - 3 + s.
template <int DK, int DVS, typename TIn>
__device__ __forceinline__ void fused_conv_out(const VerifyParams& p, const int* s_ppath, int L, int b, int g,
                                               int h0, int c0, bool owns_qk, int tid) {
  const int T = p.T, Hk = p.Hk, Hv = p.Hv, DV = p.DV;
  const int C = 2 * Hk * DK + Hv * DV;
  const float* cs = p.conv_state + size_t(b) * 3 * C;
  float* co = p.conv_state_out + size_t(b) * 3 * C;
  if (owns_qk) {
    const size_t qk_row = size_t(Hk) * DK;
    for (int i = tid; i < 3 * 2 * DK; i += kVT) {
      const int sl = i / (2 * DK), part = (i / DK) & 1, c = i % DK;
      const int ch = part * Hk * DK + g * DK + c;
      const TIn* src = static_cast<const TIn*>(part ? p.pk : p.pq);
      const float x = slot_from_path(L, sl) ? ld(src, (size_t(b) * T + s_ppath[L - 3 + sl]) * qk_row + g * DK + c)
                                            : cs[size_t(slot_old(L, sl)) * C + ch];
      co[size_t(sl) * C + ch] = x;
    }
  }
  const size_t v_row = size_t(Hv) * DV;
  const int nv = p.hpw * DVS;
  for (int i = tid; i < 3 * nv; i += kVT) {
    const int sl = i / nv, j = i % nv;
    const int col = (h0 + j / DVS) * DV + c0 + j % DVS;
    const int ch = 2 * Hk * DK + col;
    const float x = slot_from_path(L, sl)
                        ? ld(static_cast<const TIn*>(p.pv), (size_t(b) * T + s_ppath[L - 3 + sl]) * v_row + col)
                        : cs[size_t(slot_old(L, sl)) * C + ch];
    co[size_t(sl) * C + ch] = x;
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

template <int DK, int DVS, typename TIn, bool FUSED>
__global__ __launch_bounds__(kVT) void verify_kernel(VerifyParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int KPL = DK / kLPN;              // key channels per lane and node
  constexpr int VPL = DVS / kLPN;             // value channels per lane and node
  constexpr int KB = DK >= 32 ? DK / 32 : 1;  // 32-wide MFMA k blocks (dk = 16 is zero-padded)
  constexpr int KAPPA = 32 * KB;              // MFMA k extent
  constexpr int KROW = row_floats<DK>();      // k~ / staging row stride (floats)
  constexpr int NT = DVS / 16;                // 16-row value tiles of this slice
  constexpr int VROW = row_floats<DVS>();     // v~ / staging row stride (floats)
  constexpr int EPC = 16 / sizeof(TIn);
  constexpr int NS0 = FUSED ? 1 : S0Split<DK, DVS>::NS0;  // S0 float4 per thread
  constexpr int NSR = FUSED ? FusedSplit<DK, DVS>::EPT : 1;       // state floats per thread (fused)
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
  // Positions are sorted by depth, so path lengths grow with the position.
  // Wave w takes the even (w < 4) or odd (w >= 4) positions of the shallow
  // block w % 4 and of the deep block 7 - w % 4: every wave then walks about
  // the same number of steps in total.
  const int pw = wave & 3, hw = wave >> 2;
  const int base[2] = {16 * pw + hw, 16 * (7 - pw) + hw};
  // conv / pull-back layout: node n = lane / 8 of each half, lane o = lane % 8
  const int ln = lane >> 3, lo = lane & 7;
  const int ksw = chunk_swap<DK>(ln), vsw = chunk_swap<DVS>(ln);  // chunk order of this lane group
  const int pos[2] = {base[0] + 2 * ln, base[1] + 2 * ln};
  // MFMA layout: node column l16 (l16 < 8 from the shallow half, else the
  // deep one), channel group mlg
  const int l16 = lane & 15, mlg = lane >> 4;
  const int mpos = l16 < 8 ? base[0] + 2 * l16 : base[1] + 2 * (l16 - 8);

  const VerifySmem L = verify_smem(T, DK, DVS, FUSED);
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
  int* s_ppath = reinterpret_cast<int*>(s_wv + 4 * DVS);  // previous accepted path (fused step)
  float* s_rs = reinterpret_cast<float*>(s_ppath + kVMaxT);  // 1 / row scale of the S0 plane
  _Float16* s_p0 = reinterpret_cast<_Float16*>(smem + L.rk + L.rv + L.meta);  // plane rows of piece 0 (fused)
  // fused step, two row pieces per thread: piece 0's plane rows go to s_p0
  // right after the commit and its registers take the next head's rows
  // during the pull-back; piece 1 as before
  constexpr bool kSplit = FUSED && FusedSplit<DK, DVS>::R == 2;

  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const int status = m.status[b];
  const int nv = m.nvalid[b];
  // fused step: the previous step's accepted path root..a (Lp nodes, slot
  // s_ppath[j] at depth j) is read off a's ancestor bitmask; Lp = 0 when
  // nothing is committed (accepted -1 or a non-zero commit status)
  int Lp = 0;
  float sr[NSR];  // fused step: this thread's state elements of the current head
  if constexpr (FUSED) {
    const MetaPtrs pm = meta_ptrs(p.pmeta, p.B, T);
    const int pa = p.paccepted[b];
    const int pst = pm.status[b];
    int cst = pst != GDN_TREE_OK ? pst : (pa >= -1 && pa < T ? GDN_TREE_OK : GDN_TREE_BAD_ACCEPTED);
    if (cst == GDN_TREE_OK && pa >= 0) {
      const int da = pm.depth[size_t(b) * T + pa];
      if (da < 0) cst = GDN_TREE_BAD_ACCEPTED;
      else Lp = da + 1;
    }
    if (tid < kVMaxT) s_ppath[tid] = 0;  // every path index stays a valid slot
    __syncthreads();
    if (Lp > 0 && tid < T) {
      const uint64_t word = pm.anc[(size_t(b) * T + pa) * pm.W + (tid >> 6)];
      const int dj = pm.depth[size_t(b) * T + tid];
      if ((tid == pa || ((word >> (tid & 63)) & 1ull)) && dj >= 0 && dj < Lp) s_ppath[dj] = tid;
    }
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0 && p.commit_status) p.commit_status[b] = cst;
    __syncthreads();
  }
  if (status != GDN_TREE_OK) {
    if constexpr (FUSED) {  // the previous path is committed all the same
      for (int hh = 0; hh < p.hpw; ++hh) {
        load_state_rows<DK, DVS>(p.S, b, Hv, DV, h0 + hh, c0, tid, sr);
        fused_commit<DK, DVS, TIn>(p, s_rv, s_ppath, Lp, b, g, h0 + hh, c0, tid, sr);
        if (Lp > 0) store_state_rows<DK, DVS>(p.S, b, Hv, DV, h0 + hh, c0, tid, sr);
      }
      fused_conv_out<DK, DVS, TIn>(p, s_ppath, Lp, b, g, h0, c0, blockIdx.x == 0 && blockIdx.y % nhg == 0, tid);
    }
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
  __syncthreads();
  const TIn* vin = static_cast<const TIn*>(p.v);
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  float4 s0pf[NS0];
  uint4 vpf[NVC];
  HeadGates<DVS, TIn, FUSED> gpf;

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
        qpf[j] = load_stream(qsrc + off);
        kpf[j] = load_stream(ksrc + off);
      }
    }
    float* s_kst = reinterpret_cast<float*>(s_rv);
    const float* csq = p.conv_state + size_t(b) * 3 * C + g * DK;
    constexpr int NQS = (3 * DK + kVT - 1) / kVT;
    float cq[NQS], ck[NQS];
    TIn cqr[FUSED ? NQS : 1], ckr[FUSED ? NQS : 1];  // fused step: raw inputs of the committed path
#pragma unroll
    for (int j = 0; j < NQS; ++j) {
      const int i = j * kVT + tid < 3 * DK ? j * kVT + tid : 3 * DK - 1;
      const int sl = i / DK;
      cq[j] = csq[size_t(slot_old(Lp, sl)) * C + i % DK];
      ck[j] = csq[size_t(slot_old(Lp, sl)) * C + Hk * DK + i % DK];
      if constexpr (FUSED) {
        const int node = slot_from_path(Lp, sl) ? s_ppath[Lp - 3 + sl] : 0;
        const size_t off = (size_t(b) * T + node) * qk_row + size_t(g) * DK + i % DK;
        cqr[j] = static_cast<const TIn*>(p.pq)[off];
        ckr[j] = static_cast<const TIn*>(p.pk)[off];
      }
    }
#pragma unroll
    for (int j = 0; j < NQC; ++j) {
      const int idx = j * kVT + tid;
      const int row = idx / QCPR, c = (idx % QCPR) * EPC;
      if (row < T) {
        store_chunk_f32(s_k + row * KROW + c, qpf[j], static_cast<const TIn*>(nullptr));
        store_chunk_f32(s_kst + row * KROW + c, kpf[j], static_cast<const TIn*>(nullptr));
      }
    }
#pragma unroll
    for (int j = 0; j < NQS; ++j) {
      const int i = j * kVT + tid;
      if (i < 3 * DK) {
        float xq = cq[j], xk = ck[j];
        if constexpr (FUSED) {
          if (slot_from_path(Lp, i / DK)) {
            xq = to_f32(cqr[j]);
            xk = to_f32(ckr[j]);
          }
        }
        s_k[(T + i / DK) * KROW + i % DK] = xq;
        s_kst[(T + i / DK) * KROW + i % DK] = xk;
      }
    }
    // the first head's raw values and gates (and, fused step, its state
    // rows) load during the q / k conv, issued once the q and k rows have
    // arrived so that they do not queue behind them
    prefetch_v<TIn, DVS>(vin + size_t(b) * T * orow + size_t(h0) * DV + c0, orow, s_ord, T, tid, vpf);
    if constexpr (FUSED) {
      gpf.load(alpha, beta, p.conv_w, p.conv_state, s_ord, b, T, Hv, C, h0, 2 * Hk * DK + h0 * DV + c0, tid,
               static_cast<const TIn*>(p.pv), orow, h0 * DV + c0, s_ppath, Lp);
      load_state_rows<DK, DVS>(p.S, b, Hv, DV, h0, c0, tid, sr);
    } else {
      gpf.load(alpha, beta, p.conv_w, p.conv_state, s_ord, b, T, Hv, C, h0, 2 * Hk * DK + h0 * DV + c0, tid);
    }
  }
  __syncthreads();
  bool act[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) act[u] = pos[u] < nv;
  int trow[2][4];
  conv_rows(s_dep, s_ppos, T, pos, act, trow);
  float qh[2][KPL];  // q~ of this lane's two nodes (channels lane_chan(lo, r, ksw))
  float kh[2][KPL];
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const float* stage = part == 0 ? s_k : reinterpret_cast<const float*>(s_rv);
    const float* wpart = s_wqk + part * 4 * DK;
    float y[2][KPL];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int c = 0; c < KPL; ++c) y[u][c] = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      float wt[KPL];
      ld_lane<DK>(wpart + w * DK, lo, ksw, wt);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float xw[KPL];
        ld_lane<DK>(stage + trow[u][w] * KROW, lo, ksw, xw);
#pragma unroll
        for (int c = 0; c < KPL; ++c) y[u][c] += wt[c] * xw[c];
      }
      __builtin_amdgcn_sched_barrier(0);  // one tap's rows in flight at a time
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      float ss = 0.0f;
#pragma unroll
      for (int c = 0; c < KPL; ++c) {
        y[u][c] = silu(y[u][c]);
        ss += y[u][c] * y[u][c];
      }
      ss = group_sum<kLPN>(ss);
      const float inv = act[u] ? rsqrt_hw(ss + 1e-6f) : 0.0f;
#pragma unroll
      for (int c = 0; c < KPL; ++c) {
        if (part == 0) {
          qh[u][c] = y[u][c] * inv;
        } else {
          kh[u][c] = y[u][c] * inv;
          pin(kh[u][c]);
        }
      }
    }
  }
  __syncthreads();  // staged rows consumed
#pragma unroll
  for (int u = 0; u < 2; ++u)
    if (act[u]) st_lane<DK>(s_k + pos[u] * KROW, lo, ksw, kh[u]);

  // ---------------- phase 2: one value head at a time ----------------
  // MFMA lane (l16, mlg) takes node l16 from half l16 / 8 of the 8-lane
  // group starting at lane sbase
  const int mhalf = l16 >> 3;
  const int sbase = kLPN * (l16 & 7);
  for (int hh = 0; hh < p.hpw; ++hh) {
    const int h = h0 + hh;
    // fused step: commit the previous path into this head's state rows (sr
    // then holds the state the tree is verified against)
    if constexpr (FUSED) fused_commit<DK, DVS, TIn>(p, s_rv, s_ppath, Lp, b, g, h, c0, tid, sr);
    if constexpr (kSplit) plane_piece<DK, DVS, KAPPA + kSPad>(sr, 0, s_p0, s_rs, tid);
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
    }
    gpf.store(s_al, s_be, s_wv, s_v, VROW, T, tid);
    // fused step: the committed rows of this head go to S in two parts (one
    // row piece each, whole cache lines) spread over 2a .. 2c, behind compute
    constexpr int kSP = 2;
    if constexpr (FUSED)
      if (Lp > 0) store_state_rows<DK, DVS, kSP>(p.S, b, Hv, DV, h, c0, tid, sr, 0);
    __syncthreads();
    // 2b: v~ of this lane's two nodes, channels lane_chan(lo, r, vsw)
    float vt[2][VPL];
    {
      int trow[2][4];  // recomputed per head: fewer registers held across heads
      conv_rows(s_dep, s_ppos, T, pos, act, trow);
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int c = 0; c < VPL; ++c) vt[u][c] = 0.0f;
      // this head's S0 (needed after the pull-back)
      if constexpr (!FUSED)
        prefetch_s0<DK, DVS, NS0>(p.S0 + (size_t(b) * Hv + h) * DV * DK + size_t(c0) * DK, tid, s0pf);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        float wt[VPL];
        ld_lane<DVS>(s_wv + w * DVS, lo, vsw, wt);
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          float xw[VPL];
          ld_lane<DVS>(s_v + trow[u][w] * VROW, lo, vsw, xw);
#pragma unroll
          for (int c = 0; c < VPL; ++c) vt[u][c] += wt[c] * xw[c];
        }
        __builtin_amdgcn_sched_barrier(0);  // one tap's rows in flight at a time
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int c = 0; c < VPL; ++c) {
          vt[u][c] = silu(vt[u][c]);
          pin(vt[u][c]);
        }
    }
    __syncthreads();  // staged rows consumed
#pragma unroll
    for (int u = 0; u < 2; ++u)
      if (act[u]) st_lane<DVS>(s_v + pos[u] * VROW, lo, vsw, vt[u]);
    __syncthreads();

    // 2c: query pull-back along the path of each node, leaf to root; the
    //     lane walks its shallow node, then its deep one
    float x[2][KPL], acc[2][VPL];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int c = 0; c < KPL; ++c) x[u][c] = qh[u][c];
#pragma unroll
      for (int c = 0; c < VPL; ++c) acc[u][c] = 0.0f;
      float r = 1.0f;
      int t = act[u] ? pos[u] : -1;
      // a path has at most T nodes; the bound also ends the walk on corrupt metadata
      for (int step = 0; step < T && t >= 0; ++step) {
        const float be = s_be[t];
        const float al = s_al[t];
        const int nx = s_ppos[t];
        float kt[KPL], vv[VPL];
        ld_lane<DK>(s_k + row_off<DK>(t), lo, ksw, kt);
        ld_lane<DVS>(s_v + row_off<DVS>(t), lo, vsw, vv);
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int c = 0; c < KPL; c += 2) {
          s0 += kt[c] * x[u][c];
          s1 += kt[c + 1] * x[u][c + 1];
        }
        const float bs = be * group_sum<kLPN>(s0 + s1);
        const float rbs = r * bs;
#pragma unroll
        for (int c = 0; c < KPL; ++c) x[u][c] -= bs * kt[c];
#pragma unroll
        for (int c = 0; c < VPL; ++c) acc[u][c] += rbs * vv[c];
        r *= al;
        t = nx;
      }
      // a_i x~ rounded to fp32 first in both kernels (no fused multiply +
      // fp16 conversion), so that they round the B operand identically
#pragma unroll
      for (int c = 0; c < KPL; ++c) {
        x[u][c] *= r;
        pin(x[u][c]);
      }
      if constexpr (FUSED)
        if (Lp > 0 && u == 0) store_state_rows<DK, DVS, kSP>(p.S, b, Hv, DV, h, c0, tid, sr, 1);
      // the next head's rows of piece 0 (stored already, converted at the
      // head start) load during the deep walk
      if constexpr (kSplit)
        if (u == 0 && hh + 1 < p.hpw) load_state_rows<DK, DVS, 2>(p.S, b, Hv, DV, h + 1, c0, tid, sr, 0);
    }
    // a_i x~_i and the value accumulators move to the MFMA layout:
    //   X~^T B operand, k block kb: lane (l16, mlg) holds channels 32 kb + 8 mlg + e
    //   O^T accumulator, tile n:    lane (l16, mlg) holds channels 16 n + 4 mlg + e
    // x~ goes over as fp16 (the B operand's type, |x~| <= |q~| = 1).  Key
    // block kb of column (node, mlg) reads lanes 2 mlg (e < 4) and 2 mlg + 1
    // (e >= 4) of the node's group.  The even and odd lanes of a group first
    // trade registers by DPP (lane o <-> o ^ 1): even lanes then hold node 0's
    // channels of both lanes, odd lanes node 1's, packed as fp16 pairs (even
    // lane's channel low), so one ds_bpermute moves two needed values: 16 per
    // lane instead of 64.
    f16x8 xb[KB];  // B operand of X~^T
    if constexpr (DK >= 32) {
      const bool evn = (lo & 1) == 0;
      uint32_t px[KPL];
#pragma unroll
      for (int rr = 0; rr < KPL; ++rr) {
        const float send = evn ? x[1][rr] : x[0][rr];
        const float recv = dpp_f<kDppQuadXor1>(send);
        const float b0 = evn ? x[0][rr] : recv;
        const float b1 = evn ? recv : x[1][rr];
        px[rr] = uint32_t(__builtin_bit_cast(uint16_t, (_Float16)b0)) |
                 (uint32_t(__builtin_bit_cast(uint16_t, (_Float16)b1)) << 16);
      }
      __builtin_amdgcn_sched_barrier(0);  // x~ in fp32 is dead from here on
      const int src = sbase + 2 * mlg + mhalf;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t w = uint32_t(__builtin_amdgcn_ds_bpermute(src << 2, int(px[4 * kb + q])));
          xb[kb][q] = __builtin_bit_cast(_Float16, uint16_t(w & 0xffffu));
          xb[kb][q + 4] = __builtin_bit_cast(_Float16, uint16_t(w >> 16));
        }
      }
    } else {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int rr = e & 1, src = (sbase + 4 * mlg + (e >> 1)) & 63;
          const float a0 = lane_gather(x[0][rr], src);
          const float a1 = lane_gather(x[1][rr], src);
          float xv = mlg < 2 ? (mhalf ? a1 : a0) : 0.0f;
          pin(xv);
          xb[kb][e] = (_Float16)xv;
        }
      }
    }
    float am[NT][4];
    if constexpr (DVS >= 32) {
      // Tile n reads the lanes o = 4 (n & 1) + mlg of a group.  First the
      // halves of each group trade registers (lane o <-> 7 - o, one DPP move
      // per register): lanes 0..3 then hold node 0's channels of both tile
      // parities (acc[0]: own, acc[1]: from lane 7 - o), lanes 4..7 node 1's
      // (acc[0]: from lane 7 - o, acc[1]: own), so that every ds_bpermute
      // moves a value its destination column needs: 32 instead of 64.
      const bool lowh = lo < 4;
#pragma unroll
      for (int rr = 0; rr < VPL; ++rr) {
        const float send = lowh ? acc[1][rr] : acc[0][rr];
        const float recv = dpp_f<kDppRowHalfMirror>(send);
        const float b0 = lowh ? acc[0][rr] : recv;
        const float b1 = lowh ? recv : acc[1][rr];
        acc[0][rr] = b0;
        acc[1][rr] = b1;
      }
#pragma unroll
      for (int n = 0; n < NT; ++n) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rr = 4 * (n >> 1) + e;
          // source lane of (node half, tile parity): own data at mlg / 4 + mlg,
          // traded data at the mirror lane 3 - mlg / 7 - mlg
          const int sl = (n & 1) ? (mhalf ? 4 + mlg : 3 - mlg) : (mhalf ? 7 - mlg : mlg);
          am[n][e] = lane_gather((n & 1) ? acc[1][rr] : acc[0][rr], sbase + sl);
          pin(am[n][e]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int n = 0; n < NT; ++n) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rr = e & 1, src = sbase + 2 * mlg + (e >> 1);
          const float a0 = lane_gather(acc[0][rr], src);
          const float a1 = lane_gather(acc[1][rr], src);
          am[n][e] = mhalf ? a1 : a0;
          pin(am[n][e]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // a column whose source lane group is odd (l16 odd) received the 32-channel
    // chunks in the swapped order c ^ 1: put them back in place
    if (l16 & 1) {
      if constexpr (DK >= 64) {
#pragma unroll
        for (int kb = 0; kb < KB; kb += 2) {
          const f16x8 t0 = xb[kb];
          xb[kb] = xb[kb + 1];
          xb[kb + 1] = t0;
        }
      }
      if constexpr (DVS >= 64) {
#pragma unroll
        for (int n = 0; n < NT; ++n)
          if ((n & 2) == 0)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float t0 = am[n][e];
              am[n][e] = am[n + 2][e];
              am[n + 2][e] = t0;
            }
      }
    }
    __syncthreads();  // v~ consumed

    // 2d: S0 of this head -> LDS as one fp16 plane [DVS][KAPPA + kSPad] of
    //     row-scaled values (key channels in natural order, 16..31 zero for
    //     dk = 16); the inverse row scales -> s_rs
    {
      _Float16* s_h = reinterpret_cast<_Float16*>(s_rv);
      if constexpr (FUSED) {
#pragma unroll
        for (int i = kSplit ? 1 : 0; i < FusedSplit<DK, DVS>::R; ++i)
          plane_piece<DK, DVS, KAPPA + kSPad>(sr, i, s_h, s_rs, tid);
      } else if constexpr (S0Split<DK, DVS>::kRows) {
        // NS0 float4 of row tid / TPR: one scale per row from a TPR-lane max
        using SP = S0Split<DK, DVS>;
        float m = 0.0f;
#pragma unroll
        for (int j = 0; j < NS0; ++j) {
          const float4 x = s0pf[j];
          m = fmaxf(m, fmaxf(fmaxf(fabsf(x.x), fabsf(x.y)), fmaxf(fabsf(x.z), fabsf(x.w))));
        }
        m = group_max<SP::TPR>(m);
        float sc, inv;
        row_scale(m, sc, inv);
        const int row = tid / SP::TPR, k0 = (tid % SP::TPR) * NS0;
#pragma unroll
        for (int j = 0; j < NS0; ++j)
          *reinterpret_cast<uint2*>(s_h + row * (KAPPA + kSPad) + 4 * (k0 + j)) = to_f16x4(s0pf[j], sc);
        if (k0 == 0) s_rs[row] = inv;
      } else {
#pragma unroll
        for (int j = 0; j < NS0; ++j) {
          const int idx = j * kVT + tid;
          // DK / 4 consecutive threads hold one row (a power of two <= 32)
          const float4 x = s0pf[j];
          float m = fmaxf(fmaxf(fabsf(x.x), fabsf(x.y)), fmaxf(fabsf(x.z), fabsf(x.w)));
          m = group_max<DK / 4>(m);
          float sc, inv;
          row_scale(m, sc, inv);
          if (NS0 * kVT == DVS * DK / 4 || idx < DVS * DK / 4) {
            const int row = idx / (DK / 4), kch = idx % (DK / 4);
            *reinterpret_cast<uint2*>(s_h + row * (KAPPA + kSPad) + 4 * kch) = to_f16x4(x, sc);
            if (kch == 0) s_rs[row] = inv;
          }
        }
      }
      if (DK < 32) {
        for (int i = tid; i < DVS * 4; i += kVT) {
          const int row = i / 4, kch = 4 + i % 4;
          *reinterpret_cast<uint2*>(s_h + row * (KAPPA + kSPad) + 4 * kch) = make_uint2(0, 0);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // this head's S0 registers are free before the next loads
    // fused step: the next head's state rows load during the MFMA phase
    // (its fused commit at the start of the next head needs them)
    if constexpr (FUSED) {
      if (hh + 1 < p.hpw) {
        if constexpr (kSplit)
          load_state_rows<DK, DVS, 2>(p.S, b, Hv, DV, h + 1, c0, tid, sr, 1);
        else
          load_state_rows<DK, DVS>(p.S, b, Hv, DV, h + 1, c0, tid, sr);
      }
    }
    // the next head's raw values and gates load ahead of this head's output
    // stores: loads and stores complete in issue order, so the wait for
    // them at the next head's start then does not wait for the stores,
    // which drain behind the next head's work (the barriers below order LDS
    // only)
    if (hh + 1 < p.hpw) {
      const int otid = opaque(tid);
      prefetch_v<TIn, DVS>(vin + size_t(b) * T * orow + size_t(h + 1) * DV + c0, orow, s_ord, T, otid, vpf);
      if constexpr (FUSED)
        gpf.load(alpha, beta, p.conv_w, p.conv_state, s_ord, b, T, Hv, C, h + 1, vch0 + DV, otid,
                 static_cast<const TIn*>(p.pv), orow, (h + 1) * DV + c0, s_ppath, Lp);
      else
        gpf.load(alpha, beta, p.conv_w, p.conv_state, s_ord, b, T, Hv, C, h + 1, vch0 + DV, otid);
    }
    lds_barrier();

    // 2e: P^T = (D S0) X~^T on MFMA (fp16 operands, fp32 accumulation);
    //     O^T = scale (D^-1 P^T + ACC^T) in the accumulator layout; store
    {
      const _Float16* s_h = reinterpret_cast<const _Float16*>(s_rv);
      const int node = mpos < T ? s_ord[mpos] : 0;
      float* orow_p = p.out + (size_t(b) * T + node) * orow + size_t(h) * DV + c0;
      // two tiles at a time: both tiles' operands are read first and the two
      // accumulation chains interleave
#pragma unroll
      for (int n = 0; n < NT; n += 2) {
        constexpr int NP = NT > 1 ? 2 : 1;
        f16x8 a[NP][KB];
        float4 rs[NP];
#pragma unroll
        for (int u = 0; u < NP; ++u) {
#pragma unroll
          for (int kb = 0; kb < KB; ++kb)
            a[u][kb] = *reinterpret_cast<const f16x8*>((kSplit && 16 * (n + u) < DVS / 2 ? s_p0 : s_h) +
                                                       (16 * (n + u) + l16) * (KAPPA + kSPad) + 32 * kb + 8 * mlg);
          rs[u] = *reinterpret_cast<const float4*>(s_rs + 16 * (n + u) + 4 * mlg);
        }
        f32x4 d[NP];
#pragma unroll
        for (int u = 0; u < NP; ++u) d[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int u = 0; u < NP; ++u) d[u] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[u][kb], xb[kb], d[u], 0, 0, 0);
#pragma unroll
        for (int u = 0; u < NP; ++u) {
          const int t = n + u;
          if (mpos < T)
            *reinterpret_cast<float4*>(orow_p + 16 * t + 4 * mlg) =
                make_float4(p.scale * fmaf(d[u][0], rs[u].x, am[t][0]), p.scale * fmaf(d[u][1], rs[u].y, am[t][1]),
                            p.scale * fmaf(d[u][2], rs[u].z, am[t][2]), p.scale * fmaf(d[u][3], rs[u].w, am[t][3]));
        }
      }
    }
    lds_barrier();  // S0 planes consumed before the next head reuses the region
  }
  if constexpr (FUSED)
    fused_conv_out<DK, DVS, TIn>(p, s_ppath, Lp, b, g, h0, c0, blockIdx.x == 0 && blockIdx.y % nhg == 0, tid);
}

template <int DK, int DVS, typename TIn, bool FUSED>
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
  const size_t smem = verify_smem(a.T, DK, DVS, FUSED).total;
  const int rc = ensure_dynamic_lds(reinterpret_cast<const void*>(&verify_kernel<DK, DVS, TIn, FUSED>),
                                    int(verify_smem(kVMaxT, DK, DVS, FUSED).total), "verify");
  if (rc != GDN_OK) return rc;
  const int G = a.Hv / a.Hk;
  hipLaunchKernelGGL((verify_kernel<DK, DVS, TIn, FUSED>), dim3(ns, a.Hk * (G / hpw), a.B), dim3(kVT), smem,
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
  if (a.fused) {
    switch (a.dv / ns) {
      case 16: return launch_verify_t<DK, 16, TIn, true>(a, hpw, ns, s);
      case 32: return launch_verify_t<DK, 32, TIn, true>(a, hpw, ns, s);
      case 64: return launch_verify_t<DK, 64, TIn, true>(a, hpw, ns, s);
      case 128: return launch_verify_t<DK, 128, TIn, true>(a, hpw, ns, s);
    }
  } else {
    switch (a.dv / ns) {
      case 16: return launch_verify_t<DK, 16, TIn, false>(a, hpw, ns, s);
      case 32: return launch_verify_t<DK, 32, TIn, false>(a, hpw, ns, s);
      case 64: return launch_verify_t<DK, 64, TIn, false>(a, hpw, ns, s);
      case 128: return launch_verify_t<DK, 128, TIn, false>(a, hpw, ns, s);
    }
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
