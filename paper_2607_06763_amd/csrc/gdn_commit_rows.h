// gdn_commit_rows.h -- the commit of one (sequence, value head): the
// accepted slot's path root..a advances the state rows S[b][h] by Eq. 7
// (Sec. 3.4.2), one rank-1 step per path node, on NT threads that each hold
// pieces of R state rows in registers.  Shared by the commit kernel and the
// fused step above 128 slots (the pull-back kernel), which then reads the
// committed rows from registers instead of from memory.
#pragma once

#include "gdn_internal.h"

namespace gdn {

// threads per state workgroup: 512, or one per state element for tiny heads
constexpr int commit_threads(int dk, int dv) { return dk * dv >= 512 ? 512 : dk * dv; }
constexpr int kCMaxT = 512;    // tree slots supported
constexpr int kMH = kMC / 2;   // path nodes per feature half

struct CommitParams {
  int B, T, Hk, Hv;
  const void* meta;
  const int32_t* accepted;
  const void *q, *k, *v, *alpha, *beta;
  const float* conv_w;
  const float* cs_in;  // conv state before the commit
  float* cs_out;       // conv state after it (may equal cs_in)
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

// LDS of one commit (4 kCMaxT + kMC (DK + DV + 1) words)
struct CommitLds {
  int* path;    // [kCMaxT] path slot by depth
  int* dep;     // [kCMaxT] depth of every slot
  float* al;    // [kCMaxT] gates by path index
  float* be;
  float* fk;    // [kMC][DK] SiLU(conv) keys of a path chunk (before the norm)
  float* fv;    // [kMC][DV] SiLU(conv) values of a path chunk
  float* inv;   // [kMC] 1 / ||k|| per path node of the chunk
};
template <int DK, int DV>
__host__ __device__ constexpr size_t commit_lds_bytes() {
  return size_t(4 * kCMaxT + kMC * (DK + DV + 1)) * 4;
}
template <int DK, int DV>
__device__ __forceinline__ CommitLds commit_lds(unsigned char* base) {
  CommitLds l;
  l.path = reinterpret_cast<int*>(base);
  l.dep = l.path + kCMaxT;
  l.al = reinterpret_cast<float*>(l.dep + kCMaxT);
  l.be = l.al + kCMaxT;
  l.fk = l.be + kCMaxT;
  l.fv = l.fk + kMC * DK;
  l.inv = l.fv + kMC * DV;
  return l;
}

// Split of the DV x DK state over NT threads: thread tid holds rows
// tid / LPR + i RS (i < R), CPT consecutive columns from (tid % LPR) CPT.
template <int DK, int DV, int NT>
struct CommitSplit {
  static constexpr int EPT = DV * DK / NT;  // state elements per thread
  static constexpr int R = EPT >= 16 ? 2 : 1;
  static constexpr int CPT = EPT / R;
  static constexpr int LPR = DK / CPT;
  static constexpr int RS = DV / R;
  static_assert(EPT >= 1 && (EPT < 4 || EPT % 4 == 0) && DV % R == 0, "state split");
  static_assert(LPR >= 1 && LPR <= 32 && (LPR & (LPR - 1)) == 0, "row lanes");
  static_assert(2 * (DK + DV) <= NT, "one feature task per thread");
};

// Commit of the accepted path of sequence b into the rows of value head h.
// The first load wave (status, depths and gates of every slot) does not
// depend on the accepted slot a; the path is read off a's ancestor bitmask;
// one thread per (feature channel, half of a 32-node chunk) slides the
// width-4 conv window along the path (conv-state slots above the root),
// the key norms are reduced per path node, and every path node is one
// rank-1 step on the rows (replay_rows).  On return srow holds the rows
// after the commit, and the result says whether they changed (a committed
// path).  When nothing is committed the rows are loaded only if ALWAYS_LOAD
// (the fused step reads them either way).  Writes commit_status[b] from
// (h == 0, tid == 0).  Every exit is uniform over the workgroup; uses the
// LDS in l and ends with a barrier.
template <int DK, int DV, typename TIn, int NT, bool ALWAYS_LOAD>
__device__ __forceinline__ bool commit_rows(const CommitParams& p, int b, int h, int tid, const CommitLds& l,
                                            float (&srow)[CommitSplit<DK, DV, NT>::EPT]) {
  using CS = CommitSplit<DK, DV, NT>;
  constexpr int EPT = CS::EPT, R = CS::R, CPT = CS::CPT, LPR = CS::LPR, RS = CS::RS;
  const int T = p.T, Hk = p.Hk, Hv = p.Hv;
  const int g = h * Hk / Hv;
  const int C = 2 * Hk * DK + Hv * DV;
  const MetaPtrs m = meta_ptrs(p.meta, p.B, T);
  const TIn* alpha = static_cast<const TIn*>(p.alpha);
  const TIn* beta = static_cast<const TIn*>(p.beta);
  const int row = tid / LPR;
  const int col0 = (tid % LPR) * CPT;
  float* Sbh = p.S + (size_t(b) * Hv + h) * size_t(DV) * DK + size_t(row) * DK + col0;
  auto load_rows = [&]() {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      float piece[CPT];
      ld_slice<CPT>(Sbh + size_t(i) * RS * DK, piece);
#pragma unroll
      for (int e = 0; e < CPT; ++e) srow[i * CPT + e] = piece[e];
    }
  };

  // ---- first load wave: status, depths and gates of this thread's slots (raw
  //      gates are converted only once the path is known)
  constexpr int kSl = (kCMaxT + NT - 1) / NT;  // slots per thread
  const int a = p.accepted[b];
  const int tree_st = m.status[b];
  int dep[kSl];
  TIn alr[kSl], ber[kSl];
#pragma unroll
  for (int sl = 0; sl < kSl; ++sl) {
    const int j = tid + sl * NT;
    const int jj = j < T ? j : T - 1;
    dep[sl] = m.depth[size_t(b) * T + jj];
    alr[sl] = alpha[(size_t(b) * T + jj) * Hv + h];
    ber[sl] = beta[(size_t(b) * T + jj) * Hv + h];
  }
  if (tree_st != GDN_TREE_OK || a < 0 || a >= T) {
    if (h == 0 && tid == 0 && p.commit_status)
      p.commit_status[b] = tree_st != GDN_TREE_OK ? tree_st : (a == -1 ? GDN_TREE_OK : GDN_TREE_BAD_ACCEPTED);
    if (ALWAYS_LOAD) load_rows();
    __syncthreads();
    return false;
  }
  // ---- second load wave: the ancestor bitmask of a -> the path root..a
  uint64_t word[kSl];
#pragma unroll
  for (int sl = 0; sl < kSl; ++sl) {
    const int j = tid + sl * NT;
    word[sl] = m.anc[(size_t(b) * T + a) * m.W + ((j < T ? j : T - 1) >> 6)];
    if (j < T) l.dep[j] = dep[sl];
  }
  __syncthreads();
  const int d = l.dep[a];
  if (h == 0 && tid == 0 && p.commit_status)
    p.commit_status[b] = d < 0 ? GDN_TREE_BAD_ACCEPTED : GDN_TREE_OK;
  if (d < 0) {  // accepted slot is padding
    if (ALWAYS_LOAD) load_rows();
    __syncthreads();
    return false;
  }
#pragma unroll
  for (int sl = 0; sl < kSl; ++sl) {
    const int j = tid + sl * NT;
    if (j < T && (j == a || ((word[sl] >> (j & 63)) & 1ull))) {
      l.path[dep[sl]] = j;
      l.al[dep[sl]] = to_f32(alr[sl]);
      l.be[dep[sl]] = to_f32(ber[sl]);
    }
  }
  __syncthreads();
  const int L = d + 1;  // path length

  // ---- feature task of this thread: value channel (tid < 2 DV) or key
  //      channel (2 DV <= tid < 2 (DV + DK)); fhalf picks the half of a chunk
  const bool vtask = tid < 2 * DV;
  const bool ktask = !vtask && tid < 2 * (DV + DK);
  const int tt = vtask ? tid : tid - 2 * DV;
  const int fc = vtask ? tt % DV : tt % DK;
  const int fhalf = vtask ? tt / DV : tt / DK;
  const int fch = vtask ? 2 * Hk * DK + h * DV + fc : Hk * DK + g * DK + fc;  // conv channel
  const TIn* fsrc = vtask ? static_cast<const TIn*>(p.v) + size_t(b) * T * Hv * DV + size_t(h) * DV + fc
                          : static_cast<const TIn*>(p.k) + size_t(b) * T * Hk * DK + size_t(g) * DK + fc;
  const size_t fstride = vtask ? size_t(Hv) * DV : size_t(Hk) * DK;
  const float* fcs = p.cs_in + size_t(b) * 3 * C + fch;
  FeatWindow<TIn, kMH> win;
  if (vtask || ktask) win.load(fsrc, fstride, fcs, C, p.conv_w + size_t(fch) * 4, l.path, fhalf * kMH, L);

  // ---- the state rows load behind the first windows
  load_rows();

  // S_true = gamma * srow: one step costs one FMA for S.k and one for the
  // rank-1 write, S_true <- alpha S_true + c k  <=>  srow += c / (alpha gamma) k
  float gamma = 1.0f;
  for (int base = 0; base < L; base += kMC) {
    if (base > 0 && (vtask || ktask))  // long paths: later chunks load here
      win.load(fsrc, fstride, fcs, C, p.conv_w + size_t(fch) * 4, l.path, base + fhalf * kMH, L);
    // features of the chunk (window element q is path node m0 - 3 + q)
    if (vtask || ktask) {
      const int m0 = base + fhalf * kMH;
      float* dst = vtask ? l.fv + fc : l.fk + fc;
      const int stride = vtask ? DV : DK;
#pragma unroll
      for (int mr = 0; mr < kMH; ++mr)
        dst[(fhalf * kMH + mr) * stride] = silu(win.w.x * win.x(mr, m0, L) + win.w.y * win.x(mr + 1, m0, L) +
                                                win.w.z * win.x(mr + 2, m0, L) + win.w.w * win.x(mr + 3, m0, L));
    }
    __syncthreads();
    // key norms: 16 lanes per path node, DK / 16 channels per lane
#pragma unroll
    for (int nd0 = 0; nd0 < kMC; nd0 += NT / 16) {
      constexpr int CPL = DK / 16;
      const int nd = nd0 + (tid >> 4), ln = tid & 15;
      float ss = 0.0f;
      if (nd < kMC) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          const float y = l.fk[nd * DK + ln * CPL + c];
          ss += y * y;
        }
      }
      ss = group_sum<16>(ss);
      if (nd < kMC && ln == 0) l.inv[nd] = rsqrt_hw(ss + 1e-6f);
    }
    __syncthreads();
    const int cnt = L - base < kMC ? L - base : kMC;
    for (int mr = 0; mr < cnt; ++mr) {
      float kk[CPT], vr[R];
      ld_slice<CPT>(l.fk + mr * DK + col0, kk);
#pragma unroll
      for (int i = 0; i < R; ++i) vr[i] = l.fv[mr * DV + row + i * RS];
      gamma = replay_rows<R, CPT, LPR>(srow, kk, vr, l.al[base + mr], l.be[base + mr], l.inv[mr], gamma);
    }
    __syncthreads();  // chunk features consumed
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) srow[e] *= gamma;
  return true;
}

// srow (rows tid / LPR + i RS, CPT columns from (tid % LPR) CPT) back to S[b][h]
template <int DK, int DV, int NT>
__device__ __forceinline__ void store_rows(float* S, int b, int h, int Hv, int tid,
                                           const float (&srow)[CommitSplit<DK, DV, NT>::EPT]) {
  using CS = CommitSplit<DK, DV, NT>;
  const int row = tid / CS::LPR, col0 = (tid % CS::LPR) * CS::CPT;
  float* Sbh = S + (size_t(b) * Hv + h) * size_t(DV) * DK + size_t(row) * DK + col0;
#pragma unroll
  for (int i = 0; i < CS::R; ++i) {
    float* dst = Sbh + size_t(i) * CS::RS * DK;
    if constexpr (CS::CPT % 4 == 0) {
#pragma unroll
      for (int e = 0; e < CS::CPT; e += 4)
        *reinterpret_cast<float4*>(dst + e) = make_float4(srow[i * CS::CPT + e], srow[i * CS::CPT + e + 1],
                                                          srow[i * CS::CPT + e + 2], srow[i * CS::CPT + e + 3]);
    } else {
#pragma unroll
      for (int e = 0; e < CS::CPT; ++e) dst[e] = srow[i * CS::CPT + e];
    }
  }
}

// the conv-state shift of the commit (kernel 2 of launch_commit) on its own
int launch_commit_conv(const CommitParams& p, int dk, int dv, int in_dtype, hipStream_t stream);

}  // namespace gdn
