// gdn_prepare.hip -- tree preprocessing kernel (paper Sec. 3.4.1 ancestor
// relation and topological order; Sec. 3.4.2 metadata computed once per
// decode step from parent pointers: proper-ancestor sets as bitmasks packed
// in 64-bit words).
//
// One workgroup per tree, one thread per slot (T <= kPrepMaxT).  Depth and
// ancestor sets come from pointer jumping: after r rounds every slot knows
// its ancestors at distances 1..2^r and the ancestor at distance 2^r, so
// ceil(log2 T) rounds reach the root from any connected slot; a slot that
// still has an ancestor to jump to afterwards lies on a cycle.  The
// canonical order ranks slots by (depth, index) with padding last.
#include "gdn_internal.h"

namespace gdn {

constexpr int kPrepMaxT = 512;

// KW = ceil(T / 64) ancestor words per node (1, 2, 4 or 8; trees of up to
// 64 KW slots), a compile-time count so that the rows move as whole vectors
template <int KW>
__global__ __launch_bounds__(kPrepMaxT) void prepare_kernel(const int32_t* __restrict__ parent,
                                                            MetaPtrs m, int32_t* tree_status,
                                                            int T) {
  constexpr int kMaxT = 64 * KW;
  __shared__ int s_par[kMaxT];
  __shared__ int s_nxt[kMaxT];
  __shared__ __align__(16) int s_dep[kMaxT];
  __shared__ __align__(16) uint64_t s_anc[kMaxT * KW];
  __shared__ int s_bad, s_roots, s_real, s_cycle;
  __shared__ int s_more[2];  // a jump of this round is not at a root yet (rounds alternate)

  const int b = blockIdx.x;
  const int i = threadIdx.x;
  const int W = m.W;  // the blob's word count, ceil(T / 64) <= KW
  const bool slot = i < T;

  if (i == 0) {
    s_bad = 0;
    s_roots = 0;
    s_real = 0;
    s_cycle = 0;
    s_more[0] = 0;
  }
  int p = slot ? parent[size_t(b) * T + i] : kPad;
  if (slot) s_par[i] = p;
  __syncthreads();

  // validity of the parent value itself
  const bool real = slot && p != kPad;
  if (real) {
    atomicAdd(&s_real, 1);
    if (p == kRoot) {
      atomicAdd(&s_roots, 1);
    } else if (p < 0 || p >= T || p == i || s_par[p] == kPad) {
      s_bad = 1;
    }
  }
  __syncthreads();
  int status = GDN_TREE_OK;
  if (s_bad)
    status = GDN_TREE_BAD_PARENT;
  else if (s_real > 0 && s_roots == 0)
    status = GDN_TREE_NO_ROOT;
  else if (s_roots > 1)
    status = GDN_TREE_MULTI_ROOT;

  // pointer jumping (only meaningful for a tree with valid parent values)
  uint64_t anc[KW];
#pragma unroll
  for (int w = 0; w < KW; ++w) anc[w] = 0;
  int nxt = (real && p >= 0 && status == GDN_TREE_OK) ? p : -1;
  int dep = (nxt >= 0) ? 1 : 0;
#pragma unroll
  for (int w = 0; w < KW; ++w)
    if (nxt >= 0 && w == (nxt >> 6)) anc[w] |= 1ull << (nxt & 63);
  for (int span = 1, r = 0; span < T; span <<= 1, r ^= 1) {
    if (slot) {
      s_nxt[i] = nxt;
      s_dep[i] = dep;
#pragma unroll
      for (int w = 0; w < KW; ++w) s_anc[i * KW + w] = anc[w];
    }
    __syncthreads();
    // the other round's flag was last read before the barrier above
    if (i == 0) s_more[r ^ 1] = 0;
    if (nxt >= 0) {
      int j = nxt;
      dep += s_dep[j];
#pragma unroll
      for (int w = 0; w < KW; ++w) anc[w] |= s_anc[j * KW + w];
      nxt = s_nxt[j];
    }
    if (nxt >= 0) s_more[r] = 1;
    __syncthreads();
    // every jump reached a root: the remaining rounds would change nothing
    // (a cycle never gets there and keeps jumping until span >= T)
    if (!s_more[r]) break;
  }
  if (status == GDN_TREE_OK && real && nxt >= 0) s_cycle = 1;
  __syncthreads();
  if (status == GDN_TREE_OK && s_cycle) status = GDN_TREE_CYCLE;

  const int32_t base = b * T;
  if (status != GDN_TREE_OK) {
    if (slot) {
      m.depth[base + i] = -1;
      m.order[base + i] = i;
      m.pos[base + i] = i;
      m.parent[base + i] = p;
      m.pdep[base + i] = -1;
      m.ppos[base + i] = -1;
      for (int w = 0; w < W; ++w) m.anc[(size_t(base) + i) * W + w] = 0;
    }
    if (i == 0) {
      m.status[b] = status;
      m.nvalid[b] = 0;
      if (tree_status) tree_status[b] = status;
    }
    return;
  }

  // canonical order: rank by (depth, index), padding after all depths, as
  // the count of smaller keys depth * 1024 + index (distinct; T <= 512);
  // the keys are read four at a time (slots T .. up to a multiple of 4 hold
  // a key above every real one, so they never count)
  const int T4 = (T + 3) & ~3;
  if (i < T4) s_dep[i] = slot ? ((real ? dep : T + 1) << 10) | i : 0x7fffffff;
  __syncthreads();
  if (slot) {
    const int key = s_dep[i];
    int rank = 0;
#pragma unroll 4
    for (int j = 0; j < T4; j += 4) {
      const int4 k4 = *reinterpret_cast<const int4*>(s_dep + j);
      rank += (k4.x < key) + (k4.y < key) + (k4.z < key) + (k4.w < key);
    }
    m.order[base + rank] = i;
    m.pos[base + i] = rank;
    m.depth[base + i] = real ? dep : -1;
    m.parent[base + i] = p;
#pragma unroll
    for (int w = 0; w < KW; ++w)
      if (w < W) m.anc[(size_t(base) + i) * W + w] = real ? anc[w] : 0;
    s_nxt[i] = rank;  // position of slot i (s_nxt is free after the jumps)
  }
  __syncthreads();
  if (slot) {  // per-position copies: depth and parent position
    const int rank = s_nxt[i];
    m.pdep[base + rank] = real ? dep : -1;
    m.ppos[base + rank] = (real && p >= 0) ? s_nxt[p] : -1;
  }
  if (i == 0) {
    m.status[b] = GDN_TREE_OK;
    m.nvalid[b] = s_real;
    if (tree_status) tree_status[b] = GDN_TREE_OK;
  }
}

int launch_prepare(int B, int T, const int32_t* parent, void* meta, int32_t* tree_status,
                   hipStream_t stream) {
  if (T > kPrepMaxT) return set_error(GDN_EUNSUPPORTED, "prepare: T=%d exceeds %d", T, kPrepMaxT);
  MetaPtrs m = meta_ptrs(meta, B, T);
  int threads = ((T + kWave - 1) / kWave) * kWave;
  if (m.W <= 1)
    hipLaunchKernelGGL(prepare_kernel<1>, dim3(B), dim3(threads), 0, stream, parent, m, tree_status, T);
  else if (m.W <= 2)
    hipLaunchKernelGGL(prepare_kernel<2>, dim3(B), dim3(threads), 0, stream, parent, m, tree_status, T);
  else if (m.W <= 4)
    hipLaunchKernelGGL(prepare_kernel<4>, dim3(B), dim3(threads), 0, stream, parent, m, tree_status, T);
  else
    hipLaunchKernelGGL(prepare_kernel<8>, dim3(B), dim3(threads), 0, stream, parent, m, tree_status, T);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(GDN_EHIP, "prepare launch: %s", hipGetErrorString(e));
  return GDN_OK;
}

}  // namespace gdn
