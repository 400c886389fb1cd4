// gdn_internal.h -- private declarations of libgdntree (kernels + launchers).
//
// Device helpers used by the prepare / verify / commit kernels, the layout of
// the tree-metadata blob and the launcher entry points that the C ABI
// (gdn_abi.hip) dispatches to.  Everything here targets gfx950 (CDNA4,
// wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdn_tree.h"

namespace gdn {

constexpr int kWave = 64;
constexpr int kSmallMaxT = 128;  // largest tree of the LDS-resident verify kernel
constexpr int kPad = -2;   // parent value of an absent slot
constexpr int kRoot = -1;  // parent value of the root

// ---------------------------------------------------------------------------
// Tree-metadata blob (layout documented in gdn_tree.h).  Each array starts at
// a 16-byte aligned offset.
// ---------------------------------------------------------------------------
struct MetaLayout {
  size_t anc, depth, order, pos, parent, status, nvalid, pdep, ppos, total;
  int W;
};

__host__ __device__ inline size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

__host__ __device__ inline MetaLayout meta_layout(int B, int T) {
  MetaLayout m;
  m.W = (T + 63) / 64;
  size_t bt = size_t(B) * size_t(T);
  m.anc = 0;
  m.depth = align16(m.anc + 8 * bt * m.W);
  m.order = align16(m.depth + 4 * bt);
  m.pos = align16(m.order + 4 * bt);
  m.parent = align16(m.pos + 4 * bt);
  m.status = align16(m.parent + 4 * bt);
  m.nvalid = align16(m.status + 4 * size_t(B));
  m.pdep = align16(m.nvalid + 4 * size_t(B));
  m.ppos = align16(m.pdep + 4 * bt);
  size_t end = m.ppos + 4 * bt;
  m.total = (end + 255) & ~size_t(255);
  return m;
}

struct MetaPtrs {
  uint64_t* anc;
  int32_t* depth;
  int32_t* order;
  int32_t* pos;
  int32_t* parent;
  int32_t* status;
  int32_t* nvalid;
  int32_t* pdep;
  int32_t* ppos;
  int W;
};

__host__ __device__ inline MetaPtrs meta_ptrs(const void* base, int B, int T) {
  MetaLayout l = meta_layout(B, T);
  char* p = (char*)base;
  MetaPtrs m;
  m.anc = (uint64_t*)(p + l.anc);
  m.depth = (int32_t*)(p + l.depth);
  m.order = (int32_t*)(p + l.order);
  m.pos = (int32_t*)(p + l.pos);
  m.parent = (int32_t*)(p + l.parent);
  m.status = (int32_t*)(p + l.status);
  m.nvalid = (int32_t*)(p + l.nvalid);
  m.pdep = (int32_t*)(p + l.pdep);
  m.ppos = (int32_t*)(p + l.ppos);
  m.W = l.W;
  return m;
}

// ---------------------------------------------------------------------------
// Element loads: inputs are fp32 or bf16 (stored as raw 16-bit patterns).
// ---------------------------------------------------------------------------
struct BF16 {
  uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(BF16 x) {
  return __uint_as_float(uint32_t(x.bits) << 16);
}

template <typename TIn>
__device__ __forceinline__ float ld(const TIn* p, size_t i) {
  return to_f32(p[i]);
}

// 4 consecutive elements starting at p (4-element aligned).
__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4(const BF16* p) {
  uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

// SiLU(y) = y * sigmoid(y) with the hardware exp2 and reciprocal (1 ulp each)
// instead of an IEEE-exact division sequence.
__device__ __forceinline__ float silu(float y) {
  return y * __builtin_amdgcn_rcpf(1.0f + __expf(-y));
}

// 1 / sqrt(x) with the hardware reciprocal square root (1 ulp)
__device__ __forceinline__ float rsqrt_hw(float x) { return __builtin_amdgcn_rsqf(x); }

// ---------------------------------------------------------------------------
// Cross-lane sums with DPP (VALU-rate, no LDS round trip).
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;  // lane i <-> 7-i within each 8 lanes
constexpr int kDppRowMirror = 0x140;      // lane i <-> 15-i within each 16 lanes

// Sum over aligned groups of N consecutive lanes (N = 1, 2, ..., 64); every
// lane of a group receives the group's sum.  Up to 16 lanes this is DPP only;
// the steps across 16-lane rows go through ds_bpermute.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16 || N == 32 || N == 64, "group size");
  if constexpr (N >= 2) v += dpp_f<kDppQuadXor1>(v);
  if constexpr (N >= 4) v += dpp_f<kDppQuadXor2>(v);
  if constexpr (N >= 8) v += dpp_f<kDppRowHalfMirror>(v);
  if constexpr (N >= 16) v += dpp_f<kDppRowMirror>(v);
  if constexpr (N >= 32) v += __shfl_xor(v, 16);
  if constexpr (N >= 64) v += __shfl_xor(v, 32);
  return v;
}

// Sum over the whole wave (64 lanes), returned in every lane.
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<16>(v);
  const int b = __float_as_int(v);
  return __int_as_float(__builtin_amdgcn_readlane(b, 0)) + __int_as_float(__builtin_amdgcn_readlane(b, 16)) +
         __int_as_float(__builtin_amdgcn_readlane(b, 32)) + __int_as_float(__builtin_amdgcn_readlane(b, 48));
}

// ---------------------------------------------------------------------------
// MFMA helpers: v_mfma_f32_16x16x32_bf16 operands and a bf16 hi/lo split
// that keeps about 16 bits of the fp32 mantissa (three products per tile).
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

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

// Three bf16 products of a hi/lo split pair into an fp32 accumulator:
// (ah + al)(bh + bl) - al bl, ~1e-5 relative error.
__device__ __forceinline__ f32x4 mfma3(const bf16x8& ah, const bf16x8& al, const bf16x8& bh,
                                       const bf16x8& bl, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, c, 0, 0, 0);
  return c;
}

// ---------------------------------------------------------------------------
// fp16 operands of the S0 readout: power-of-two row scaling.
// ---------------------------------------------------------------------------
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// Largest magnitude over aligned groups of N consecutive lanes (N <= 32).
template <int N>
__device__ __forceinline__ float group_max(float v) {
  static_assert(N >= 1 && N <= 32 && (N & (N - 1)) == 0, "group size");
  if constexpr (N >= 2) v = fmaxf(v, dpp_f<kDppQuadXor1>(v));
  if constexpr (N >= 4) v = fmaxf(v, dpp_f<kDppQuadXor2>(v));
  if constexpr (N >= 8) v = fmaxf(v, dpp_f<kDppRowHalfMirror>(v));
  if constexpr (N >= 16) v = fmaxf(v, dpp_f<kDppRowMirror>(v));
  if constexpr (N >= 32) v = fmaxf(v, __shfl_xor(v, 16));
  return v;
}

// Power-of-two row scale for the fp16 S0 plane: for a row whose largest
// magnitude is m, scale = 2^-floor(log2 m) puts m into [1, 2) and
// inv = 1 / scale; both are exact.  Zero (or subnormal) rows keep scale 1;
// the exponent is clamped so that both factors stay normal floats.
__device__ __forceinline__ void row_scale(float m, float& scale, float& inv) {
  int ex = int((__float_as_uint(m) >> 23) & 0xffu);
  if (ex == 0) {
    scale = inv = 1.0f;
    return;
  }
  ex = ex > 253 ? 253 : ex;
  scale = __uint_as_float(uint32_t(254 - ex) << 23);
  inv = __uint_as_float(uint32_t(ex) << 23);
}

// 4 floats times a scale -> 4 fp16 (round to nearest even), packed in 8 bytes
__device__ __forceinline__ uint2 to_f16x4(float4 x, float sc) {
  const _Float16 h0 = (_Float16)(x.x * sc), h1 = (_Float16)(x.y * sc);
  const _Float16 h2 = (_Float16)(x.z * sc), h3 = (_Float16)(x.w * sc);
  return make_uint2(uint32_t(__builtin_bit_cast(uint16_t, h0)) | (uint32_t(__builtin_bit_cast(uint16_t, h1)) << 16),
                    uint32_t(__builtin_bit_cast(uint16_t, h2)) | (uint32_t(__builtin_bit_cast(uint16_t, h3)) << 16));
}

// ---------------------------------------------------------------------------
// Commit building blocks shared by the commit kernel and the fused step.
// ---------------------------------------------------------------------------
constexpr int kMC = 32;  // path nodes featurised per chunk

// Inputs of one commit feature task: one conv channel over NW consecutive
// path nodes m0 .. m0 + NW - 1 (the width-4 conv reaches back to m0 - 3;
// positions above the root read the conv-state slots).  Every load is
// unconditional (indices clamped) so that nothing waits for it before the
// features are computed; the conv-state / padding choice is made when the
// window is used.
template <typename TIn, int NW>
struct FeatWindow {
  static constexpr int kWin = NW + 3;
  TIn xr[kWin];  // raw inputs of path nodes m0 - 3 .. m0 + NW - 1 (clamped)
  float xc[3];   // conv-state slots 0..2 of the channel
  float4 w;      // conv weights of the channel
  __device__ __forceinline__ void load(const TIn* src, size_t stride, const float* cs, size_t cstride,
                                       const float* wrow, const int* s_path, int m0, int L) {
#pragma unroll
    for (int q = 0; q < kWin; ++q) {
      int mi = m0 - 3 + q;
      mi = mi < 0 ? 0 : (mi < L ? mi : L - 1);
      xr[q] = src[size_t(s_path[mi]) * stride];
    }
#pragma unroll
    for (int sl = 0; sl < 3; ++sl) xc[sl] = cs[size_t(sl) * cstride];
    w = *reinterpret_cast<const float4*>(wrow);
  }
  // input of the window element q (path node m0 - 3 + q); the conv-state
  // slot is picked by selects, not by indexing (keeps xc in registers)
  __device__ __forceinline__ float x(int q, int m0, int L) const {
    const int mi = m0 - 3 + q;
    const float c = mi == -3 ? xc[0] : (mi == -2 ? xc[1] : xc[2]);
    return mi < 0 ? c : (mi < L ? to_f32(xr[q]) : 0.0f);
  }
};


// One rank-1 step of the commit replay, Eq. 7 in the stored orientation,
//   S_r <- alpha S_r + beta (v_r - alpha (S_r . k)) k^T,
// on a thread's pieces of R state rows (CPT consecutive columns each, LPR
// lanes per row; element i CPT + e is column e of piece i).  The rows are
// kept as S = gamma * stored (gamma: running product of alpha), so a step is
// two FMAs per element; kk is the thread's slice of the raw key, inv =
// 1 / ||k|| is folded into the scalars and vr[i] is v of row piece i.  The
// R rows share the key slice, which halves the LDS reads per element for
// R = 2.  Returns the new gamma.
template <int R, int CPT, int LPR>
__device__ __forceinline__ float replay_rows(float (&sr)[R * CPT], const float (&kk)[CPT], const float (&vr)[R],
                                            float al, float be, float inv, float gamma) {
  float uu[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float u[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int e = 0; e < CPT; ++e) u[e & 3] += sr[i * CPT + e] * kk[e];
    uu[i] = (u[0] + u[1]) + (u[2] + u[3]);
  }
#pragma unroll
  for (int i = 0; i < R; ++i) uu[i] = group_sum<LPR>(uu[i]) * inv;  // S_stored . k_hat
  // c = beta (v_r - alpha S_true.k_hat) times 1 / ||k|| (it applies to the
  // raw key).  The decay product is the same in every lane of the workgroup:
  // made visibly uniform so that the rescale below is a scalar branch.
  const float ag = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(al * gamma)));
  // stored frame while ag stays normal: S_true' = ag (stored + c / ag k);
  // a tiny decay (ag < 2^-60, possibly 0) first moves the rows to the true
  // frame, S_true' = ag stored + c k, with no division by ag
  const bool tiny = ag < 0x1p-60f;
  const float mult = tiny ? inv : __builtin_amdgcn_rcpf(ag) * inv;
  if (tiny) {
#pragma unroll
    for (int e = 0; e < R * CPT; ++e) sr[e] *= ag;
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const float c = be * (vr[i] - ag * uu[i]) * mult;
#pragma unroll
    for (int e = 0; e < CPT; ++e) sr[i * CPT + e] += c * kk[e];
  }
  return tiny ? 1.0f : ag;
}

// CPT floats of an LDS row (16-byte pieces when CPT % 4 == 0)
template <int CPT>
__device__ __forceinline__ void ld_slice(const float* src, float (&x)[CPT]) {
  if constexpr (CPT % 4 == 0) {
#pragma unroll
    for (int e = 0; e < CPT; e += 4) {
      const float4 v = *reinterpret_cast<const float4*>(src + e);
      x[e] = v.x;
      x[e + 1] = v.y;
      x[e + 2] = v.z;
      x[e + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < CPT; ++e) x[e] = src[e];
  }
}

// ---------------------------------------------------------------------------
// Launchers (defined in the kernel sources).  All return a gdn_status value.
// ---------------------------------------------------------------------------
int launch_prepare(int B, int T, const int32_t* parent, void* meta, int32_t* tree_status,
                   hipStream_t stream);

struct VerifyArgs {
  int B, T, Hk, Hv, dk, dv, in_dtype;
  float scale;
  const void* meta;
  const void *q, *k, *v, *alpha, *beta;
  const float *conv_w, *conv_state, *S0;
  float* out;
  // fused step (commit of the previous step's accepted path, then verify)
  bool fused = false;
  const void* pmeta = nullptr;
  const int32_t* paccepted = nullptr;
  const void *pq = nullptr, *pk = nullptr, *pv = nullptr, *palpha = nullptr, *pbeta = nullptr;
  float* conv_state_out = nullptr;
  float* S = nullptr;
  int32_t* commit_status = nullptr;
};
int launch_verify(const VerifyArgs& a, hipStream_t stream);
// trees of 129..512 slots: fp16 features into the workspace, then the
// pull-back (the workspace holds large_workspace_bytes(...) bytes)
size_t large_workspace_bytes(int B, int T, int Hk, int Hv, int dk, int dv);
int launch_verify_large(const VerifyArgs& a, void* ws, size_t ws_bytes, hipStream_t stream);
// A device buffer of at least bytes for work on stream, cached per (device,
// stream) and grown on demand (never while the stream is being captured).
void* stream_workspace(size_t bytes, hipStream_t stream, int* rc);
// gdn_tree_verify without any allocation: the workspace of T > 128 is the
// library's static device array
int launch_verify_noalloc(const VerifyArgs& a, hipStream_t stream);
// post-conv features of every position into F[B][T][C] (fp32, canonical
// position order; features_f32_bytes(...) bytes), as the chunked form reads
// them
size_t features_f32_bytes(int B, int T, int Hk, int Hv, int dk, int dv);
int launch_features(const VerifyArgs& a, float* F, hipStream_t stream);
// the paper's chunked form (Eq. 9-13) of the same verification; ws holds
// chunked_workspace_bytes(...) bytes
size_t chunked_workspace_bytes(int B, int T, int Hk, int Hv, int dk, int dv);
int launch_verify_chunked(const VerifyArgs& a, void* ws, size_t ws_bytes, hipStream_t stream);

struct CommitArgs {
  int B, T, Hk, Hv, dk, dv, in_dtype;
  const void* meta;
  const int32_t* accepted;
  const void *q, *k, *v, *alpha, *beta;
  const float* conv_w;
  float* conv_state;                      // in/out, or out when conv_state_in is set
  const float* conv_state_in = nullptr;   // conv state before the commit (not in place)
  float* S;
  int32_t* commit_status;
};
int launch_commit(const CommitArgs& a, hipStream_t stream);

// Records a message for gdn_last_error() and returns code.
int set_error(int code, const char* fmt, ...);

// Raises the dynamic-LDS limit of kernel fn to bytes on the current device,
// once per (kernel, device); thread-safe.  Returns a gdn_status.
int ensure_dynamic_lds(const void* fn, int bytes, const char* who);

}  // namespace gdn
