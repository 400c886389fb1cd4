/*
 * gdn_tree.h -- C ABI of libgdntree: rollback-free verification of a draft
 * token tree through one Gated DeltaNet (GDN) layer on AMD Instinct MI355X
 * (gfx950).
 *
 * Method: "Trees from Marginals", Sec. 3.4.  Every tree node's output is the
 * gated delta rule (Eq. 7) applied along that node's own root-to-node path,
 * starting from the cached per-sequence state S0, followed by the readout of
 * Eq. 8.  Verification only reads the cached state and conv state; the
 * state changes in one place per decode step, the commit, which runs Eq. 7
 * over the accepted node's path once that node has been chosen (Sec. 3.4.2).
 * The tree metadata (depths, a topological order, proper-ancestor bitmasks)
 * is computed once per decode step from the parent pointers and can be
 * shared by every GDN layer of the step (Sec. 3.4.2).
 *
 * Which entry point takes which tree size: gdn_tree_prepare, gdn_tree_commit,
 * gdn_tree_verify, gdn_tree_verify_noalloc, gdn_tree_verify_chunked and
 * gdn_tree_step all accept 1 <= T <= GDN_MAX_T = 512.  Up to 128 slots verify
 * and step run entirely on chip (step as one fused launch); above 128 they
 * go through a feature workspace (see gdn_tree_verify), and the step shifts
 * the conv state, writes the features and then commits each head's state
 * rows inside the verification launch (heads of dk dv < 512: the commit
 * kernels, then the verification).
 *
 * Conventions shared by all entry points
 * --------------------------------------
 *  * All tensor pointers are DEVICE pointers, contiguous row-major, owned by
 *    the caller.  Work is enqueued on the caller's stream and is ordered with
 *    it; nothing synchronises the host except a workspace allocation (trees
 *    above 128 slots, see gdn_tree_verify).  Pointers must be 16-byte
 *    aligned.
 *  * Recurrence orientation: the stored state of (sequence b, value head h) is
 *    S[b][h] in R^{dv x dk} (dk contiguous), the transpose of the paper's
 *    S in R^{dk x dv}; one step is S <- alpha S (I - beta k k^T) + beta v k^T
 *    and the readout is o = scale * S q (Eq. 7-8).
 *  * Short convolution (width 4, depthwise, no bias) and activation: the raw
 *    inputs of node t are the C = 2 Hk dk + Hv dv channels
 *    x_t = [q_t (Hk heads) | k_t (Hk heads) | v_t (Hv heads)].  For a node i
 *    at depth d with path p_0 = root, ..., p_d = i:
 *        y_i[c] = SiLU( sum_{w=0..3} conv_w[c][w] * x_{p_{d-3+w}}[c] ),
 *    where a tap above the root (d-3+w < 0) reads conv_state[b][d+w][c]
 *    (slot 2 = most recent committed token, slot 0 = oldest).  q and k are
 *    then L2-normalised per head: x / sqrt(sum x^2 + 1e-6).  v is not.
 *  * GQA: value head h reads key head floor(h * Hk / Hv); Hv % Hk == 0.
 *  * alpha (decay) and beta (write strength) are per value head, in (0, 1].
 *  * Trees: parent[b][i] = -1 for the root, -2 for an absent (padding) slot,
 *    else the parent's slot index.  Node numbering is arbitrary.
 *
 * Errors: every entry point returns gdn_status.  Problems visible on the
 * host (null pointers, unsupported sizes) return an error before any work is
 * enqueued; gdn_last_error() then describes it.  Problems that only the
 * device can see (an invalid tree, an invalid accepted node) are reported per
 * sequence in the status arrays below and the affected sequence is skipped.
 */
#ifndef GDN_TREE_H
#define GDN_TREE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GDN_OK = 0,
  GDN_EINVAL = -1,       /* null pointer, negative or inconsistent size */
  GDN_EUNSUPPORTED = -2, /* valid but unsupported shape (head dims, T)   */
  GDN_EHIP = -3          /* a HIP launch or attribute call failed        */
} gdn_status;

typedef enum { GDN_F32 = 0, GDN_BF16 = 1 } gdn_dtype;

/* Per-sequence status codes written by prepare (tree) and commit. */
enum {
  GDN_TREE_OK = 0,
  GDN_TREE_NO_ROOT = 1,      /* real nodes but none with parent -1              */
  GDN_TREE_MULTI_ROOT = 2,   /* more than one node with parent -1              */
  GDN_TREE_BAD_PARENT = 3,   /* parent outside {-2,-1,0..T-1}, self, or padding */
  GDN_TREE_CYCLE = 4,        /* a real node whose parent chain misses the root */
  GDN_TREE_BAD_ACCEPTED = 5  /* commit only: accepted outside [-1,T) or padding */
};

/* Problem sizes.  B sequences, T node slots per tree (padded tree size),
 * Hk key heads, Hv value heads, head dims dk and dv.
 * in_dtype is the element type of q, k, v, alpha and beta (GDN_F32 or
 * GDN_BF16); the state, conv weights, conv state and outputs are fp32.
 * scale multiplies the readout; 0 selects 1/sqrt(dk) (Eq. 8).
 * Supported: dk, dv in {16, 32, 64, 128}; 1 <= T <= GDN_MAX_T; B >= 0. */
typedef struct {
  int32_t B, T, Hk, Hv, dk, dv;
  int32_t in_dtype;
  float scale;
} gdn_dims;

#define GDN_MAX_T 512

/* Size in bytes of the tree-metadata blob for B trees of T slots (host only,
 * no device work).  Layout, W = ceil(T/64); each array starts at the next
 * 16-byte aligned offset after the previous one, in this order:
 *   uint64 anc   [B][T][W]  bit (j mod 64) of word j/64 of anc[b][i] is set
 *                           iff slot j is a proper ancestor of slot i
 *                           (Sec. 3.4.2 bitmask, node-index space)
 *   int32  depth [B][T]     edges to the root; -1 for padding
 *   int32  order [B][T]     canonical topological order: real nodes sorted
 *                           by (depth, index), then padding by index
 *   int32  pos   [B][T]     inverse permutation of order
 *   int32  parent[B][T]     copy of the input parent array
 *   int32  status[B]        GDN_TREE_* code of each tree
 *   int32  nvalid[B]        number of real (non-padding) nodes
 *   int32  pdep  [B][T]     depth of the node at canonical position p
 *                           (depth[order[p]]), -1 for padding
 *   int32  ppos  [B][T]     canonical position of the parent of the node at
 *                           position p (pos[parent[order[p]]]), -1 for the
 *                           root and padding
 * The blob is padded to a multiple of 256 bytes.  A tree with a non-zero
 * status gets depth/pdep/ppos -1, identity order/pos, empty ancestor sets and
 * nvalid 0.  Returns 0 for B <= 0 or T <= 0. */
size_t gdn_tree_meta_bytes(int32_t B, int32_t T);

/* Tree preprocessing (Sec. 3.4.1 topological order and ancestor relation,
 * Sec. 3.4.2 metadata computed once per decode step).
 *   parent      int32 [B][T]   device, read-only
 *   meta        device buffer of gdn_tree_meta_bytes(B, T) bytes, written
 *   tree_status int32 [B]      device, written (may be NULL)
 * Reads only dims->B and dims->T.  One workgroup per tree. */
int gdn_tree_prepare(const gdn_dims* dims, const int32_t* parent, void* meta,
                     int32_t* tree_status, hipStream_t stream);

/* Read-only tree verification (Sec. 3.4: Eq. 7-8 per node along its path).
 * Up to 128 slots everything stays on chip and nothing is allocated; above
 * 128 the post-conv features go through a device workspace of
 * B T (2 C + 4 Hv) bytes (fp16 features, fp32 scales of the value rows;
 * C = 2 Hk dk + Hv dv, the first part rounded up to 256 bytes) that the
 * library allocates on the first call that needs it and keeps per
 * (device, stream) until the process ends (a call under stream capture that
 * would have to grow it returns GDN_EUNSUPPORTED).
 *   meta        written by gdn_tree_prepare for the same B, T
 *   q, k        in_dtype [B][T][Hk][dk]   raw (pre-conv) queries / keys
 *   v           in_dtype [B][T][Hv][dv]   raw values
 *   alpha, beta in_dtype [B][T][Hv]
 *   conv_w      fp32 [C][4]               C = 2 Hk dk + Hv dv
 *   conv_state  fp32 [B][3][C]            read-only
 *   S0          fp32 [B][Hv][dv][dk]      read-only cached state
 *   out         fp32 [B][T][Hv][dv]       written: o_i = scale * S_i q_i
 * Rows of padding slots and every row of a sequence whose tree status is
 * non-zero are written as zeros.  conv_state and S0 are never written. */
int gdn_tree_verify(const gdn_dims* dims, const void* meta, const void* q, const void* k,
                    const void* v, const void* alpha, const void* beta, const float* conv_w,
                    const float* conv_state, const float* S0, float* out, hipStream_t stream);

/* gdn_tree_verify for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops that forbid hipMalloc).  Same
 * arguments, layouts, outputs and errors as gdn_tree_verify, whose kernels
 * it runs; it calls no allocating routine.  Trees of more than 128 slots
 * need the feature workspace of gdn_tree_verify, B T (2 C + 4 Hv) bytes:
 * here it is a static device array of GDN_NOALLOC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends, and
 * larger problems return GDN_EUNSUPPORTED before any device work.  All
 * calls on one device share that array: calls that overlap in time on one
 * device (different streams, or host threads) race and must be serialized
 * by the caller. */
#define GDN_NOALLOC_SCRATCH_BYTES (64u << 20)
int gdn_tree_verify_noalloc(const gdn_dims* dims, const void* meta, const void* q, const void* k,
                            const void* v, const void* alpha, const void* beta,
                            const float* conv_w, const float* conv_state, const float* S0,
                            float* out, hipStream_t stream);

/* The same verification in the paper's chunked form (Sec. 3.4.1-3.4.2,
 * Eq. 9-13): per (sequence, value head) the interaction matrices X (strict
 * ancestors: decayed key-key products scaled by beta) and Y (ancestors and
 * self: decayed query-key products) are built from Gram products, (I + X) U =
 * beta (V - a K S0^T) is solved by forward substitution over sub-blocks of 32
 * positions (each diagonal block inverted by repeated squaring), and O =
 * scale (a Q S0^T + Y U); the Gram, solve and readout products on bf16
 * MFMA as hi/lo three-product splits (about 16 significant bits), the
 * diagonal-block inverses on fp32 MFMA, features in fp32.  Arguments,
 * layouts, outputs and errors are those of gdn_tree_verify (any supported
 * dk, dv and T).  Needs a workspace of B T (C + Hv dv) 4 bytes, cached per
 * (device, stream) like gdn_tree_verify's above 128 slots.  Its cost does not
 * grow with the depth of the tree, while gdn_tree_verify's grows with the sum
 * of the path lengths. */
int gdn_tree_verify_chunked(const gdn_dims* dims, const void* meta, const void* q, const void* k,
                            const void* v, const void* alpha, const void* beta,
                            const float* conv_w, const float* conv_state, const float* S0,
                            float* out, hipStream_t stream);

/* Commit of the accepted node (Sec. 3.4.2): Eq. 7 is run over the path
 * root..accepted, starting from S, and the result replaces S.
 *   accepted      int32 [B]  accepted slot per sequence, -1 = commit nothing
 *   q, k, v, alpha, beta, conv_w: as for verify (same step's tensors)
 *   conv_state    fp32 [B][3][C]   in/out: replaced by the last 3 raw inputs
 *                 of (old slots 0..2 followed by the path's raw inputs)
 *   S             fp32 [B][Hv][dv][dk]  in/out: state after the path
 *   commit_status int32 [B] (may be NULL): the tree status if non-zero, else
 *                 GDN_TREE_BAD_ACCEPTED for an accepted slot outside [-1, T)
 *                 or naming padding, else 0.
 * Sequences with accepted == -1 or a non-zero commit status are untouched.
 * Enqueues two kernels (state replay, then conv-state shift). */
int gdn_tree_commit(const gdn_dims* dims, const void* meta, const int32_t* accepted,
                    const void* q, const void* k, const void* v, const void* alpha,
                    const void* beta, const float* conv_w, float* conv_state, float* S,
                    int32_t* commit_status, hipStream_t stream);

/* Fused decode step: the commit of the previous step's accepted node
 * (Sec. 3.4.2) followed by the verification of the current tree (Sec. 3.4,
 * Eq. 7-8) against the state it produces, in one launch up to 128 slots
 * (above: conv-state shift, features, then one launch that commits and
 * verifies each head).  Results equal gdn_tree_commit(previous step)
 * followed by gdn_tree_verify(current step) with the committed S and conv
 * state; the committed state is formed in registers and verified against
 * without being read back.
 *   prev_meta      meta of the previous step's tree (same B, T)
 *   prev_accepted  int32 [B]: accepted slot of the previous tree, -1 = none
 *   prev_q, prev_k, prev_v, prev_alpha, prev_beta: the previous step's raw
 *                  inputs (shapes and in_dtype as for verify)
 *   commit_status  int32 [B] (may be NULL): as for gdn_tree_commit
 *   meta, q, k, v, alpha, beta: the current step's tree and raw inputs
 *   conv_w         fp32 [C][4] (one layer: shared by both steps)
 *   conv_state     fp32 [B][3][C]  read-only: conv state before the commit
 *   conv_state_out fp32 [B][3][C]  written: conv state after the commit; must
 *                  not overlap conv_state (checked, GDN_EINVAL)
 *   S              fp32 [B][Hv][dv][dk]  in/out: the state before the commit
 *                  on entry, after it on return
 *   out            fp32 [B][T][Hv][dv]  written: outputs of the current tree
 * A sequence with nothing to commit (prev_accepted -1 or a non-zero commit
 * status) keeps S and gets conv_state_out = conv_state; a sequence whose
 * current tree is invalid still commits and gets zero outputs.  Each
 * (sequence, value head, dv slice) of S is read and written by one
 * workgroup only, so the in-place update is race-free; S must not alias
 * any other argument. */
int gdn_tree_step(const gdn_dims* dims, const void* prev_meta, const int32_t* prev_accepted,
                  const void* prev_q, const void* prev_k, const void* prev_v,
                  const void* prev_alpha, const void* prev_beta, int32_t* commit_status,
                  const void* meta, const void* q, const void* k, const void* v,
                  const void* alpha, const void* beta, const float* conv_w,
                  const float* conv_state, float* conv_state_out, float* S, float* out,
                  hipStream_t stream);

/* Message describing the last non-OK return on the calling thread. */
const char* gdn_last_error(void);

/* Library version string. */
const char* gdn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GDN_TREE_H */
