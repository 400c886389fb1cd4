/*
 * gdn_oracle.c -- CPU oracle for rollback-free GDN draft-tree verification.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or helper with the HIP library: it is a plain, slow and
 * obviously-correct restatement of the method's definitions, in float64.
 *
 * What it computes (paper: "Trees from Marginals", Sec. 3.4):
 *
 *  - Tree metadata (Sec. 3.4.1 ancestor relation / topological order;
 *    Sec. 3.4.2 parent pointers -> proper-ancestor sets as bitmasks packed in
 *    64-bit words): depth, a canonical topological order, proper-ancestor
 *    bitmasks, and a per-sequence validity status.
 *
 *  - The width-4 causal short convolution + SiLU that precede the recurrence
 *    in a gated-delta-net block, evaluated along each node's own root-to-node
 *    path (positions above the root come from the cached conv state), and the
 *    per-head L2 normalisation of q and k.  The paper does not spell this out;
 *    the reading used is the standard GDN block order (raw q,k,v -> depthwise
 *    causal conv -> SiLU -> L2-norm of q,k -> recurrence).
 *
 *  - Verify: for every node i, the gated delta rule (Eq. 7)
 *        S_t = alpha_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T
 *    applied along the path root..i starting from the cached S0, followed by
 *    the readout (Eq. 8)  o_i = q_i^T S_i * scale  (scale = 1/sqrt(dk) by
 *    default).  S0 is never written (Sec. 3.4: read-only verification).
 *    The computation is done in the paper's orientation S in R^{dk x dv};
 *    the stored state is laid out [Hv][dv][dk] (Sec. 3.4.2), i.e. the stored
 *    matrix is the transpose, and is transposed on load and store.
 *
 *  - Commit (Sec. 3.4.2, last paragraph): replay Eq. 7 along the accepted
 *    node's path and write the resulting state; shift the conv state by the
 *    accepted path's raw inputs.
 *
 * Parity pins: see the oracle tests (closed forms, the chunked tree form of
 * Eq. 9-11 and the end-of-path state of Eq. 12, library convolution, special
 * cases, node locality, relabelling invariance).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_PAD (-2)
#define ORC_ROOT (-1)

/* per-sequence tree status codes */
#define ORC_OK 0
#define ORC_NO_ROOT 1
#define ORC_MULTI_ROOT 2
#define ORC_BAD_PARENT 3
#define ORC_CYCLE 4
#define ORC_BAD_ACCEPTED 5

typedef struct {
  int B, T, Hk, Hv, dk, dv;
  double scale; /* readout scale; <= 0 means 1/sqrt(dk) */
} orc_dims;

static int orc_C(const orc_dims* d) { return 2 * d->Hk * d->dk + d->Hv * d->dv; }

/* ------------------------------------------------------------------------ */
/* tree                                                                      */
/* ------------------------------------------------------------------------ */

/* Status of one parent array.  Checks, in this order:
 *   a parent value outside {-2, -1, 0..T-1}, a self-parent, or a parent that
 *   is itself padding                               -> ORC_BAD_PARENT
 *   no root among the real nodes                    -> ORC_NO_ROOT
 *   more than one root                              -> ORC_MULTI_ROOT
 *   a real node whose parent chain never reaches the root  -> ORC_CYCLE
 * A sequence made only of padding is valid (an empty tree). */
int oracle_tree_status(int T, const int32_t* par) {
  int roots = 0, real = 0;
  for (int i = 0; i < T; ++i) {
    int p = par[i];
    if (p == ORC_PAD) continue;
    if (p == ORC_ROOT) continue;
    if (p < 0 || p >= T || p == i) return ORC_BAD_PARENT;
    if (par[p] == ORC_PAD) return ORC_BAD_PARENT;
  }
  for (int i = 0; i < T; ++i) {
    if (par[i] == ORC_PAD) continue;
    real++;
    if (par[i] == ORC_ROOT) roots++;
  }
  if (real == 0) return ORC_OK;
  if (roots == 0) return ORC_NO_ROOT;
  if (roots > 1) return ORC_MULTI_ROOT;
  for (int i = 0; i < T; ++i) {
    if (par[i] == ORC_PAD) continue;
    int t = i, steps = 0;
    while (par[t] != ORC_ROOT && steps <= T) {
      t = par[t];
      steps++;
    }
    if (par[t] != ORC_ROOT) return ORC_CYCLE;
  }
  return ORC_OK;
}

/* Number of edges from node i up to the root (valid tree assumed). */
static int orc_depth(const int32_t* par, int i) {
  int d = 0;
  while (par[i] != ORC_ROOT) {
    i = par[i];
    d++;
  }
  return d;
}

/* path[0] = root, ..., path[d] = i; returns d. */
static int orc_path(const int32_t* par, int i, int* path) {
  int d = orc_depth(par, i);
  for (int m = d; m >= 0; --m) {
    path[m] = i;
    i = par[i];
  }
  return d;
}

/* Tree metadata for B sequences of T slots each.
 *   depth[b][i] : edges to the root; -1 for padding
 *   order[b][p] : canonical topological order = real nodes stably sorted by
 *                 (depth, index), then padding nodes by index
 *   anc[b][i][w]: bit (j mod 64) of word j/64 set iff j is a proper ancestor
 *                 of i (Sec. 3.4.2)
 *   nvalid[b]   : number of real nodes
 *   status[b]   : oracle_tree_status
 * A sequence with a non-zero status gets depth -1, identity order, empty
 * ancestor sets and nvalid 0. */
void oracle_prepare(int B, int T, const int32_t* parent, int32_t* depth, int32_t* order,
                    uint64_t* anc, int32_t* nvalid, int32_t* status) {
  int W = (T + 63) / 64;
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    int32_t* dep = depth + (size_t)b * T;
    int32_t* ord = order + (size_t)b * T;
    uint64_t* an = anc + (size_t)b * T * W;
    int st = oracle_tree_status(T, par);
    status[b] = st;
    memset(an, 0, sizeof(uint64_t) * (size_t)T * W);
    if (st != ORC_OK) {
      for (int i = 0; i < T; ++i) {
        dep[i] = -1;
        ord[i] = i;
      }
      nvalid[b] = 0;
      continue;
    }
    int nv = 0;
    for (int i = 0; i < T; ++i) {
      if (par[i] == ORC_PAD) {
        dep[i] = -1;
        continue;
      }
      nv++;
      dep[i] = orc_depth(par, i);
      for (int t = par[i]; t != ORC_ROOT; t = par[t]) an[(size_t)i * W + t / 64] |= 1ull << (t % 64);
    }
    nvalid[b] = nv;
    /* stable insertion sort of the indices by key (depth, index), padding last */
    for (int i = 0; i < T; ++i) ord[i] = i;
    for (int a = 1; a < T; ++a) {
      int x = ord[a];
      long kx = dep[x] < 0 ? (long)T + 1 : dep[x];
      int c = a - 1;
      while (c >= 0) {
        int y = ord[c];
        long ky = dep[y] < 0 ? (long)T + 1 : dep[y];
        if (ky > kx || (ky == kx && y > x)) {
          ord[c + 1] = ord[c];
          c--;
        } else {
          break;
        }
      }
      ord[c + 1] = x;
    }
  }
}

/* ------------------------------------------------------------------------ */
/* short convolution along the path                                          */
/* ------------------------------------------------------------------------ */

static double orc_silu(double y) { return y / (1.0 + exp(-y)); }

/* Raw (pre-conv) channel c of node t: channels are [q heads | k heads | v heads]. */
static double orc_raw(const orc_dims* d, int b, int t, int c, const double* q, const double* k,
                      const double* v) {
  int nq = d->Hk * d->dk;
  if (c < nq) return q[((size_t)b * d->T + t) * nq + c];
  c -= nq;
  if (c < nq) return k[((size_t)b * d->T + t) * nq + c];
  c -= nq;
  return v[((size_t)b * d->T + t) * (size_t)(d->Hv * d->dv) + c];
}

/* Post-conv features of node i of sequence b (valid tree):
 *   y[c] = SiLU( sum_{w=0..3} conv_w[c][w] * x_w[c] )
 * where tap w=3 is node i itself, w=2 its parent, w=1 its grandparent,
 * w=0 its great-grandparent; a tap above the root reads the cached conv state
 * (slot 2 = most recent committed token, slot 0 = oldest).
 * Then q and k are L2-normalised per key head: x / sqrt(sum x^2 + 1e-6).
 * feat has C entries. */
static void orc_features(const orc_dims* d, int b, const int32_t* par, int i, const double* q,
                         const double* k, const double* v, const double* conv_w,
                         const double* conv_state, double* feat, int* path) {
  int C = orc_C(d);
  int dep = orc_path(par, i, path);
  for (int c = 0; c < C; ++c) {
    double y = 0.0;
    for (int w = 0; w < 4; ++w) {
      int m = dep - 3 + w; /* depth of the tap's node on the path */
      double x;
      if (m >= 0)
        x = orc_raw(d, b, path[m], c, q, k, v);
      else
        x = conv_state[((size_t)b * 3 + (3 + m)) * C + c];
      y += conv_w[(size_t)c * 4 + w] * x;
    }
    feat[c] = orc_silu(y);
  }
  for (int part = 0; part < 2; ++part) {
    for (int g = 0; g < d->Hk; ++g) {
      double* x = feat + (size_t)part * d->Hk * d->dk + (size_t)g * d->dk;
      double ss = 0.0;
      for (int c = 0; c < d->dk; ++c) ss += x[c] * x[c];
      double inv = 1.0 / sqrt(ss + 1e-6);
      for (int c = 0; c < d->dk; ++c) x[c] *= inv;
    }
  }
}

/* Exported for tests: post-conv features of every real node, [B][T][C];
 * rows of padding nodes and of invalid sequences are zero. */
void oracle_features(const orc_dims* d, const int32_t* parent, const double* q, const double* k,
                     const double* v, const double* conv_w, const double* conv_state,
                     double* feat) {
  int C = orc_C(d);
  int T = d->T;
  int* path = (int*)malloc(sizeof(int) * (T + 1));
  for (int b = 0; b < d->B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    int st = oracle_tree_status(T, par);
    for (int i = 0; i < T; ++i) {
      double* f = feat + ((size_t)b * T + i) * C;
      if (st != ORC_OK || par[i] == ORC_PAD) {
        memset(f, 0, sizeof(double) * C);
        continue;
      }
      orc_features(d, b, par, i, q, k, v, conv_w, conv_state, f, path);
    }
  }
  free(path);
}

/* ------------------------------------------------------------------------ */
/* gated delta rule, paper orientation S in R^{dk x dv}                      */
/* ------------------------------------------------------------------------ */

/* One step of Eq. 7 on S (dk x dv, row-major):
 *   S <- alpha (I - beta k k^T) S + beta k v^T                              */
static void orc_eq7(int dk, int dv, double* S, const double* kk, const double* vv, double alpha,
                    double beta, double* w) {
  /* w = k^T S  (row vector of length dv) */
  for (int j = 0; j < dv; ++j) w[j] = 0.0;
  for (int c = 0; c < dk; ++c)
    for (int j = 0; j < dv; ++j) w[j] += kk[c] * S[(size_t)c * dv + j];
  for (int c = 0; c < dk; ++c)
    for (int j = 0; j < dv; ++j)
      S[(size_t)c * dv + j] =
          alpha * (S[(size_t)c * dv + j] - beta * kk[c] * w[j]) + beta * kk[c] * vv[j];
}

/* Load S (dk x dv) from the stored [dv][dk] state of (b, h). */
static void orc_load_state(const orc_dims* d, const double* S0, int b, int h, double* S) {
  const double* src = S0 + ((size_t)b * d->Hv + h) * (size_t)d->dv * d->dk;
  for (int c = 0; c < d->dk; ++c)
    for (int j = 0; j < d->dv; ++j) S[(size_t)c * d->dv + j] = src[(size_t)j * d->dk + c];
}

/* Verify (read-only): out[b][i][h][j] = (q_i^T S_i)[j] * scale, with S_i the
 * result of Eq. 7 along the path root..i of node i, starting from S0[b][h].
 * node_mask [B][T] (may be NULL = all) selects which outputs to compute;
 * unselected, padding and invalid-sequence outputs are written as 0. */
void oracle_verify(const orc_dims* d, const int32_t* parent, const double* q, const double* k,
                   const double* v, const double* alpha, const double* beta,
                   const double* conv_w, const double* conv_state, const double* S0,
                   const uint8_t* node_mask, double* out) {
  int B = d->B, T = d->T, Hk = d->Hk, Hv = d->Hv, dk = d->dk, dv = d->dv;
  int C = orc_C(d);
  double scale = d->scale > 0 ? d->scale : 1.0 / sqrt((double)dk);
  size_t nunits = (size_t)B * T;
  memset(out, 0, sizeof(double) * nunits * Hv * dv);
#pragma omp parallel
  {
    double* S = (double*)malloc(sizeof(double) * (size_t)dk * dv);
    double* w = (double*)malloc(sizeof(double) * dv);
    int* path = (int*)malloc(sizeof(int) * (T + 1));
    double* feat = (double*)malloc(sizeof(double) * (size_t)(T + 1) * C);
#pragma omp for schedule(dynamic, 1)
    for (long u = 0; u < (long)nunits; ++u) {
      int b = (int)(u / T), i = (int)(u % T);
      const int32_t* par = parent + (size_t)b * T;
      if (node_mask && !node_mask[u]) continue;
      if (par[i] == ORC_PAD || oracle_tree_status(T, par) != ORC_OK) continue;
      int dep = orc_path(par, i, path);
      int pathcopy[dep + 1];
      memcpy(pathcopy, path, sizeof(int) * (dep + 1));
      /* features of every node on the path (feat row m <-> path node m) */
      for (int m = 0; m <= dep; ++m)
        orc_features(d, b, par, pathcopy[m], q, k, v, conv_w, conv_state, feat + (size_t)m * C,
                     path);
      for (int h = 0; h < Hv; ++h) {
        int g = h * Hk / Hv; /* key head shared by this value head */
        orc_load_state(d, S0, b, h, S);
        for (int m = 0; m <= dep; ++m) {
          const double* f = feat + (size_t)m * C;
          const double* kk = f + (size_t)Hk * dk + (size_t)g * dk;
          const double* vv = f + (size_t)2 * Hk * dk + (size_t)h * dv;
          size_t ab = ((size_t)b * T + pathcopy[m]) * Hv + h;
          orc_eq7(dk, dv, S, kk, vv, alpha[ab], beta[ab], w);
        }
        const double* qq = feat + (size_t)dep * C + (size_t)g * dk;
        double* o = out + (((size_t)b * T + i) * Hv + h) * dv;
        for (int j = 0; j < dv; ++j) {
          double acc = 0.0;
          for (int c = 0; c < dk; ++c) acc += qq[c] * S[(size_t)c * dv + j];
          o[j] = acc * scale; /* Eq. 8 */
        }
      }
    }
    free(S);
    free(w);
    free(path);
    free(feat);
  }
}

/* Commit: for each sequence with accepted[b] != -1, replay Eq. 7 along the
 * path root..accepted[b] from S[b][h] (every value head) and write the result
 * back into S; then replace conv_state[b] by the last 3 raw inputs of
 * (old conv_state slots 0,1,2 followed by the path's raw inputs, root first).
 * status[b]: the tree status if non-zero; ORC_BAD_ACCEPTED if accepted[b] is
 * outside [-1, T) or names a padding node; 0 otherwise.  Sequences with a
 * non-zero status or accepted[b] == -1 are left untouched. */
void oracle_commit(const orc_dims* d, const int32_t* parent, const int32_t* accepted,
                   const double* q, const double* k, const double* v, const double* alpha,
                   const double* beta, const double* conv_w, double* conv_state, double* S,
                   int32_t* status) {
  int B = d->B, T = d->T, Hk = d->Hk, Hv = d->Hv, dk = d->dk, dv = d->dv;
  int C = orc_C(d);
  int* apath = (int*)malloc(sizeof(int) * (size_t)B * (T + 1));
  int* adep = (int*)malloc(sizeof(int) * B);
  double* feat = (double*)malloc(sizeof(double) * (size_t)B * (T + 1) * C);
  for (int b = 0; b < B; ++b) {
    const int32_t* par = parent + (size_t)b * T;
    int st = oracle_tree_status(T, par);
    int a = accepted[b];
    adep[b] = -1;
    if (st != ORC_OK) {
      status[b] = st;
      continue;
    }
    if (a == -1) {
      status[b] = ORC_OK;
      continue;
    }
    if (a < -1 || a >= T || par[a] == ORC_PAD) {
      status[b] = ORC_BAD_ACCEPTED;
      continue;
    }
    status[b] = ORC_OK;
    int* path = apath + (size_t)b * (T + 1);
    int dep = orc_path(par, a, path);
    adep[b] = dep;
    int tmp[T + 1];
    for (int m = 0; m <= dep; ++m)
      orc_features(d, b, par, path[m], q, k, v, conv_w, conv_state,
                   feat + ((size_t)b * (T + 1) + m) * C, tmp);
  }
#pragma omp parallel
  {
    double* Sp = (double*)malloc(sizeof(double) * (size_t)dk * dv);
    double* w = (double*)malloc(sizeof(double) * dv);
#pragma omp for schedule(dynamic, 1)
    for (long u = 0; u < (long)B * Hv; ++u) {
      int b = (int)(u / Hv), h = (int)(u % Hv);
      int dep = adep[b];
      if (dep < 0) continue;
      int g = h * Hk / Hv;
      const int* path = apath + (size_t)b * (T + 1);
      orc_load_state(d, S, b, h, Sp);
      for (int m = 0; m <= dep; ++m) {
        const double* f = feat + ((size_t)b * (T + 1) + m) * C;
        size_t ab = ((size_t)b * T + path[m]) * Hv + h;
        orc_eq7(dk, dv, Sp, f + (size_t)Hk * dk + (size_t)g * dk, f + (size_t)2 * Hk * dk + (size_t)h * dv,
                alpha[ab], beta[ab], w);
      }
      double* dst = S + ((size_t)b * Hv + h) * (size_t)dv * dk;
      for (int c = 0; c < dk; ++c)
        for (int j = 0; j < dv; ++j) dst[(size_t)j * dk + c] = Sp[(size_t)c * dv + j];
    }
    free(Sp);
    free(w);
  }
  /* conv state: last 3 entries of (old slots 0..2 | path raw inputs) */
  for (int b = 0; b < B; ++b) {
    int dep = adep[b];
    if (dep < 0) continue;
    int L = dep + 1;
    const int* path = apath + (size_t)b * (T + 1);
    double* cs = conv_state + (size_t)b * 3 * C;
    for (int c = 0; c < C; ++c) {
      double seq[3 + T + 1];
      for (int s = 0; s < 3; ++s) seq[s] = cs[(size_t)s * C + c];
      for (int m = 0; m < L; ++m) seq[3 + m] = orc_raw(d, b, path[m], c, q, k, v);
      for (int s = 0; s < 3; ++s) cs[(size_t)s * C + c] = seq[L + s];
    }
  }
  free(apath);
  free(adep);
  free(feat);
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads used by the parallel loops from now on (n >= 1); a timing knob of
 * the benchmark's CPU baseline, no effect on any result. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
