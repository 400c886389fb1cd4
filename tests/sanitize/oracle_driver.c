/* Sanitizer driver for the CPU oracle (test infrastructure): runs prepare,
 * features, verify (with and without a node mask) and commit on random
 * valid, padded and invalid trees of 1..300 slots, with head dims 4..32,
 * and checks the tree statuses and that every result is finite.  Built with
 * -fsanitize=address,undefined by tests/test_sanitize_cpu.py; any sanitizer
 * report aborts with a non-zero exit status. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef struct {
  int B, T, Hk, Hv, dk, dv;
  double scale;
} dims_t; /* the oracle's dimension record */

int oracle_tree_status(int T, const int32_t* par);
void oracle_prepare(int B, int T, const int32_t* parent, int32_t* depth, int32_t* order, uint64_t* anc,
                    int32_t* nvalid, int32_t* status);
void oracle_features(const dims_t* d, const int32_t* parent, const double* q, const double* k, const double* v,
                     const double* conv_w, const double* conv_state, double* feat);
void oracle_verify(const dims_t* d, const int32_t* parent, const double* q, const double* k, const double* v,
                   const double* alpha, const double* beta, const double* conv_w, const double* conv_state,
                   const double* S0, const uint8_t* node_mask, double* out);
void oracle_commit(const dims_t* d, const int32_t* parent, const int32_t* accepted, const double* q,
                   const double* k, const double* v, const double* alpha, const double* beta,
                   const double* conv_w, double* conv_state, double* S, int32_t* status);

static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(void) {
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(g_state >> 33);
}
static double unif(void) { return (rnd() + 0.5) / 2147483648.0 - 1.0; }
static double* vec(size_t n, double lo, double hi) {
  double* x = malloc(n * sizeof(double));
  for (size_t i = 0; i < n; ++i) x[i] = lo + (hi - lo) * 0.5 * (unif() + 1.0);
  return x;
}
static int finite_all(const double* x, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return 0;
  return 1;
}

/* parent arrays: kind 0 random tree (parent < i, then relabelled), 1 chain,
 * 2 padded, 3 cycle, 4 bad parent, 5 two roots, 6 empty */
static void make_parent(int32_t* par, int T, int kind) {
  int* lab = malloc(T * sizeof(int));
  for (int i = 0; i < T; ++i) lab[i] = i;
  for (int i = T - 1; i > 0; --i) {
    int j = rnd() % (i + 1), t = lab[i];
    lab[i] = lab[j];
    lab[j] = t;
  }
  int n = kind == 2 ? 1 + (int)(rnd() % T) : T;
  for (int i = 0; i < T; ++i) par[i] = -2;
  for (int i = 0; i < n; ++i) {
    int p = i == 0 ? -1 : (kind == 1 ? i - 1 : (int)(rnd() % i));
    par[lab[i]] = p < 0 ? -1 : lab[p];
  }
  if (kind == 3 && T >= 3) { par[lab[1]] = lab[2]; par[lab[2]] = lab[1]; }
  if (kind == 4) par[lab[T - 1]] = T + 5;
  if (kind == 5 && T >= 2) par[lab[T - 1]] = -1;
  if (kind == 6)
    for (int i = 0; i < T; ++i) par[i] = -2;
  free(lab);
}

int main(void) {
  const int Ts[] = {1, 2, 7, 64, 65, 130, 300};
  int fails = 0;
  for (int ti = 0; ti < 7; ++ti) {
    for (int kind = 0; kind < 7; ++kind) {
      const int T = Ts[ti];
      const int B = 2;
      dims_t d = {B, T, 1 + (int)(rnd() % 2), 0, 4 << (rnd() % 4), 4 << (rnd() % 4), 0.0};
      d.Hv = d.Hk * (1 + (int)(rnd() % 3));
      const int C = 2 * d.Hk * d.dk + d.Hv * d.dv, W = (T + 63) / 64;
      int32_t* par = malloc((size_t)B * T * sizeof(int32_t));
      for (int b = 0; b < B; ++b) make_parent(par + (size_t)b * T, T, b == 0 ? kind : 0);
      int32_t* depth = malloc((size_t)B * T * 4);
      int32_t* order = malloc((size_t)B * T * 4);
      uint64_t* anc = malloc((size_t)B * T * W * 8);
      int32_t nvalid[2], status[2], cst[2], acc[2];
      oracle_prepare(B, T, par, depth, order, anc, nvalid, status);
      for (int b = 0; b < B; ++b)
        if (status[b] != oracle_tree_status(T, par + (size_t)b * T)) fails++;
      if (kind == 0 || kind == 1 || kind == 6) fails += status[0] != 0;
      if ((kind == 3 && T >= 3) || kind == 4 || (kind == 5 && T >= 2)) fails += status[0] == 0;
      double* q = vec((size_t)B * T * d.Hk * d.dk, -1, 1);
      double* k = vec((size_t)B * T * d.Hk * d.dk, -1, 1);
      double* v = vec((size_t)B * T * d.Hv * d.dv, -1, 1);
      double* al = vec((size_t)B * T * d.Hv, 0.0, 1.0);
      double* be = vec((size_t)B * T * d.Hv, 0.0, 1.0);
      double* cw = vec((size_t)C * 4, -0.5, 0.5);
      double* cs = vec((size_t)B * 3 * C, -1, 1);
      double* S = vec((size_t)B * d.Hv * d.dv * d.dk, -0.1, 0.1);
      double* feat = malloc((size_t)B * T * C * sizeof(double));
      double* out = malloc((size_t)B * T * d.Hv * d.dv * sizeof(double));
      uint8_t* mask = malloc((size_t)B * T);
      for (int i = 0; i < B * T; ++i) mask[i] = (uint8_t)(rnd() & 1);
      oracle_features(&d, par, q, k, v, cw, cs, feat);
      oracle_verify(&d, par, q, k, v, al, be, cw, cs, S, NULL, out);
      fails += !finite_all(out, (size_t)B * T * d.Hv * d.dv);
      oracle_verify(&d, par, q, k, v, al, be, cw, cs, S, mask, out);
      for (int b = 0; b < B; ++b) {  /* the deepest real node, or -1 / out of range */
        int best = -1;
        for (int i = 0; i < T; ++i)
          if (depth[(size_t)b * T + i] >= 0 && (best < 0 || depth[(size_t)b * T + i] > depth[(size_t)b * T + best])) best = i;
        acc[b] = b == 1 && kind == 2 ? T + 3 : best;
      }
      oracle_commit(&d, par, acc, q, k, v, al, be, cw, cs, S, cst);
      fails += !finite_all(S, (size_t)B * d.Hv * d.dv * d.dk) + !finite_all(cs, (size_t)B * 3 * C);
      if (kind == 2) fails += cst[1] != 5;
      free(par); free(depth); free(order); free(anc); free(q); free(k); free(v); free(al); free(be);
      free(cw); free(cs); free(S); free(feat); free(out); free(mask);
    }
  }
  printf("oracle sanitizer driver: %d failed checks\n", fails);
  return fails != 0;
}
