// Sanitizer driver for the host side of the C ABI (test infrastructure):
// gdn_abi.hip is linked against stub launchers that record that they were
// reached, and every entry point is called with invalid sizes, dtypes,
// scales, NULL pointers, overlapping buffers and empty problems.  Each call
// must return its documented status without reaching a launcher (except the
// valid calls, which must reach exactly their launcher), and gdn_last_error
// must hold a message.  Built with -fsanitize=address,undefined by
// tests/test_sanitize_cpu.py.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <string.h>

#include "gdn_internal.h"

static int g_reached = 0;
namespace gdn {
int launch_prepare(int, int, const int32_t*, void*, int32_t*, hipStream_t) { return ++g_reached, GDN_OK; }
int launch_verify(const VerifyArgs&, hipStream_t) { return ++g_reached, GDN_OK; }
int launch_verify_large(const VerifyArgs&, void*, size_t, hipStream_t) { return ++g_reached, GDN_OK; }
int launch_verify_noalloc(const VerifyArgs&, hipStream_t) { return ++g_reached, GDN_OK; }
int launch_verify_chunked(const VerifyArgs&, void*, size_t, hipStream_t) { return ++g_reached, GDN_OK; }
int launch_commit(const CommitArgs&, hipStream_t) { return ++g_reached, GDN_OK; }
size_t large_workspace_bytes(int B, int T, int Hk, int Hv, int dk, int dv) {
  return ((size_t(B) * T * (2 * Hk * dk + Hv * dv) * 2 + 255) & ~size_t(255)) + size_t(B) * T * Hv * 4;
}
size_t chunked_workspace_bytes(int B, int T, int Hk, int Hv, int dk, int dv) {
  return size_t(B) * T * (2 * Hk * dk + Hv * dv) * 4 + size_t(B) * Hv * T * dv * 4;
}
static char g_ws[64];
void* stream_workspace(size_t, hipStream_t, int* rc) { return *rc = GDN_OK, g_ws; }
}  // namespace gdn

static int fails = 0;
static void expect(const char* what, int got, int want, int reached_want) {
  const int r = g_reached;
  g_reached = 0;
  if (got != want || r != reached_want || (want != GDN_OK && strlen(gdn_last_error()) == 0)) {
    printf("FAIL %s: status %d (want %d), launchers reached %d (want %d), msg '%s'\n", what, got, want, r,
           reached_want, gdn_last_error());
    ++fails;
  }
}

int main() {
  void* p = reinterpret_cast<void*>(0x1000);  // never dereferenced by the host code
  const float* f = static_cast<const float*>(p);
  float* fo = static_cast<float*>(p);
  const int32_t* ci = static_cast<const int32_t*>(p);
  int32_t* io = static_cast<int32_t*>(p);
  gdn_dims ok = {2, 40, 2, 4, 64, 32, GDN_BF16, 0.0f};
  gdn_dims bad[] = {
      {2, 40, 2, 3, 64, 32, GDN_BF16, 0.0f},   // Hv % Hk
      {2, 40, 0, 4, 64, 32, GDN_BF16, 0.0f},   // Hk
      {-1, 40, 2, 4, 64, 32, GDN_BF16, 0.0f},  // B
      {2, -3, 2, 4, 64, 32, GDN_BF16, 0.0f},   // T
      {2, 40, 2, 4, 48, 32, GDN_BF16, 0.0f},   // dk
      {2, 40, 2, 4, 64, 256, GDN_BF16, 0.0f},  // dv
      {2, 513, 2, 4, 64, 32, GDN_BF16, 0.0f},  // T > GDN_MAX_T
      {2, 40, 2, 4, 64, 32, 7, 0.0f},          // dtype
      {2, 40, 2, 4, 64, 32, GDN_BF16, -1.0f},  // scale
  };
  const int want[] = {GDN_EINVAL, GDN_EINVAL, GDN_EINVAL, GDN_EINVAL, GDN_EUNSUPPORTED,
                      GDN_EUNSUPPORTED, GDN_EUNSUPPORTED, GDN_EINVAL, GDN_EINVAL};
  for (int i = 0; i < 9; ++i) {
    expect("verify bad dims", gdn_tree_verify(&bad[i], p, p, p, p, p, p, f, f, f, fo, nullptr), want[i], 0);
    expect("verify_noalloc bad dims", gdn_tree_verify_noalloc(&bad[i], p, p, p, p, p, p, f, f, f, fo, nullptr),
           want[i], 0);
    expect("verify_chunked bad dims", gdn_tree_verify_chunked(&bad[i], p, p, p, p, p, p, f, f, f, fo, nullptr),
           want[i], 0);
    expect("commit bad dims", gdn_tree_commit(&bad[i], p, ci, p, p, p, p, p, f, fo, fo, io, nullptr), want[i], 0);
    expect("step bad dims",
           gdn_tree_step(&bad[i], p, ci, p, p, p, p, p, io, p, p, p, p, p, p, f, f, fo + 100000, fo, fo, nullptr),
           want[i], 0);
  }
  expect("verify NULL dims", gdn_tree_verify(nullptr, p, p, p, p, p, p, f, f, f, fo, nullptr), GDN_EINVAL, 0);
  expect("verify NULL out", gdn_tree_verify(&ok, p, p, p, p, p, p, f, f, f, nullptr, nullptr), GDN_EINVAL, 0);
  expect("commit NULL S", gdn_tree_commit(&ok, p, ci, p, p, p, p, p, f, fo, nullptr, io, nullptr), GDN_EINVAL, 0);
  expect("prepare NULL", gdn_tree_prepare(&ok, nullptr, p, io, nullptr), GDN_EINVAL, 0);
  // conv_state and conv_state_out overlap by one float
  const size_t C = 2 * 2 * 64 + 4 * 32;
  expect("step overlap",
         gdn_tree_step(&ok, p, ci, p, p, p, p, p, io, p, p, p, p, p, p, f, f, fo + 2 * 3 * C - 1, fo, fo, nullptr),
         GDN_EINVAL, 0);
  // the no-alloc variant refuses workspaces above its static array
  gdn_dims big = {64, 512, 16, 48, 128, 128, GDN_BF16, 0.0f};
  expect("noalloc oversize", gdn_tree_verify_noalloc(&big, p, p, p, p, p, p, f, f, f, fo, nullptr),
         GDN_EUNSUPPORTED, 0);
  // empty problems succeed without touching anything
  gdn_dims empty = {0, 40, 2, 4, 64, 32, GDN_BF16, 0.0f};
  expect("verify empty", gdn_tree_verify(&empty, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                         nullptr, nullptr, nullptr, nullptr), GDN_OK, 0);
  expect("prepare empty", gdn_tree_prepare(&empty, nullptr, nullptr, nullptr, nullptr), GDN_OK, 0);
  // valid calls reach exactly their launchers
  expect("prepare ok", gdn_tree_prepare(&ok, ci, p, io, nullptr), GDN_OK, 1);
  expect("verify ok", gdn_tree_verify(&ok, p, p, p, p, p, p, f, f, f, fo, nullptr), GDN_OK, 1);
  gdn_dims large = ok;
  large.T = 300;
  expect("verify large ok", gdn_tree_verify(&large, p, p, p, p, p, p, f, f, f, fo, nullptr), GDN_OK, 1);
  expect("chunked ok", gdn_tree_verify_chunked(&large, p, p, p, p, p, p, f, f, f, fo, nullptr), GDN_OK, 1);
  expect("commit ok", gdn_tree_commit(&ok, p, ci, p, p, p, p, p, f, fo, fo, io, nullptr), GDN_OK, 1);
  expect("step ok", gdn_tree_step(&ok, p, ci, p, p, p, p, p, io, p, p, p, p, p, p, f, f, fo + 2 * 3 * C, fo, fo,
                                  nullptr), GDN_OK, 1);
  expect("step large ok (fused pull-back)",
         gdn_tree_step(&large, p, ci, p, p, p, p, p, io, p, p, p, p, p, p, f, f, fo + 2 * 3 * C, fo, fo, nullptr),
         GDN_OK, 1);
  gdn_dims tiny = large;  // 16 x 16 heads: the commit kernels, then verify
  tiny.dk = 16;
  tiny.dv = 16;
  expect("step large tiny heads (commit + verify)",
         gdn_tree_step(&tiny, p, ci, p, p, p, p, p, io, p, p, p, p, p, p, f, f, fo + 2 * 3 * C, fo, fo, nullptr),
         GDN_OK, 2);
  if (gdn_tree_meta_bytes(0, 5) != 0 || gdn_tree_meta_bytes(3, 0) != 0 || gdn_tree_meta_bytes(32, 512) % 256) {
    printf("FAIL meta_bytes\n");
    ++fails;
  }
  printf("abi sanitizer driver: %d failed checks (%s)\n", fails, gdn_version());
  return fails != 0;
}
