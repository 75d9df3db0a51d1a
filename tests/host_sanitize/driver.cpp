// Drives every entry point of the host layer (glance_api.cpp) with the
// launchers stubbed, under AddressSanitizer and UndefinedBehaviorSanitizer:
// rejected arguments must come back with the documented status before any
// launch, accepted ones must hand the stubs a workspace carve-up that holds
// every index the kernels use, and the host-only tree check must read no
// byte outside its arrays.  Placeholder device pointers are never
// dereferenced (the stubs launch nothing).
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "glance.h"
#include "stubs.h"

static int g_checks = 0;
#define CHECK(cond)                                                                     \
  do {                                                                                  \
    ++g_checks;                                                                         \
    if (!(cond)) {                                                                      \
      fprintf(stderr, "CHECK failed at line %d: %s (%s)\n", __LINE__, #cond, glance_last_error()); \
      exit(1);                                                                          \
    }                                                                                   \
  } while (0)

static void* fake(uintptr_t k) { return reinterpret_cast<void*>(uintptr_t(1) << 32 | k << 8); }

static glance_attn_shape shape(int batch, int n, int hq, int hkv, int d, int cap, glance_dtype dt) {
  glance_attn_shape s;
  s.batch = batch;
  s.n_new = n;
  s.n_q_heads = hq;
  s.n_kv_heads = hkv;
  s.head_dim = d;
  s.ctx_capacity = cap;
  s.sm_scale = 0.f;
  s.dtype = dt;
  return s;
}

// A workspace of exactly `bytes` (heap, so ASan sees its bounds); the stubs
// check the carve-up against it.
static std::vector<char>* workspace(size_t bytes) {
  static std::vector<char> buf;
  buf.assign(bytes + 256, 0);
  char* p = buf.data();
  p += (256 - (reinterpret_cast<uintptr_t>(p) & 255)) & 255;
  g_stub.ws = p;
  g_stub.ws_bytes = bytes;
  return &buf;
}

static void attention() {
  const glance_dtype dts[] = {GLANCE_BF16, GLANCE_F32};
  const int shapes[][6] = {{1, 16, 28, 4, 128, 2048}, {4, 64, 28, 4, 128, 16384}, {16, 64, 28, 4, 128, 32768},
                           {1, 1, 4, 4, 64, 0},       {3, 7, 6, 3, 64, 129},      {40, 64, 16, 2, 128, 720},
                           {1, 64, 64, 4, 128, 5}};
  for (auto dt : dts)
    for (auto& sh : shapes) {
      glance_attn_shape s = shape(sh[0], sh[1], sh[2], sh[3], sh[4], sh[5], dt);
      const size_t need = glance_attn_workspace_size(&s, 1);
      CHECK(need > 0);
      CHECK(need == glance_attn_workspace_size(&s, 0));
      for (int tree = 0; tree < 2; ++tree) {
        workspace(need);
        const int before = g_stub.attn_bf16 + g_stub.attn_f32;
        void* ws = const_cast<void*>(g_stub.ws);
        void* kc = s.ctx_capacity ? fake(2) : nullptr;
        glance_status st = tree ? glance_tree_verify_attn(&s, fake(1), kc, kc ? fake(3) : nullptr, fake(4), fake(5),
                                                          (const int32_t*)fake(6), (const int32_t*)fake(7),
                                                          fake(8), (float*)fake(9), ws, need, nullptr)
                                : glance_block_draft_attn(&s, fake(1), kc, kc ? fake(3) : nullptr, fake(4), fake(5),
                                                          (const int32_t*)fake(6), fake(8), (float*)fake(9), ws,
                                                          need, nullptr);
        CHECK(st == GLANCE_OK);
        CHECK(g_stub.attn_bf16 + g_stub.attn_f32 == before + 1);
        CHECK(g_stub.tree == (tree == 1));
        // one byte short: rejected, nothing launched
        st = glance_block_draft_attn(&s, fake(1), kc, kc ? fake(3) : nullptr, fake(4), fake(5),
                                     (const int32_t*)fake(6), fake(8), nullptr, ws, need - 1, nullptr);
        CHECK(st == GLANCE_ERR_WORKSPACE);
        CHECK(g_stub.attn_bf16 + g_stub.attn_f32 == before + 1);
      }
    }
  // rejected shapes: no workspace size, no launch
  const int before = g_stub.attn_bf16 + g_stub.attn_f32;
  glance_attn_shape bad[] = {shape(0, 16, 28, 4, 128, 64, GLANCE_BF16), shape(1, 0, 28, 4, 128, 64, GLANCE_BF16),
                             shape(1, 65, 28, 4, 128, 64, GLANCE_BF16), shape(1, 16, 27, 4, 128, 64, GLANCE_BF16),
                             shape(1, 16, 68, 4, 128, 64, GLANCE_BF16), shape(1, 16, 28, 4, 96, 64, GLANCE_BF16),
                             shape(1, 16, 28, 4, 128, -1, GLANCE_BF16), shape(1, 16, 28, 0, 128, 64, GLANCE_BF16),
                             shape(1, 16, 28, 4, 128, 64, (glance_dtype)7),
                             shape(2147483647, 64, 64, 4, 128, 2147483647, GLANCE_BF16),
                             shape(2147483647, 64, 64, 4, 128, 2147483647, GLANCE_F32)};
  for (auto& s : bad) {
    CHECK(glance_attn_workspace_size(&s, 1) == 0);
    CHECK(glance_block_draft_attn(&s, fake(1), fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6), fake(8),
                                  nullptr, fake(10), size_t(1) << 40, nullptr) != GLANCE_OK);
  }
  glance_attn_shape s = shape(1, 16, 28, 4, 128, 64, GLANCE_BF16);
  s.sm_scale = NAN;
  CHECK(glance_attn_workspace_size(&s, 0) == 0);
  s.sm_scale = INFINITY;
  CHECK(glance_attn_workspace_size(&s, 0) == 0);
  CHECK(glance_attn_workspace_size(nullptr, 0) == 0);
  // null and misaligned pointers
  s = shape(1, 16, 28, 4, 128, 64, GLANCE_BF16);
  const size_t need = glance_attn_workspace_size(&s, 0);
  CHECK(glance_block_draft_attn(&s, nullptr, fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6), fake(8),
                                nullptr, fake(10), need, nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_block_draft_attn(&s, (char*)fake(1) + 8, fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6),
                                fake(8), nullptr, fake(10), need, nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_block_draft_attn(&s, fake(1), fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6), fake(8),
                                nullptr, (char*)fake(10) + 128, need, nullptr) == GLANCE_ERR_WORKSPACE);
  CHECK(glance_tree_verify_attn(&s, fake(1), fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6), nullptr,
                                fake(8), nullptr, fake(10), need, nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(g_stub.attn_bf16 + g_stub.attn_f32 == before);
}

static void profiling_hook() {
  glance_attn_shape s = shape(1, 16, 28, 4, 128, 256, GLANCE_BF16);
  const size_t need = glance_attn_workspace_size(&s, 0);
  workspace(need);
  CHECK(glance_set_kernel_events(fake(20), fake(21)) == GLANCE_OK);
  CHECK(glance_block_draft_attn(&s, fake(1), fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6), fake(8),
                                nullptr, const_cast<void*>(g_stub.ws), need, nullptr) == GLANCE_OK);
  CHECK(g_stub.ev0 == (hipEvent_t)fake(20) && g_stub.ev1 == (hipEvent_t)fake(21));
  CHECK(glance_block_draft_attn(&s, fake(1), fake(2), fake(3), fake(4), fake(5), (const int32_t*)fake(6), fake(8),
                                nullptr, const_cast<void*>(g_stub.ws), need, nullptr) == GLANCE_OK);
  CHECK(g_stub.ev0 == nullptr && g_stub.ev1 == nullptr);  // the pair is used once
}

static void acceptance() {
  const int shapes[][3] = {{4, 64, 152064}, {1, 1, 1}, {16, 64, 152064}, {1, 16, 1000}, {7, 33, 5}, {1, 64, 1 << 30}};
  for (auto& sh : shapes)
    for (int dt = 0; dt < 2; ++dt) {
      const size_t need = glance_accept_workspace_size(sh[0], sh[1], sh[2]);
      CHECK(need > 0);
      workspace(need);
      void* ws = const_cast<void*>(g_stub.ws);
      const int before = g_stub.accept;
      CHECK(glance_greedy_accept(sh[0], sh[1], sh[2], (glance_dtype)dt, fake(1), (const int32_t*)fake(2),
                                 (const int32_t*)fake(3), (int32_t*)fake(4), (int32_t*)fake(5), (int32_t*)fake(6),
                                 16, (int32_t*)fake(7), ws, need, nullptr) == GLANCE_OK);
      CHECK(glance_greedy_accept_entropy(sh[0], sh[1], sh[2], (glance_dtype)dt, fake(1), (const int32_t*)fake(2),
                                         (const int32_t*)fake(3), (int32_t*)fake(4), (int32_t*)fake(5),
                                         (int32_t*)fake(6), 16, (int32_t*)fake(7), (float*)fake(8), ws, need,
                                         nullptr) == GLANCE_OK);
      CHECK(glance_sample_accept(sh[0], sh[1], sh[2], (glance_dtype)dt, fake(1), (const int32_t*)fake(2),
                                 (const int32_t*)fake(3), 0.7f, ~0ull, ~0u, nullptr, (int32_t*)fake(4),
                                 (int32_t*)fake(5), (int32_t*)fake(6), 16, (int32_t*)fake(7), ws, need,
                                 nullptr) == GLANCE_OK);
      CHECK(g_stub.accept == before + 2);
      CHECK(glance_greedy_accept(sh[0], sh[1], sh[2], (glance_dtype)dt, fake(1), (const int32_t*)fake(2),
                                 (const int32_t*)fake(3), (int32_t*)fake(4), (int32_t*)fake(5), (int32_t*)fake(6),
                                 16, (int32_t*)fake(7), ws, need - 1, nullptr) == GLANCE_ERR_WORKSPACE);
      const int b2 = g_stub.accept;
      const glance_status st = glance_greedy_accept_noalloc(
          sh[0], sh[1], sh[2], (glance_dtype)dt, fake(1), (const int32_t*)fake(2), (const int32_t*)fake(3),
          (int32_t*)fake(4), (int32_t*)fake(5), (int32_t*)fake(6), 16, (int32_t*)fake(7), nullptr);
      CHECK(st == (need <= (size_t(1) << 20) ? GLANCE_OK : GLANCE_ERR_UNSUPPORTED));
      CHECK(g_stub.accept == b2 + (st == GLANCE_OK));
    }
  const int before = g_stub.accept + g_stub.sample;
  CHECK(glance_accept_workspace_size(0, 1, 1) == 0);
  CHECK(glance_accept_workspace_size(1, 65, 1) == 0);
  CHECK(glance_accept_workspace_size(1, 1, 0) == 0);
  CHECK(glance_accept_workspace_size(2147483647, 64, 1 << 30) == 0);
  const float temps[] = {0.f, -1.f, NAN, INFINITY, 1e-40f};
  for (float t : temps)
    CHECK(glance_sample_accept(1, 8, 100, GLANCE_BF16, fake(1), (const int32_t*)fake(2), (const int32_t*)fake(3), t,
                               1, 1, nullptr, (int32_t*)fake(4), (int32_t*)fake(5), (int32_t*)fake(6), 8,
                               (int32_t*)fake(7), fake(9), size_t(1) << 20, nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_greedy_accept(1, 8, 100, GLANCE_BF16, fake(1), nullptr, (const int32_t*)fake(3), (int32_t*)fake(4),
                             (int32_t*)fake(5), (int32_t*)fake(6), 8, (int32_t*)fake(7), fake(9), size_t(1) << 20,
                             nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_greedy_accept(1, 8, 100, GLANCE_BF16, fake(1), (const int32_t*)fake(2), (const int32_t*)fake(3),
                             (int32_t*)fake(4), (int32_t*)fake(5), (int32_t*)fake(6), 0, (int32_t*)fake(7), fake(9),
                             size_t(1) << 20, nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_greedy_accept_entropy(1, 8, 100, GLANCE_BF16, fake(1), (const int32_t*)fake(2),
                                     (const int32_t*)fake(3), (int32_t*)fake(4), (int32_t*)fake(5), (int32_t*)fake(6),
                                     8, (int32_t*)fake(7), nullptr, fake(9), size_t(1) << 20,
                                     nullptr) == GLANCE_ERR_INVALID_ARG);
  CHECK(g_stub.accept + g_stub.sample == before);
}

static void tree_builder_and_commit() {
  const int shapes[][4] = {{4, 15, 152064, 63}, {1, 1, 1000, 63}, {1, 2, 2, 6}, {64, 15, 100, 63}, {1, 15, 1 << 30, 1}};
  for (auto& sh : shapes) {
    const size_t need = glance_tree_workspace_size(sh[0], sh[1], sh[2], sh[3]);
    CHECK(need > 0);
    workspace(need);
    const int before = g_stub.tree_calls;
    CHECK(glance_build_tree(sh[0], sh[1], sh[2], sh[3], GLANCE_BF16, fake(1), (int64_t)sh[1] * sh[2],
                            (const int32_t*)fake(2), (int32_t*)fake(3), (int32_t*)fake(4), (float*)fake(5),
                            const_cast<void*>(g_stub.ws), need, nullptr) == GLANCE_OK);
    CHECK(g_stub.tree_calls == before + 1);
    CHECK(glance_build_tree(sh[0], sh[1], sh[2], sh[3], GLANCE_BF16, fake(1), (int64_t)sh[1] * sh[2] - 1,
                            (const int32_t*)fake(2), (int32_t*)fake(3), (int32_t*)fake(4), nullptr,
                            const_cast<void*>(g_stub.ws), need, nullptr) == GLANCE_ERR_INVALID_ARG);
  }
  CHECK(glance_tree_workspace_size(1, 16, 152064, 63) == 0);
  CHECK(glance_tree_workspace_size(1, 15, 152064, 64) == 0);
  CHECK(glance_tree_workspace_size(1, 2, 2, 7) == 0);
  CHECK(glance_tree_workspace_size(65536, 15, 152064, 63) == 0);
  const int c0 = g_stub.commit;
  CHECK(glance_commit_path(4, 64, 4, 128, 16448, GLANCE_BF16, fake(1), fake(2), (const int32_t*)fake(3),
                           (const int32_t*)fake(4), 16, fake(5), fake(6), (int32_t*)fake(7), nullptr) == GLANCE_OK);
  CHECK(glance_commit_path(4, 65, 4, 128, 16448, GLANCE_BF16, fake(1), fake(2), (const int32_t*)fake(3),
                           (const int32_t*)fake(4), 16, fake(5), fake(6), (int32_t*)fake(7), nullptr) != GLANCE_OK);
  CHECK(glance_commit_path(4, 64, 4, 128, 0, GLANCE_BF16, fake(1), fake(2), (const int32_t*)fake(3),
                           (const int32_t*)fake(4), 16, fake(5), fake(6), (int32_t*)fake(7), nullptr) != GLANCE_OK);
  CHECK(glance_commit_path(4, 64, 4, 128, 100, GLANCE_BF16, fake(1), nullptr, (const int32_t*)fake(3),
                           (const int32_t*)fake(4), 16, fake(5), fake(6), (int32_t*)fake(7), nullptr) != GLANCE_OK);
  CHECK(g_stub.commit == c0 + 1);
}

// Host-only tree check: heap arrays of exactly n entries.
static void validate_tree() {
  for (int n = 1; n <= 64; ++n) {
    int32_t* par = (int32_t*)malloc(sizeof(int32_t) * n);
    int32_t* tok = (int32_t*)malloc(sizeof(int32_t) * n);
    for (int i = 0; i < n; ++i) {
      par[i] = i - 1;  // chain
      tok[i] = i;
    }
    CHECK(glance_validate_tree(n, par, tok, -1) == GLANCE_OK);
    CHECK(glance_validate_tree(n, par, tok, n - 1) == GLANCE_OK);
    if (n > 1) CHECK(glance_validate_tree(n, par, tok, n - 2) == GLANCE_ERR_INVALID_ARG);
    for (int i = 1; i < n; ++i) par[i] = 0;  // star
    CHECK(glance_validate_tree(n, par, tok, 1) == GLANCE_OK);
    CHECK(glance_validate_tree(n, par, nullptr, 1) == GLANCE_OK);
    if (n > 2) {
      tok[2] = tok[1];  // two children of the root carry one token
      CHECK(glance_validate_tree(n, par, tok, 1) == GLANCE_ERR_INVALID_ARG);
      par[2] = 2;  // not before itself
      CHECK(glance_validate_tree(n, par, nullptr, -1) == GLANCE_ERR_INVALID_ARG);
      par[2] = 5000;
      CHECK(glance_validate_tree(n, par, nullptr, -1) == GLANCE_ERR_INVALID_ARG);
    }
    par[0] = 0;
    CHECK(glance_validate_tree(n, par, nullptr, -1) == GLANCE_ERR_INVALID_ARG);
    free(par);
    free(tok);
  }
  int32_t one = -1;
  CHECK(glance_validate_tree(0, &one, nullptr, -1) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_validate_tree(65, &one, nullptr, -1) == GLANCE_ERR_INVALID_ARG);
  CHECK(glance_validate_tree(1, nullptr, nullptr, -1) == GLANCE_ERR_INVALID_ARG);
}

static void status_strings() {
  for (int c = -10; c <= 10; ++c) CHECK(glance_status_string((glance_status)c) != nullptr);
  CHECK(strlen(glance_last_error()) > 0);
  CHECK(glance_version() >= 100);
}

int main() {
  attention();
  profiling_hook();
  acceptance();
  tree_builder_and_commit();
  validate_tree();
  status_strings();
  printf("host layer under sanitizers: %d checks passed\n", g_checks);
  return 0;
}
