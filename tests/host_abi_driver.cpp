// Host-side ABI driver for the sanitizer test (built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code only).
//
// Every call below stops at a host-side check or is a pure host function
// (status strings, workspace sizing, split planning): none reaches a kernel
// launch, so the driver is safe with or without a GPU. Pointers are fake
// non-null values where a check only tests for null.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "cure.h"

static int failures = 0;

static void expect(int got, int want, const char* what) {
  if (got != want) {
    std::printf("FAIL %s: got %d want %d\n", what, got, want);
    ++failures;
  }
}

int main() {
  void* const P = reinterpret_cast<void*>(uintptr_t(0x1000));
  float* const F = reinterpret_cast<float*>(P);
  int32_t* const I = reinterpret_cast<int32_t*>(P);
  const int64_t* const I64 = reinterpret_cast<const int64_t*>(P);

  for (int s = -3; s < 10; ++s)
    if (!cure_status_string(s)) ++failures;
  expect(cure_version() >= 100, 1, "version");

  // Margin pass: argument errors, and a missing workspace when rows are split.
  auto margins = [&](int dtype, int batch, int rows, int vocab, int64_t ld, const void* logits,
                     int chain, int depth, int32_t* ufp_pos, int32_t* ufp_cnt) {
    return (int)cure_margins(logits, dtype, batch, rows, vocab, ld, F, I, F, I, F, F, chain, 1.0f,
                             16, depth, ufp_pos, ufp_cnt, nullptr, 0, nullptr);
  };
  expect(margins(7, 1, 4, 1000, 1000, P, 2, 4, I, I), CURE_ERR_INVALID_ARG, "margins dtype");
  expect(margins(1, 1, 4, 1, 1, P, 2, 4, I, I), CURE_ERR_INVALID_ARG, "margins vocab");
  expect(margins(1, 1, 4, 1000, 999, P, 2, 4, I, I), CURE_ERR_INVALID_ARG, "margins ld");
  expect(margins(1, 1, 4, 1000, 1000, nullptr, 2, 4, I, I), CURE_ERR_INVALID_ARG, "margins null");
  expect(margins(1, 1, 4, 1000, 1000, P, 5, 4, I, I), CURE_ERR_INVALID_ARG, "margins chain");
  expect(margins(1, 1, 4, 1000, 1000, P, 2, 0, I, I), CURE_ERR_INVALID_ARG, "margins depth");
  expect(margins(1, 1, 4, 1000, 1000, P, 2, 4, I, nullptr), CURE_ERR_INVALID_ARG, "margins gate");
  expect(margins(1, 1, 2000, 1000, 1000, P, 1500, 4, I, I), CURE_ERR_UNSUPPORTED, "margins chain max");
  expect(margins(1, 1, 4, 100000, 100000, P, 2, 4, I, I), CURE_ERR_WORKSPACE, "margins workspace");
  expect(margins(1, 0, 4, 100000, 100000, P, 2, 4, I, I), CURE_OK, "margins empty");
  expect(margins(1, 1 << 20, 4096, 128256, 128256, P, 2, 4, I, I), CURE_ERR_UNSUPPORTED,
         "margins too many rows");
  // The allocation-free entry point: the same checks, before any device call.
  auto margins_na = [&](int dtype, int batch, int rows, int vocab, int64_t ld,
                        const void* logits, int chain, int depth, int32_t* ufp_pos,
                        int32_t* ufp_cnt) {
    return (int)cure_margins_noalloc(logits, dtype, batch, rows, vocab, ld, F, I, F, I, F, F,
                                     chain, 1.0f, 16, depth, ufp_pos, ufp_cnt, nullptr);
  };
  expect(margins_na(7, 1, 4, 1000, 1000, P, 2, 4, I, I), CURE_ERR_INVALID_ARG, "noalloc dtype");
  expect(margins_na(1, 1, 4, 1000, 999, P, 2, 4, I, I), CURE_ERR_INVALID_ARG, "noalloc ld");
  expect(margins_na(1, 1, 4, 1000, 1000, P, 2, 4, nullptr, I), CURE_ERR_INVALID_ARG,
         "noalloc gate");
  expect(margins_na(1, 0, 4, 100000, 100000, P, 2, 4, I, I), CURE_OK, "noalloc empty");
  expect(margins_na(1, 1 << 20, 4096, 128256, 128256, P, 2, 4, I, I), CURE_ERR_UNSUPPORTED,
         "noalloc too many rows");
  expect(cure_margins_noalloc_scratch_bytes() == 256 * 1024, 1, "noalloc scratch size");

  // Margin pass with the acceptance walk: its own checks after cure_margins'.
  auto margins_acc = [&](int batch, int rows, int vocab, int chain, const int32_t* parent,
                         int32_t* path) {
    return (int)cure_margins_accept(P, 1, batch, rows, vocab, vocab, F, I, F, I, F, F, chain,
                                    1.0f, 4, 2, nullptr, nullptr, parent, I, I, I, I, path, I,
                                    I, I, nullptr, 0, nullptr);
  };
  expect(margins_acc(1, 4, 1000, 2, nullptr, I), CURE_ERR_INVALID_ARG, "margins_accept parent");
  expect(margins_acc(1, 4, 1000, 2, I, nullptr), CURE_ERR_INVALID_ARG, "margins_accept path");
  expect(margins_acc(1, 4, 1000, -1, I, I), CURE_ERR_INVALID_ARG, "margins_accept chain");
  expect(margins_acc(1, 300, 1000, 2, I, I), CURE_ERR_UNSUPPORTED, "margins_accept rows");
  expect(margins_acc(1, 4, 100000, 2, I, I), CURE_ERR_WORKSPACE, "margins_accept workspace");
  expect(margins_acc(0, 4, 100000, 2, I, I), CURE_OK, "margins_accept empty");
  size_t last = 0;
  for (int b : {1, 7, 16, 1024})
    for (int r : {1, 32, 48, 333})
      for (int v : {2, 1000, 128256, 1 << 22}) {
        const size_t ws = cure_margins_workspace_size(b, r, v);
        if (ws % 256 != 0) ++failures;
        last ^= ws;
      }

  // Tree attention: the split planner over ragged, long and degenerate batches
  // (pure host), and argument errors that stop before any launch.
  std::vector<int32_t> ctx, nn;
  auto plan = [&](int batch, int hq, int hkv, int d, int n_max, int split) {
    return cure_tree_attn_workspace_size(batch, hq, hkv, d, n_max, ctx.data(), nn.data(), split);
  };
  for (int batch : {1, 3, 16, 257, 4096}) {
    ctx.assign(batch, 0);
    nn.assign(batch, 0);
    for (int b = 0; b < batch; ++b) {
      ctx[b] = (b * 7919) % 70000 + (b % 5 == 0 ? 0 : 1);
      nn[b] = b % 9 == 0 ? 0 : 1 + (b * 31) % 256;
    }
    for (int d : {64, 128})
      for (int hq_hkv : {1, 4, 8})
        for (int split : {0, 1, 2, 7, 1000, 1 << 20})
          last ^= plan(batch, 8 * hq_hkv, 8, d, 256, split);
  }
  ctx.assign(2, 1 << 30);
  nn.assign(2, 256);
  last ^= plan(2, 32, 8, 128, 256, 0);                      // splits capped by the grid limit
  last ^= plan(2, 32, 8, 128, 256, 3);
  ctx.assign(4, 32768);
  nn.assign(4, 32);
  auto attn = [&](int dtype, int d, int n_max, int hq, int hkv, void* ws) {
    return (int)cure_tree_attn(P, P, P, P, F, dtype, 1, 4, hq, hkv, d, 0.125f, I64, I, I, I,
                               n_max, ctx.data(), nn.data(), 0, 0u, I, ws, 0, nullptr);
  };
  expect(attn(3, 128, 32, 32, 8, nullptr), CURE_ERR_INVALID_ARG, "attn dtype");
  expect(attn(1, 96, 32, 32, 8, nullptr), CURE_ERR_UNSUPPORTED, "attn head dim");
  expect(attn(1, 128, 300, 32, 8, nullptr), CURE_ERR_UNSUPPORTED, "attn n_max");
  expect(attn(1, 128, 32, 30, 8, nullptr), CURE_ERR_INVALID_ARG, "attn gqa");
  expect(attn(1, 128, 16, 32, 8, nullptr), CURE_ERR_INVALID_ARG, "attn nodes > n_max");
  expect(attn(1, 128, 32, 32, 8, nullptr), CURE_ERR_WORKSPACE, "attn workspace");
  void* const P4 = reinterpret_cast<void*>(uintptr_t(0x1004));
  expect((int)cure_tree_attn(P, P, P, P4, F, 1, 1, 4, 32, 8, 128, 0.125f, I64, I, I, I, 32,
                             ctx.data(), nn.data(), 0, 0u, I, P, size_t(1) << 40, nullptr),
         CURE_ERR_INVALID_ARG, "attn o alignment");
  expect((int)cure_tree_attn(P, P, P, P, F, 1, 1, 4, 32, 8, 128, 0.125f, I64, I, I, I, 32,
                             ctx.data(), nn.data(), 0, 0u, I, P4, size_t(1) << 40, nullptr),
         CURE_ERR_INVALID_ARG, "attn workspace alignment");

  // Acceptance walk, repair tree, commit, read ceiling: argument errors.
  expect((int)cure_accept(I, I, I, I, I, 4, 2, 300, I, I, I, I, I, nullptr), CURE_ERR_UNSUPPORTED,
         "accept n_max");
  expect((int)cure_accept(nullptr, I, I, I, I, 4, 2, 8, I, I, I, I, I, nullptr),
         CURE_ERR_INVALID_ARG, "accept null");
  expect((int)cure_accept(I, I, I, I, I, 4, 0, 8, I, I, I, I, I, nullptr), CURE_OK, "accept empty");
  auto repair = [&](int batch, int rows, int vocab, int chain, int budget, int depth, int bmin,
                    int bmax, float scale, int n_max, void* ws) {
    return (int)cure_repair_tree(P, 1, batch, rows, vocab, vocab, F, I, I, I, chain, budget, depth,
                                 scale, bmin, bmax, nullptr, n_max, I, I, I, nullptr, ws, 0,
                                 nullptr);
  };
  expect(repair(1, 16, 32000, 16, 16, 4, 1, 5, 1.f, 31, nullptr), CURE_ERR_INVALID_ARG, "repair n_max");
  expect(repair(1, 16, 32000, 16, 16, 4, 3, 2, 1.f, 32, nullptr), CURE_ERR_INVALID_ARG, "repair b range");
  expect(repair(1, 16, 32000, 16, 16, 4, 1, 8, 1.f, 32, nullptr), CURE_ERR_UNSUPPORTED, "repair b_max");
  expect(repair(1, 16, 32000, 16, 16, 4, 1, 5, 0.f, 32, nullptr), CURE_ERR_INVALID_ARG, "repair scale");
  expect(repair(1, 16, 32000, 16, 16, 4, 1, 5, 1.f, 32, nullptr), CURE_ERR_WORKSPACE, "repair workspace");
  expect(repair(0, 16, 32000, 16, 16, 4, 1, 5, 1.f, 32, nullptr), CURE_OK, "repair empty");
  for (int b : {1, 16, 4096})
    for (int v : {6, 32000, 128256, 524288})
      for (int budget : {0, 3, 16, 64, 256}) last ^= cure_repair_tree_workspace_size(b, 16, v, budget, 4);
  auto commit = [&](int dtype, int layers, int64_t stride, int hkv, int d, int batch, int n_max,
                    int32_t* new_ctx) {
    return (int)cure_commit(P, P, dtype, layers, stride, hkv, d, batch, I64, I, I, I, I, I, I, 16,
                            n_max, new_ctx, I, I, I, I, nullptr);
  };
  int32_t other[1];
  expect(commit(3, 2, 4096, 8, 128, 2, 32, other), CURE_ERR_INVALID_ARG, "commit dtype");
  expect(commit(1, 2, 0, 8, 128, 2, 32, other), CURE_ERR_INVALID_ARG, "commit stride");
  expect(commit(1, 2, 4096, 8, 128, 2, 32, I), CURE_ERR_INVALID_ARG, "commit alias");
  expect(commit(1, 2, 4096, 1, 4, 2, 32, other), CURE_ERR_UNSUPPORTED, "commit row bytes");
  expect(commit(1, 2, 4096, 8, 128, 2, 257, other), CURE_ERR_UNSUPPORTED, "commit n_max");
  expect(commit(1, 2, 4096, 8, 128, 70000, 32, other), CURE_ERR_UNSUPPORTED, "commit batch");
  expect(commit(1, 2, 4096, 8, 128, 0, 32, other), CURE_OK, "commit empty");
  expect((int)cure_read_ceiling(P, 60, reinterpret_cast<uint32_t*>(P), nullptr),
         CURE_ERR_INVALID_ARG, "ceiling size");
  expect((int)cure_read_ceiling(nullptr, 0, nullptr, nullptr), CURE_OK, "ceiling empty");
  if (cure_read_ceiling_chunks((size_t(1) << 40) + 1) != (size_t(1) << 22) + 1) ++failures;

  std::printf("host ABI driver: %d failure(s) (checksum %zu)\n", failures, last);
  return failures == 0 ? 0 : 1;
}
