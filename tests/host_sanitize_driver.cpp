// Host-side driver of the C ABI for sanitizer builds (AddressSanitizer, UndefinedBehaviorSanitizer).
// Calls every entry point of dels.h with rejected arguments, extreme sizes for the size queries
// and, unless "--no-valid" is given, valid arguments that stop at the device check on a host
// without a GPU.  Fake device addresses are never dereferenced on the host: every call that gets
// them fails validation or the device check first.  Threads check that the last-error message
// is per thread.  Exit status 0 when every expectation holds.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "../include/dels.h"

namespace {

int g_fail = 0;

void expect(bool ok, const char* what, int line) {
  if (!ok) {
    std::fprintf(stderr, "line %d: %s (last error: %s)\n", line, what, dls_last_error());
    ++g_fail;
  }
}
#define EXPECT(c) expect((c), #c, __LINE__)

void* fake(int i) { return reinterpret_cast<void*>(static_cast<uintptr_t>(0x7f0000000000ull + 0x100000ull * i)); }
void* off(int i, int b) { return static_cast<char*>(fake(i)) + b; }

dls_local_head rnn(int32_t V = 1000, int32_t d = 64, int32_t H = 32, int32_t r = 16) {
  dls_local_head h;
  std::memset(&h, 0, sizeof h);
  h.V = V;
  h.d = d;
  h.H = H;
  h.r = r;
  h.dtype = DLS_BF16;
  h.emb = fake(0);
  h.w_ih = fake(1);
  h.w_hh = fake(2);
  h.w_rank = fake(3);
  h.w_vocab = fake(4);
  h.kind = DLS_HEAD_RNN;
  return h;
}

dls_local_head markov(int32_t V = 1000, int32_t r = 16) {
  dls_local_head h = rnn(V, 0, 0, r);
  h.w_ih = h.w_hh = h.w_rank = nullptr;
  h.kind = DLS_HEAD_MARKOV;
  return h;
}

dls_fusion fusion(float wl = 1.f, float a = 0.3f, float b = 0.3f, uint32_t flags = 0) { return {wl, a, b, flags}; }

dls_status draft(const dls_local_head& h, int32_t batch = 2, int32_t B = 4, dls_fusion f = fusion(),
                 const void* longp = fake(5), dls_dtype ldt = DLS_BF16, const int32_t* last = (int32_t*)fake(6),
                 int32_t* tok = (int32_t*)fake(7), void* ws = fake(9), size_t wsb = (size_t)1 << 30) {
  return dls_draft_block(&h, longp, ldt, last, nullptr, batch, B, f, tok, (dls_row_stats*)fake(8), ws, wsb, nullptr);
}

void rejected_arguments() {
  const float nan = std::nanf("");
  // drafting: head, shapes, dtypes, pointers, alignment, workspace, fusion
  EXPECT(draft(rnn(0)) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(1 << 25)) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(1000, 12)) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(1000, 64, 4)) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(1000, 64, 32, 1024)) == DLS_ERR_SHAPE);
  dls_local_head h = rnn();
  h.dtype = (dls_dtype)7;
  EXPECT(draft(h) == DLS_ERR_DTYPE);
  h = rnn();
  h.w_rank = nullptr;
  EXPECT(draft(h) == DLS_ERR_ARG);
  h = rnn();
  h.w_vocab = off(4, 2);
  EXPECT(draft(h) == DLS_ERR_ARG);
  h = rnn();
  h.kind = 9;
  EXPECT(draft(h) == DLS_ERR_ARG);
  h = rnn();
  h.prepared = fake(11);
  h.prepared_bytes = 64;   // far less than this head's prepared form
  EXPECT(draft(h) == DLS_ERR_WORKSPACE);
  h.prepared = off(11, 16);
  h.prepared_bytes = (size_t)1 << 40;
  EXPECT(draft(h) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 257) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(), -1) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(), 2, 65) == DLS_ERR_SHAPE);
  EXPECT(draft(rnn(), 2, 4, fusion(nan)) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(1.f, INFINITY)) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(1.f, 0.3f, 0.3f, 0x100)) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), nullptr) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), off(5, 4)) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), (dls_dtype)5) == DLS_ERR_DTYPE);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), DLS_BF16, nullptr) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), DLS_BF16, (int32_t*)off(6, 1)) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), DLS_BF16, (int32_t*)fake(6), nullptr) == DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), DLS_BF16, (int32_t*)fake(6), (int32_t*)fake(7), fake(9), 16) ==
         DLS_ERR_WORKSPACE);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), DLS_BF16, (int32_t*)fake(6), (int32_t*)fake(7), nullptr) ==
         DLS_ERR_ARG);
  EXPECT(draft(rnn(), 2, 4, fusion(), fake(5), DLS_BF16, (int32_t*)fake(6), (int32_t*)fake(7), off(9, 16)) ==
         DLS_ERR_ARG);
  dls_local_head m = markov(1000, 12);
  EXPECT(draft(m) == DLS_ERR_SHAPE);
  EXPECT(dls_draft_block(nullptr, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(), (int32_t*)fake(7),
                         nullptr, fake(9), 1 << 30, nullptr) == DLS_ERR_ARG);
  // empty work is a no-op even with NULL pointers
  EXPECT(draft(rnn(), 0, 4, fusion(), nullptr, DLS_BF16, nullptr, nullptr) == DLS_OK);
  EXPECT(draft(rnn(), 2, 0, fusion(), nullptr, DLS_BF16, nullptr, nullptr) == DLS_OK);

  // schedules, sampling and the adaptive rule
  std::vector<float> al(4, 0.5f), be(4, 0.1f);
  al[3] = nan;
  dls_local_head r = rnn();
  EXPECT(dls_draft_block_scheduled(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                   dls_fusion_schedule{al.data(), be.data()}, (int32_t*)fake(7), nullptr, fake(9),
                                   1 << 30, nullptr) == DLS_ERR_ARG);
  const float temps[] = {-1.f, nan, INFINITY, 1e-45f, 1e31f};
  for (float T : temps)
    EXPECT(dls_draft_block_sampled(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                   dls_fusion_schedule{nullptr, nullptr}, dls_sampling{T, 0u, 7ull},
                                   (int32_t*)fake(7), nullptr, fake(9), 1 << 30, nullptr) == DLS_ERR_ARG);
  EXPECT(dls_draft_block_sampled(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                 dls_fusion_schedule{nullptr, nullptr}, dls_sampling{1.f, 1u, 7ull}, (int32_t*)fake(7),
                                 nullptr, fake(9), 1 << 30, nullptr) == DLS_ERR_ARG);
  const dls_adaptive bad_rules[] = {{2, 0.f, 1.f, 0u}, {-1, 0.f, 1.f, 0u}, {0, 0.5f, 0.5f, 0u}, {1, 0.7f, 0.2f, 0u},
                                    {0, nan, 1.f, 0u}, {0, 0.f, INFINITY, 0u}, {0, 0.f, 1.f, 3u}};
  for (const dls_adaptive& ru : bad_rules) {
    EXPECT(dls_draft_block_adaptive(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                    dls_fusion_schedule{nullptr, nullptr}, dls_sampling{0.f, 0u, 0ull}, ru,
                                    (dls_row_uncertainty*)fake(10), (int32_t*)fake(7), nullptr, fake(9), 1 << 30,
                                    nullptr) == DLS_ERR_ARG);
    EXPECT(dls_long_uncertainty(fake(0), DLS_BF16, 16, 151936, ru, (dls_row_uncertainty*)fake(1), fake(2), 1 << 24,
                                nullptr) == DLS_ERR_ARG);
  }
  const dls_adaptive good = {DLS_UNC_ENTROPY, 0.1f, 0.9f, 0u};
  EXPECT(dls_draft_block_adaptive(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                  dls_fusion_schedule{nullptr, nullptr}, dls_sampling{0.f, 0u, 0ull}, good, nullptr,
                                  (int32_t*)fake(7), nullptr, fake(9), 1 << 30, nullptr) == DLS_ERR_ARG);
  EXPECT(dls_long_uncertainty(fake(0), (dls_dtype)9, 16, 1000, good, (dls_row_uncertainty*)fake(1), fake(2), 1 << 24,
                              nullptr) == DLS_ERR_DTYPE);
  EXPECT(dls_long_uncertainty(fake(0), DLS_BF16, -1, 1000, good, (dls_row_uncertainty*)fake(1), fake(2), 1 << 24,
                              nullptr) == DLS_ERR_SHAPE);
  EXPECT(dls_long_uncertainty(fake(0), DLS_BF16, 16, 0, good, (dls_row_uncertainty*)fake(1), fake(2), 1 << 24,
                              nullptr) == DLS_ERR_SHAPE);
  EXPECT(dls_long_uncertainty(off(0, 4), DLS_BF16, 16, 1000, good, (dls_row_uncertainty*)fake(1), fake(2), 1 << 24,
                              nullptr) == DLS_ERR_ARG);
  EXPECT(dls_long_uncertainty(fake(0), DLS_BF16, 16, 151936, good, (dls_row_uncertainty*)fake(1), fake(2), 8,
                              nullptr) == DLS_ERR_WORKSPACE);
  EXPECT(dls_long_uncertainty(nullptr, DLS_BF16, 0, 1000, good, nullptr, nullptr, 0, nullptr) == DLS_OK);

  // allocation-free drafting: a call beyond the scratch array is refused before any device call
  dls_local_head big = rnn(1 << 24, 16384, 4096, 512);
  EXPECT(dls_draft_block_noalloc(&big, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 256, 64, fusion(),
                                 (int32_t*)fake(7), nullptr, nullptr) == DLS_ERR_WORKSPACE);
  EXPECT(dls_draft_block_error(fake(0), 1 << 20, nullptr, nullptr) == DLS_ERR_ARG);
  EXPECT(dls_draft_block_error(fake(0), 64, (int32_t*)fake(1), nullptr) == DLS_ERR_WORKSPACE);
  EXPECT(dls_draft_block_error(off(0, 16), 1 << 20, (int32_t*)fake(1), nullptr) == DLS_ERR_WORKSPACE);

  // combine, accept length, prior
  EXPECT(dls_combine_logits(fake(0), fake(1), (dls_dtype)3, nullptr, 4, 1000, fusion(), (int32_t*)fake(2), nullptr,
                            nullptr, fake(3), 1 << 20, nullptr) == DLS_ERR_DTYPE);
  EXPECT(dls_combine_logits(fake(0), fake(1), DLS_BF16, nullptr, -1, 1000, fusion(), (int32_t*)fake(2), nullptr,
                            nullptr, fake(3), 1 << 20, nullptr) == DLS_ERR_SHAPE);
  EXPECT(dls_combine_logits(fake(0), nullptr, DLS_BF16, nullptr, 4, 1000, fusion(), (int32_t*)fake(2), nullptr,
                            nullptr, fake(3), 1 << 20, nullptr) == DLS_ERR_ARG);
  EXPECT(dls_combine_logits(fake(0), fake(1), DLS_BF16, nullptr, 1 << 20, 1 << 24, fusion(), (int32_t*)fake(2),
                            nullptr, nullptr, fake(3), 16, nullptr) == DLS_ERR_WORKSPACE);
  EXPECT(dls_accept_len((int32_t*)fake(0), nullptr, 4, 16, (int32_t*)fake(2), nullptr) == DLS_ERR_ARG);
  EXPECT(dls_accept_len((int32_t*)fake(0), (int32_t*)fake(1), -4, 16, (int32_t*)fake(2), nullptr) == DLS_ERR_SHAPE);
  EXPECT(dls_unigram_log_prior((int32_t*)fake(0), 100, 0, 1.f, (uint64_t*)fake(1), (float*)fake(2), nullptr) ==
         DLS_ERR_SHAPE);
  EXPECT(dls_unigram_log_prior((int32_t*)fake(0), 100, 1000, nan, (uint64_t*)fake(1), (float*)fake(2), nullptr) ==
         DLS_ERR_ARG);
  dls_local_head r32 = rnn(1000, 64, 32, 32);
  EXPECT(dls_prepare_head(&r32, fake(11), 8, nullptr) == DLS_ERR_WORKSPACE);
  EXPECT(dls_prepare_head(&r, fake(11), (size_t)1 << 40, nullptr) == DLS_ERR_SHAPE);   // r = 16 cannot be prepared
  dls_local_head mk = markov(1000, 32);
  EXPECT(dls_prepare_head(&mk, nullptr, 1 << 30, nullptr) == DLS_ERR_ARG);
  EXPECT(dls_draft_block_path(&h, 2, 4, DLS_BF16, 0) == -1);
  EXPECT(dls_draft_block_path(&r, 0, 4, DLS_BF16, 0) == -1);
}

void size_queries() {
  // extremes of every size query: no overflow, no read past a table
  dls_local_head big = rnn(1 << 24, 16384, 4096, 512);
  EXPECT(dls_prepare_head_size(&big) == 0);   // r = 512 has no prepared form
  EXPECT(dls_draft_block_workspace_size(&big, 256, 64) > 0);
  dls_local_head big256 = rnn(1 << 24, 16384, 4096, 256);
  EXPECT(dls_prepare_head_size(&big256) > ((size_t)1 << 39));   // the folded table alone is 2^24 x 12288 x 4 B
  dls_local_head mk = markov(1 << 24, 256);
  EXPECT(dls_prepare_head_size(&mk) > 0);
  EXPECT(dls_draft_block_workspace_size(&mk, 256, 64) > 0);
  dls_local_head bad = rnn(0);
  EXPECT(dls_prepare_head_size(&bad) == 0);
  EXPECT(dls_draft_block_workspace_size(&bad, 1, 1) == 0);
  EXPECT(dls_draft_block_workspace_size(nullptr, 1, 1) == 0);
  EXPECT(dls_draft_block_workspace_size(&big, 0, 16) == 0);
  EXPECT(dls_combine_logits_workspace_size(1 << 20, 1 << 24) > 0);
  EXPECT(dls_combine_logits_workspace_size(1, 1) > 0);
  EXPECT(dls_combine_logits_workspace_size(0, 100) == 0);
  EXPECT(dls_long_uncertainty_workspace_size(1, 1 << 24) > 0);
  EXPECT(dls_long_uncertainty_workspace_size(1 << 24, 1 << 24) == 0);
  EXPECT(dls_long_uncertainty_workspace_size(-5, 100) == 0);
  EXPECT(dls_abi_version() == DLS_ABI_VERSION);
  for (int s = -2; s < 10; ++s) EXPECT(std::strlen(dls_status_string((dls_status)s)) > 0);
}

void valid_arguments_stop_at_device() {
  // on a host without a GPU every valid call ends at the device check
  EXPECT(draft(rnn()) == DLS_ERR_DEVICE);
  EXPECT(draft(markov()) == DLS_ERR_DEVICE);
  EXPECT(draft(rnn(), 2, 4, fusion(1.f, 0.3f, 0.3f, DLS_FIRST_ROW_LONG_ONLY | DLS_EXCLUSIVE_DEVICE), fake(5),
               DLS_BF16, nullptr) == DLS_ERR_DEVICE);
  dls_local_head r = rnn();
  const dls_adaptive good = {DLS_UNC_MAXPROB, -0.5f, 0.5f, 0u};
  EXPECT(dls_draft_block_adaptive(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                  dls_fusion_schedule{nullptr, nullptr}, dls_sampling{1.f, 0u, 9ull}, good,
                                  (dls_row_uncertainty*)fake(10), (int32_t*)fake(7), nullptr, fake(9), 1 << 30,
                                  nullptr) == DLS_ERR_DEVICE);
  EXPECT(dls_long_uncertainty(fake(0), DLS_F32, 16, 151936, good, (dls_row_uncertainty*)fake(1), fake(2), 1 << 24,
                              nullptr) == DLS_ERR_DEVICE);
  EXPECT(dls_draft_block_noalloc(&r, fake(5), DLS_BF16, (int32_t*)fake(6), nullptr, 2, 4, fusion(),
                                 (int32_t*)fake(7), nullptr, nullptr) == DLS_ERR_DEVICE);
  EXPECT(dls_draft_block_error(nullptr, 0, (int32_t*)fake(1), nullptr) == DLS_ERR_DEVICE);
  EXPECT(dls_combine_logits(fake(0), fake(1), DLS_BF16, nullptr, 4, 1000, fusion(), (int32_t*)fake(2), nullptr,
                            nullptr, fake(3), 1 << 20, nullptr) == DLS_ERR_DEVICE);
  EXPECT(dls_accept_len((int32_t*)fake(0), (int32_t*)fake(1), 4, 16, (int32_t*)fake(2), nullptr) == DLS_ERR_DEVICE);
  dls_local_head r32 = rnn(1000, 64, 32, 32);
  EXPECT(dls_prepare_head(&r32, fake(11), (size_t)1 << 40, nullptr) == DLS_ERR_DEVICE);
  EXPECT(dls_draft_block_path(&r, 2, 4, DLS_BF16, 0) == 0);   // not prepared: no device needed
}

void per_thread_errors() {
  // each thread fails with its own shape and must read back its own message
  std::vector<std::thread> ts;
  std::vector<int> bad(8, 0);
  for (int t = 0; t < 8; ++t) {
    ts.emplace_back([t, &bad] {
      for (int i = 0; i < 2000; ++i) {
        const int batch = 300 + t;
        dls_local_head h = rnn();
        dls_status s = draft(h, batch);
        const std::string msg = dls_last_error();
        if (s != DLS_ERR_SHAPE || msg.find(std::to_string(batch)) == std::string::npos) ++bad[t];
      }
    });
  }
  for (auto& th : ts) th.join();
  for (int t = 0; t < 8; ++t) EXPECT(bad[t] == 0);
}

}  // namespace

int main(int argc, char** argv) {
  const bool valid = !(argc > 1 && std::strcmp(argv[1], "--no-valid") == 0);
  rejected_arguments();
  size_queries();
  per_thread_errors();
  if (valid) valid_arguments_stop_at_device();
  std::printf("host driver: %d failed expectations\n", g_fail);
  return g_fail == 0 ? 0 : 1;
}
