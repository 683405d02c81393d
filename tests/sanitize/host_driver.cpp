// Drives the C-ABI host layer (argument validation, workspace layout, launch
// sequencing) built with AddressSanitizer and UndefinedBehaviorSanitizer
// against the launcher stand-ins of launch_stubs.cpp: no GPU is touched. Data
// pointers are only handed on to the stand-ins, except the workspace status
// word that jacap_read_status copies back. Exits non-zero on the first
// unexpected result (a sanitizer report aborts the run by itself).
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "jacap.h"
#include "stub_log.hpp"

static int failures = 0;
#define EXPECT(cond)                                                       \
  do {                                                                     \
    if (!(cond)) {                                                         \
      fprintf(stderr, "FAILED at line %d: %s\n", __LINE__, #cond);         \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

// Distinct, suitably aligned stand-ins for device pointers (never dereferenced).
static void* fake(uintptr_t slot) { return reinterpret_cast<void*>((slot + 1) << 20); }

struct Shape {
  int L, H, Hq, d, w, k, B;
  int64_t lens[16];
  int dtype, cov, gqa, ridge_mode, protect;
  float ridge;
};

static void fill(const Shape& s, jacap_config* c, jacap_batch* b, int32_t* offs) {
  memset(c, 0, sizeof(*c));
  memset(b, 0, sizeof(*b));
  c->num_layers = s.L;
  c->num_kv_heads = s.H;
  c->num_q_heads = s.Hq;
  c->head_dim = s.d;
  c->window = s.w;
  c->budget_k = s.k;
  c->temperature = 10.0f;
  c->ridge = s.ridge;
  c->cov_mode = s.cov;
  c->dtype = s.dtype;
  c->ridge_mode = s.ridge_mode;
  c->gqa_mode = s.gqa;
  c->protect_last = s.protect;
  int64_t T = 0, maxn = 0;
  offs[0] = 0;
  for (int i = 0; i < s.B; ++i) {
    T += s.lens[i];
    offs[i + 1] = (int32_t)T;
    if (s.lens[i] > maxn) maxn = s.lens[i];
  }
  b->num_seqs = s.B;
  b->max_seq_len = (int32_t)maxn;
  b->total_tokens = T;
  b->seq_offsets = offs;  // read by the kernels only
  b->k_stride_token = b->v_stride_token = s.d;
  b->k_stride_head = b->v_stride_head = T * s.d;
  b->k_stride_layer = b->v_stride_layer = T * s.d * s.H;
  b->q_stride_pos = s.d;
  b->q_stride_head = (int64_t)s.w * s.d;
  b->q_stride_layer = (int64_t)s.Hq * s.w * s.d;
  b->q_stride_seq = (int64_t)s.L * s.Hq * s.w * s.d;
  b->out_stride_row = s.d;
  b->out_stride_head = (int64_t)s.k * s.d;
  b->out_stride_layer = (int64_t)s.H * s.k * s.d;
  b->out_stride_seq = (int64_t)s.L * s.H * s.k * s.d;
  b->ridge_mat = s.ridge_mode == JACAP_RIDGE_MATRIX ? (const double*)fake(40) : nullptr;
}

// One valid problem through every entry point; checks the launch sequences.
static void run_valid(const Shape& s, const char* name) {
  jacap_config c;
  jacap_batch b;
  int32_t offs[17];
  fill(s, &c, &b, offs);
  size_t ws = 0;
  EXPECT(jacap_workspace_size(&c, &b, &ws) == JACAP_OK);
  EXPECT(ws > 0 && ws % 256 == 0);
  void* W = fake(1000);
  const bool bf = s.dtype == JACAP_DTYPE_BF16;
  const bool tokens = b.total_tokens > 0;

  stub::reset();
  EXPECT(jacap_score(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4), W, ws, nullptr) == JACAP_OK);
  if (tokens) {
    EXPECT(stub::calls[stub::kInit] == 1 && stub::calls[stub::kQstats] == 1);
    EXPECT(stub::calls[stub::kKpass] == 1 && stub::calls[stub::kWeights] == 1);
    EXPECT(stub::calls[stub::kGram] == (bf ? 2 : 1));
    // the reduce kernel only for units of more than four Gram chunks
    EXPECT(stub::calls[stub::kGramReduce] == ((bf ? stub::last.gchunks : stub::last.pchunks) > 4 ? 1 : 0));
    EXPECT(stub::calls[stub::kFactor] == (bf ? 2 : 1));
    EXPECT(stub::calls[stub::kLeverage] == 1);
    EXPECT(stub::calls[stub::kLeveragePrecise] == (bf ? 1 : 0));
    const bool per_head = s.gqa == JACAP_GQA_PER_HEAD && s.Hq > s.H;
    EXPECT(stub::calls[stub::kHeadMean] == (per_head ? 1 : 0));
    EXPECT(stub::last.ws_total <= ws);
  } else {
    EXPECT(stub::calls[stub::kInit] == 1 && stub::calls[stub::kGram] == 0);
  }

  stub::reset();
  EXPECT(jacap_evict(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4), (int32_t*)fake(5),
                     fake(6), fake(7), W, ws, nullptr) == JACAP_OK);
  EXPECT(stub::calls[stub::kSelect] == (s.k > 0 ? 1 : 0));
  EXPECT(stub::calls[stub::kCompact] == (s.k > 0 ? 1 : 0));

  stub::reset();
  const int32_t cap = b.max_seq_len > s.k ? b.max_seq_len - s.k : 0;
  EXPECT(jacap_evict_slots(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4), (int32_t*)fake(8),
                           cap, W, ws, nullptr) == JACAP_OK);
  EXPECT(stub::calls[stub::kSelectEvicted] == 1);
  EXPECT(jacap_evict_slots(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4), (int32_t*)fake(8),
                           cap - 1, W, ws, nullptr) == JACAP_ERR_INVALID_ARG);

  stub::reset();
  EXPECT(jacap_select(&c, &b, (const float*)fake(4), (int32_t*)fake(5), W, ws, nullptr) == JACAP_OK);
  EXPECT(jacap_compact(&c, &b, (const int32_t*)fake(5), fake(2), fake(3), fake(6), fake(7), nullptr) == JACAP_OK);

  // too small, or misaligned, workspaces enqueue nothing
  stub::reset();
  EXPECT(jacap_score(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4), W, ws - 1, nullptr) == JACAP_ERR_WORKSPACE);
  EXPECT(jacap_score(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4),
                     (char*)W + 16, ws, nullptr) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_score(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4), nullptr, 0, nullptr) == JACAP_ERR_INVALID_ARG);
  if (tokens) {
    EXPECT(jacap_score(&c, &b, nullptr, fake(2), fake(3), (float*)fake(4), W, ws, nullptr) == JACAP_ERR_INVALID_ARG);
    EXPECT(jacap_score(&c, &b, fake(1), (char*)fake(2) + 8, fake(3), (float*)fake(4), W, ws, nullptr) == JACAP_ERR_INVALID_ARG);
  }
  for (int i = 0; i < stub::kNumLaunchers; ++i) EXPECT(stub::calls[i] == 0);

  // Algorithm 1 from given statistics (pooled GQA only)
  stub::reset();
  const jacap_status fs = jacap_score_from_stats(&c, &b, (const double*)fake(9), (const double*)fake(10),
                                                 fake(2), fake(3), (float*)fake(4), W, ws, nullptr);
  if (s.gqa == JACAP_GQA_PER_HEAD && s.Hq > s.H) EXPECT(fs == JACAP_ERR_UNSUPPORTED);
  else EXPECT(fs == JACAP_OK && stub::calls[stub::kStatsIn] == (tokens ? 1 : 0));

  // greedy: scalar ridge > 0, pooled GQA
  size_t gws = 0;
  const jacap_status gs = jacap_greedy_workspace_size(&c, &b, &gws);
  const bool greedy_ok = s.ridge_mode == JACAP_RIDGE_SCALAR && s.ridge > 0.0f &&
                         !(s.gqa == JACAP_GQA_PER_HEAD && s.Hq > s.H) && b.max_seq_len <= 524288;
  EXPECT((gs == JACAP_OK) == greedy_ok);
  if (greedy_ok) {
    stub::reset();
    EXPECT(jacap_greedy(&c, &b, fake(1), fake(2), fake(3), (int32_t*)fake(5), (int32_t*)fake(11),
                        (double*)fake(12), fake(1001), gws, nullptr) == JACAP_OK);
    EXPECT(stub::calls[stub::kGreedy] == 1);
  }
  if (failures) fprintf(stderr, "  in %s\n", name);
}

// Host-detectable errors: each returns its code and enqueues nothing.
static void run_invalid() {
  Shape base = {2, 2, 4, 128, 8, 16, 2, {100, 3000}, JACAP_DTYPE_BF16, JACAP_COV_DIAG,
                JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 1.0f};
  jacap_config c;
  jacap_batch b;
  int32_t offs[17];
  size_t ws = 0;
  auto check = [&](jacap_status want, int line) {
    stub::reset();
    size_t w2 = 0;
    const jacap_status got = jacap_workspace_size(&c, &b, &w2);
    const jacap_status got2 = jacap_score(&c, &b, fake(1), fake(2), fake(3), (float*)fake(4),
                                          fake(1000), (size_t)1 << 40, nullptr);
    for (int i = 0; i < stub::kNumLaunchers && want != JACAP_OK; ++i)
      if (stub::calls[i]) { fprintf(stderr, "launch on an invalid problem, line %d\n", line); ++failures; }
    if (got != want || got2 != want) {
      fprintf(stderr, "line %d: want %d got %d / %d\n", line, want, got, got2);
      ++failures;
    }
  };
#define CASE(want, mutate) do { fill(base, &c, &b, offs); mutate; check(want, __LINE__); } while (0)
  CASE(JACAP_OK, (void)0);
  CASE(JACAP_ERR_UNSUPPORTED, c.head_dim = 96);
  CASE(JACAP_ERR_UNSUPPORTED, c.head_dim = 256);
  CASE(JACAP_ERR_UNSUPPORTED, c.dtype = 7);
  CASE(JACAP_ERR_UNSUPPORTED, c.cov_mode = 2);
  CASE(JACAP_ERR_UNSUPPORTED, c.gqa_mode = -1);
  CASE(JACAP_ERR_UNSUPPORTED, c.ridge_mode = 5);
  CASE(JACAP_ERR_INVALID_ARG, c.num_q_heads = 5);
  CASE(JACAP_ERR_INVALID_ARG, c.num_layers = 0);
  CASE(JACAP_ERR_INVALID_ARG, c.window = 0);
  CASE(JACAP_ERR_INVALID_ARG, c.budget_k = -1);
  CASE(JACAP_ERR_INVALID_ARG, c.temperature = 0.0f);
  CASE(JACAP_ERR_INVALID_ARG, c.temperature = __builtin_nanf(""));
  CASE(JACAP_ERR_INVALID_ARG, c.ridge = -1.0f);
  CASE(JACAP_ERR_INVALID_ARG, c.ridge = __builtin_inff());
  CASE(JACAP_ERR_INVALID_ARG, c.protect_last = -3);
  CASE(JACAP_ERR_INVALID_ARG, b.num_seqs = 0);
  CASE(JACAP_ERR_INVALID_ARG, b.seq_offsets = nullptr);
  CASE(JACAP_ERR_INVALID_ARG, b.k_stride_token = 100);        // not a multiple of 8
  CASE(JACAP_ERR_INVALID_ARG, b.v_stride_token = 64);         // below head_dim
  CASE(JACAP_ERR_INVALID_ARG, b.q_stride_head = -8);
  CASE(JACAP_ERR_UNSUPPORTED, b.k_stride_token = ((int64_t)1 << 24) + 8);
  CASE(JACAP_ERR_INVALID_ARG, (c.ridge_mode = JACAP_RIDGE_MATRIX, b.ridge_mat = nullptr));
  CASE(JACAP_ERR_INVALID_ARG, (c.ridge_mode = JACAP_RIDGE_MATRIX, b.ridge_mat = (const double*)((char*)fake(3) + 4)));
  CASE(JACAP_ERR_UNSUPPORTED, (c.num_layers = 4096, c.num_kv_heads = 16, c.num_q_heads = 16));
  CASE(JACAP_ERR_UNSUPPORTED, b.total_tokens = (int64_t)INT32_MAX + 1);
  CASE(JACAP_ERR_UNSUPPORTED, (b.num_seqs = 16, c.num_layers = 64, c.num_kv_heads = 64,
                               c.num_q_heads = 64, b.max_seq_len = INT32_MAX));
  CASE(JACAP_ERR_UNSUPPORTED, (c.gqa_mode = JACAP_GQA_PER_HEAD, c.num_q_heads = 64,
                               b.num_seqs = 16, c.num_layers = 64, b.max_seq_len = 1 << 26));
  EXPECT(jacap_workspace_size(nullptr, &b, &ws) == JACAP_ERR_INVALID_ARG);
  fill(base, &c, &b, offs);
  EXPECT(jacap_workspace_size(&c, nullptr, &ws) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_workspace_size(&c, &b, nullptr) == JACAP_ERR_INVALID_ARG);
  // selection / compaction argument checks
  EXPECT(jacap_workspace_size(&c, &b, &ws) == JACAP_OK);
  EXPECT(jacap_select(&c, &b, (const float*)fake(4), nullptr, fake(1000), ws, nullptr) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_select(&c, &b, (const float*)((char*)fake(4) + 4), (int32_t*)fake(5), fake(1000), ws, nullptr) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_compact(&c, &b, nullptr, fake(2), fake(3), fake(6), fake(7), nullptr) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_compact(&c, &b, (const int32_t*)fake(5), nullptr, fake(3), fake(6), fake(7), nullptr) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_compact(&c, &b, (const int32_t*)fake(5), fake(2), fake(3), (char*)fake(6) + 2, fake(7), nullptr) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_select_evicted(&c, &b, (const float*)fake(4), (int32_t*)fake(8), 5000, nullptr, 0, nullptr) == JACAP_ERR_INVALID_ARG);
  // greedy's own conditions
  c.ridge = 0.0f;
  EXPECT(jacap_greedy_workspace_size(&c, &b, &ws) == JACAP_ERR_INVALID_ARG);
  c.ridge = 1.0f;
  c.gqa_mode = JACAP_GQA_PER_HEAD;
  EXPECT(jacap_greedy_workspace_size(&c, &b, &ws) == JACAP_ERR_UNSUPPORTED);
  c.gqa_mode = JACAP_GQA_POOLED;
  b.max_seq_len = 524289;
  EXPECT(jacap_greedy_workspace_size(&c, &b, &ws) == JACAP_ERR_UNSUPPORTED);
}

static void run_status() {
  // the status word is the first 4 bytes of the workspace (host memory here)
  void* ws = nullptr;
  EXPECT(posix_memalign(&ws, 256, 4096) == 0);
  memset(ws, 0, 4096);
  *(uint32_t*)ws = JACAP_FLAG_SINGULAR | JACAP_FLAG_NONFINITE;
  uint32_t flags = 0;
  EXPECT(jacap_read_status(ws, nullptr, &flags) == JACAP_OK);
  EXPECT(flags == (JACAP_FLAG_SINGULAR | JACAP_FLAG_NONFINITE));
  EXPECT(jacap_read_status(nullptr, nullptr, &flags) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_read_status((char*)ws + 16, nullptr, &flags) == JACAP_ERR_INVALID_ARG);
  EXPECT(jacap_read_status(ws, nullptr, nullptr) == JACAP_ERR_INVALID_ARG);
  free(ws);
  // every code, and values of the enum's range that name no code
  for (int s = 0; s <= 7; ++s) EXPECT(jacap_status_string((jacap_status)s) != nullptr);
  EXPECT(strcmp(jacap_status_string((jacap_status)7), "JACAP_ERR_UNKNOWN") == 0);
  EXPECT(strcmp(jacap_status_string(JACAP_ERR_WORKSPACE), "JACAP_ERR_WORKSPACE") == 0);
}

int main() {
  const Shape shapes[] = {
      // tiny fp32; one Llama layer; long128k; ragged lengths; per-head; FULL; W_O; token-free
      {1, 1, 1, 64, 16, 64, 1, {512}, JACAP_DTYPE_FP32, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 1.0f},
      {1, 8, 32, 128, 32, 512, 1, {8192}, JACAP_DTYPE_BF16, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 1.0f},
      {32, 8, 32, 128, 64, 1024, 1, {131072}, JACAP_DTYPE_BF16, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 1.0f},
      {32, 8, 32, 128, 32, 256, 16, {4096, 32768, 5000, 17, 0, 1, 255, 256, 257, 1000, 8193, 20000, 31000, 4097, 9999, 12345},
       JACAP_DTYPE_BF16, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 1.0f},
      {2, 2, 8, 64, 4, 100, 3, {0, 900, 4000}, JACAP_DTYPE_FP32, JACAP_COV_FULL, JACAP_GQA_PER_HEAD, JACAP_RIDGE_SCALAR, 7, 0.0f},
      {4, 8, 32, 128, 64, 1024, 1, {131072}, JACAP_DTYPE_BF16, JACAP_COV_FULL, JACAP_GQA_PER_HEAD, JACAP_RIDGE_SCALAR, 64, 0.5f},
      {1, 2, 4, 128, 8, 32, 2, {300, 77}, JACAP_DTYPE_BF16, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_MATRIX, 0, 0.0f},
      {2, 2, 4, 64, 8, 16, 2, {0, 0}, JACAP_DTYPE_BF16, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 0.5f},
      {1, 1, 4, 128, 8, 0, 1, {2097152}, JACAP_DTYPE_BF16, JACAP_COV_DIAG, JACAP_GQA_POOLED, JACAP_RIDGE_SCALAR, 0, 1.0f},
  };
  int i = 0;
  for (const Shape& s : shapes) {
    char name[32];
    snprintf(name, sizeof(name), "shape %d", i++);
    run_valid(s, name);
  }
  run_invalid();
  run_status();
  if (failures) {
    fprintf(stderr, "%d failure(s)\n", failures);
    return 1;
  }
  printf("host layer ok under the sanitizers\n");
  return 0;
}
