// C-ABI entry points of libjacap.so: argument validation, workspace layout
// and the launch sequences of jacap_score / jacap_select / jacap_compact /
// jacap_evict. Host-detectable errors return before anything is enqueued.
#include <math.h>
#include <string.h>

#include <algorithm>

#include "jacap_internal.hpp"

using namespace jacap;

namespace {

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

jacap_status check_config(const jacap_config* c) {
  if (!c) return JACAP_ERR_INVALID_ARG;
  if (c->num_layers < 1 || c->num_kv_heads < 1 || c->num_q_heads < 1) return JACAP_ERR_INVALID_ARG;
  if (c->num_q_heads % c->num_kv_heads != 0) return JACAP_ERR_INVALID_ARG;
  if (c->window < 1 || c->budget_k < 0) return JACAP_ERR_INVALID_ARG;
  if (!(c->temperature > 0.0f) || !isfinite(c->temperature)) return JACAP_ERR_INVALID_ARG;
  if (!(c->ridge >= 0.0f) || !isfinite(c->ridge)) return JACAP_ERR_INVALID_ARG;
  if (c->head_dim != 64 && c->head_dim != 128) return JACAP_ERR_UNSUPPORTED;
  if (c->dtype != JACAP_DTYPE_FP32 && c->dtype != JACAP_DTYPE_BF16) return JACAP_ERR_UNSUPPORTED;
  if (c->cov_mode != JACAP_COV_DIAG && c->cov_mode != JACAP_COV_FULL) return JACAP_ERR_UNSUPPORTED;
  if (c->ridge_mode != JACAP_RIDGE_SCALAR && c->ridge_mode != JACAP_RIDGE_MATRIX) return JACAP_ERR_UNSUPPORTED;
  if (c->gqa_mode != JACAP_GQA_POOLED && c->gqa_mode != JACAP_GQA_PER_HEAD) return JACAP_ERR_UNSUPPORTED;
  if (c->protect_last < 0) return JACAP_ERR_INVALID_ARG;
  return JACAP_OK;
}

// Query heads scored apart per KV head: the group size with per-head GQA, else 1.
int64_t scored_heads(const jacap_config* c) {
  return c->gqa_mode == JACAP_GQA_PER_HEAD && c->num_q_heads > c->num_kv_heads
             ? c->num_q_heads / c->num_kv_heads
             : 1;
}

jacap_status check_batch(const jacap_config* c, const jacap_batch* b) {
  if (!b || !b->seq_offsets) return JACAP_ERR_INVALID_ARG;
  if (b->num_seqs < 1 || b->max_seq_len < 0 || b->total_tokens < 0) return JACAP_ERR_INVALID_ARG;
  if ((int64_t)b->num_seqs * c->num_layers * c->num_kv_heads > 65535) return JACAP_ERR_UNSUPPORTED;
  if (b->total_tokens > (int64_t)INT32_MAX) return JACAP_ERR_UNSUPPORTED;
  // The streaming kernels run one-dimensional grids of units x chunks (chunks
  // of at least 1024 tokens; per-head GQA scores every query head as a unit
  // and pads the grid by fewer than 8 units per head).
  const int64_t vh = scored_heads(c);
  if ((int64_t)b->num_seqs * c->num_layers * c->num_kv_heads * vh * ((b->max_seq_len + 1023) / 1024) +
          8 * vh > (int64_t)INT32_MAX)
    return JACAP_ERR_UNSUPPORTED;
  const int64_t st[] = {b->k_stride_layer, b->k_stride_head, b->k_stride_token,
                        b->v_stride_layer, b->v_stride_head, b->v_stride_token,
                        b->q_stride_seq, b->q_stride_layer, b->q_stride_head, b->q_stride_pos,
                        b->out_stride_seq, b->out_stride_layer, b->out_stride_head,
                        b->out_stride_row};
  for (int64_t s : st)
    if (s < 0 || (s % 8) != 0) return JACAP_ERR_INVALID_ARG;
  if (b->k_stride_token < c->head_dim || b->v_stride_token < c->head_dim) return JACAP_ERR_INVALID_ARG;
  // The streaming kernels address a step's rows with 32-bit byte offsets.
  if (b->k_stride_token > kMaxTokenStride || b->v_stride_token > kMaxTokenStride)
    return JACAP_ERR_UNSUPPORTED;
  if (b->q_stride_pos < c->head_dim || b->out_stride_row < c->head_dim) return JACAP_ERR_INVALID_ARG;
  if (c->ridge_mode == JACAP_RIDGE_MATRIX &&
      (!b->ridge_mat || (reinterpret_cast<uintptr_t>(b->ridge_mat) & 7u)))
    return JACAP_ERR_INVALID_ARG;
  return JACAP_OK;
}

// Workspace of jacap_score / _select / _evict, or (greedy) of jacap_greedy,
// which needs the weight buffers but none of the Gram / factor storage.
Workspace layout(const jacap_config* c, const jacap_batch* b, bool greedy = false) {
  Workspace w{};
  // Units and per-token rows: one per query head with per-head GQA.
  const int64_t V = greedy ? 1 : scored_heads(c);
  const int64_t U = (int64_t)b->num_seqs * c->num_layers * c->num_kv_heads * V;
  const int64_t D = c->head_dim;
  const int64_t LHT = (int64_t)c->num_layers * c->num_kv_heads * b->total_tokens * V;
  const int maxn = b->max_seq_len;
  w.mfma = c->dtype == JACAP_DTYPE_BF16;
  w.kchunks = (maxn + kKChunk - 1) / kKChunk;
  w.wchunks = (maxn + kWChunk - 1) / kWChunk;
  w.gchunk = w.mfma ? kGChunkMfma : kGChunkPrecise;
  // Larger chunks write and re-read fewer partials. The longest sequence is
  // cut into the fewest equal chunks (whole 128-token flush spans) that keep
  // kGramMinBlocks blocks in the grid and no chunk above kGChunkMfmaMax
  // tokens; chunks stay at least kGChunkMfma tokens.
  if (w.mfma && maxn > 0) {
    const int64_t span = kGramSpan;
    const int64_t nmin = (kGramMinBlocks + U - 1) / U;
    const int64_t nch = std::max(nmin, (int64_t)(maxn + kGChunkMfmaMax - 1) / kGChunkMfmaMax);
    const int64_t per = ((maxn + nch - 1) / nch + span - 1) / span * span;
    w.gchunk = (int)std::min<int64_t>(std::max<int64_t>(per, kGChunkMfma), kGChunkMfmaMax);
  }
  w.gchunks = (maxn + w.gchunk - 1) / w.gchunk;
  w.gparts = 1;
  // Leverage chunks: kLChunkMfma tokens, halved (down to kLChunkMfmaMin) while
  // the grid would have fewer than kLevMinBlocks blocks.
  w.lchunk = w.mfma ? kLChunkMfma : kLChunkPrecise;
  if (w.mfma)
    while (w.lchunk > kLChunkMfmaMin &&
           U * (int64_t)((maxn + w.lchunk - 1) / w.lchunk) < kLevMinBlocks)
      w.lchunk /= 2;
  w.lchunks = (maxn + w.lchunk - 1) / w.lchunk;
  // The fp64 Gram pass (every unit of fp32 keys; the units of bf16 keys that
  // need it): about kPrecisePartials partials per batch, so that its buffer
  // stays bounded at any unit count, and no chunk below kGChunkPrecise tokens
  // (whole 32-token steps).
  {
    const int64_t want = std::max<int64_t>(1, kPrecisePartials / std::max<int64_t>(U, 1));
    const int64_t most = std::max<int64_t>(1, (maxn + kGChunkPrecise - 1) / kGChunkPrecise);
    const int64_t np = std::min(want, most);
    const int64_t per = std::max<int64_t>(kGChunkPrecise, ((maxn + np - 1) / np + 31) / 32 * 32);
    w.pchunk = (int)per;
    w.pchunks = maxn > 0 ? (int)((maxn + per - 1) / per) : 0;
  }
  // fp64 leverage chunks: kLChunkRefine tokens for the marked bf16 units;
  // for fp32 inputs kLChunkPrecise, halved (down to kLChunkPreciseMin) while
  // the grid would have fewer than kLevMinBlocks blocks.
  w.plchunk = w.mfma ? kLChunkRefine : kLChunkPrecise;
  if (!w.mfma)
    while (w.plchunk > kLChunkPreciseMin &&
           U * (int64_t)((maxn + w.plchunk - 1) / w.plchunk) < kLevMinBlocks)
      w.plchunk /= 2;
  w.plchunks = (maxn + w.plchunk - 1) / w.plchunk;
  const int64_t NB = D / 16;
  const int64_t npair = NB * (NB + 1) / 2;
  const int64_t nlp = (NB / 2) * (NB / 2 + 1);
  const int64_t mfma_part_bytes = w.mfma ? U * (int64_t)w.gchunks * npair * 256 * 4 : 0;
  const int64_t fp64_part_bytes = U * (int64_t)w.pchunks * npair * 256 * 8;
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t r = o; o = align256(o + bytes); return r; };
  w.status = take(4);
  w.uflags = take(4 * U);
  w.mu = take(8 * U * D);
  w.lam = take(8 * U * D);
  w.lamfull = take(c->cov_mode == JACAP_COV_FULL ? 4 * U * D * D : 4);
  w.smax_m = take(4 * U);
  w.smax_z = take(8 * U);
  w.wscale = take(8 * U);
  w.z = take(4 * LHT);
  w.kappa = take(4 * LHT);
  w.cstat = take(8 * U * (int64_t)w.kchunks);
  w.wgt = take(4 * LHT);
  if (greedy) {
    const int64_t nblk = (maxn + 255) / 256;
    w.gc = take(8 * LHT);
    w.gst = take(4 * LHT);
    w.gent = take(sizeof(GreedyEntry) * U * nblk);
    // the factor of Lambda_Q on the FULL covariance's triangular K pass
    w.lfrag = take(w.mfma && c->cov_mode == JACAP_COV_FULL ? 2 * U * nlp * 2 * 64 * 8 : 8);
    w.total = o;
    return w;
  }
  w.hscore = take(V > 1 ? 4 * LHT : 4);
  w.kept = take(4 * (int64_t)b->num_seqs * c->num_layers * c->num_kv_heads * std::max(c->budget_k, 1));
  w.gram = take((size_t)std::max(mfma_part_bytes, fp64_part_bytes));
  w.gram_red = take(8 * U * npair * 256);
  w.lfrag = take(w.mfma ? 2 * U * nlp * 2 * 64 * 8 : 8);
  w.total = o;
  return w;
}

Geo make_geo(const jacap_config* c, const jacap_batch* b) {
  Geo g{};
  g.L = c->num_layers;
  g.H = c->num_kv_heads;
  g.Hq = c->num_q_heads;
  g.G = c->num_q_heads / c->num_kv_heads;
  g.D = c->head_dim;
  g.w = c->window;
  g.B = b->num_seqs;
  g.U = b->num_seqs * c->num_layers * c->num_kv_heads;
  g.V = 1;
  g.maxn = b->max_seq_len;
  g.T = b->total_tokens;
  g.seq_off = b->seq_offsets;
  g.ridge_mat = c->ridge_mode == JACAP_RIDGE_MATRIX ? b->ridge_mat : nullptr;
  g.ksl = b->k_stride_layer; g.ksh = b->k_stride_head; g.kst = b->k_stride_token;
  g.vsl = b->v_stride_layer; g.vsh = b->v_stride_head; g.vst = b->v_stride_token;
  g.qss = b->q_stride_seq; g.qsl = b->q_stride_layer; g.qsh = b->q_stride_head; g.qsp = b->q_stride_pos;
  g.oss = b->out_stride_seq; g.osl = b->out_stride_layer; g.osh = b->out_stride_head; g.osr = b->out_stride_row;
  return g;
}

// Extra conditions of jacap_greedy (after check_config / check_batch).
jacap_status check_greedy(const jacap_config* c, const jacap_batch* b) {
  if (c->ridge_mode != JACAP_RIDGE_SCALAR) return JACAP_ERR_UNSUPPORTED;
  if (!(c->ridge > 0.0f)) return JACAP_ERR_INVALID_ARG;
  if (c->gqa_mode == JACAP_GQA_PER_HEAD && c->num_q_heads > c->num_kv_heads) return JACAP_ERR_UNSUPPORTED;
  if (b->max_seq_len > kGreedyMaxLen) return JACAP_ERR_UNSUPPORTED;
  return JACAP_OK;
}

jacap_status prepare(const jacap_config* c, const jacap_batch* b, void* ws, size_t ws_bytes,
                     void* stream, Launch* L, bool greedy = false) {
  jacap_status s = check_config(c);
  if (s != JACAP_OK) return s;
  s = check_batch(c, b);
  if (s != JACAP_OK) return s;
  if (greedy) {
    s = check_greedy(c, b);
    if (s != JACAP_OK) return s;
  }
  L->cfg = c;
  L->geo = make_geo(c, b);
  L->ws = layout(c, b, greedy);
  L->wsp = static_cast<char*>(ws);
  L->stream = static_cast<hipStream_t>(stream);
  if (ws != nullptr || ws_bytes != 0) {
    if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return JACAP_ERR_INVALID_ARG;
    if (ws_bytes < L->ws.total) return JACAP_ERR_WORKSPACE;
  }
  return JACAP_OK;
}

#define JACAP_TRY(expr)                         \
  do {                                          \
    if ((expr) != hipSuccess) return JACAP_ERR_HIP; \
  } while (0)

// Runs `expr` inside a timed scope of phase `ph`.
#define JACAP_PHASE(ph, expr)               \
  do {                                      \
    TimedPhase tp_(L.stream, (ph), L.timed); \
    JACAP_TRY(expr);                        \
  } while (0)

// One scoring pass (Algorithm 1 steps 1-4) over every unit, from the window
// queries q, or (mu != nullptr) from caller-supplied statistics.
jacap_status score_pass(const Launch& L, const void* q, const void* k, const void* v,
                        float* scores, const double* mu = nullptr,
                        const double* lambda = nullptr) {
  JACAP_PHASE(JACAP_PHASE_INIT, launch_init(L));
  if (mu) JACAP_PHASE(JACAP_PHASE_QSTATS, launch_stats_in(L, mu, lambda));
  else JACAP_PHASE(JACAP_PHASE_QSTATS, launch_qstats(L, q));
  JACAP_PHASE(JACAP_PHASE_KPASS, launch_kpass(L, k, mu ? nullptr : q));
  JACAP_PHASE(JACAP_PHASE_WEIGHTS, launch_softmax_weights(L));
  JACAP_PHASE(JACAP_PHASE_GRAM, launch_gram(L, v, false));
  if (gram_reduced(L)) JACAP_PHASE(JACAP_PHASE_GRAM_REDUCE, launch_gram_reduce(L));
  JACAP_PHASE(JACAP_PHASE_FACTOR, launch_factor(L, false));
  if (L.ws.mfma) {  // the units marked by the factorisation, again in fp64
    TimedPhase tp(L.stream, JACAP_PHASE_REFINE, L.timed);
    JACAP_TRY(launch_gram(L, v, true));
    JACAP_TRY(launch_factor(L, true));  // sums the fp64 partials itself
    JACAP_TRY(launch_leverage_precise(L, v, scores));
  }
  JACAP_PHASE(JACAP_PHASE_LEVERAGE, launch_leverage(L, v, scores));
  return JACAP_OK;
}

jacap_status run_score(const Launch& L, const void* q, const void* k, const void* v, float* scores) {
  const int G = L.geo.G;
  if (scored_heads(L.cfg) == 1) return score_pass(L, q, k, v, scores);
  // Per-head GQA: every query head of a group is a unit of its own (own
  // statistics, weights and A; the G units of a KV head read its K and V rows
  // together), then the mean of the G score rows.
  Launch Lv = L;
  Lv.geo.V = G;
  Lv.geo.G = 1;
  Lv.geo.U = L.geo.U * G;
  float* hs = ws_ptr<float>(L.wsp, L.ws.hscore);
  const jacap_status s = score_pass(Lv, q, k, v, hs);
  if (s != JACAP_OK) return s;
  JACAP_TRY(launch_head_mean(L, hs, scores));
  return JACAP_OK;
}

// The evicted-slot lists: int32 [B][L][H][slot_cap], room for every eviction.
bool slots_ok(const jacap_config* c, const jacap_batch* b, const float* scores,
              const int32_t* slots, int32_t slot_cap) {
  if (!slots || !aligned16(slots) || (!scores && b->total_tokens > 0)) return false;
  if (scores && !aligned16(scores)) return false;
  return slot_cap >= 0 && slot_cap >= b->max_seq_len - c->budget_k;
}

// A data pointer: 16-byte aligned, and non-null unless the batch holds no
// tokens (the arrays are then empty and nothing reads them).
bool data_ptr_ok(const void* p, const jacap_batch* b) {
  return p ? aligned16(p) : b->total_tokens == 0;
}

bool score_ptrs_ok(const jacap_batch* b, const void* q, const void* k, const void* v,
                   const float* scores) {
  return data_ptr_ok(q, b) && data_ptr_ok(k, b) && data_ptr_ok(v, b) && data_ptr_ok(scores, b);
}

}  // namespace

namespace jacap {

jacap_status prepare_launch(const jacap_config* c, const jacap_batch* b, void* ws, size_t ws_bytes,
                            void* stream, Launch* L) {
  return prepare(c, b, ws, ws_bytes, stream, L);
}

jacap_status check_evict_ptrs(const jacap_config* c, const jacap_batch* b, const void* q,
                              const void* k, const void* v, const float* scores,
                              const int32_t* idx, const void* k_out, const void* v_out) {
  if (!score_ptrs_ok(b, q, k, v, scores)) return JACAP_ERR_INVALID_ARG;
  if (c->budget_k > 0) {
    if (!idx || !aligned16(idx)) return JACAP_ERR_INVALID_ARG;
    if (!data_ptr_ok(k_out, b) || !data_ptr_ok(v_out, b)) return JACAP_ERR_INVALID_ARG;
  }
  return JACAP_OK;
}

// Scoring, selection and compaction of a prepared problem, on L.stream.
jacap_status evict_prepared(const Launch& L, const void* q, const void* k, const void* v,
                            float* scores, int32_t* idx, void* k_out, void* v_out) {
  if (L.geo.T > 0) {
    const jacap_status s = run_score(L, q, k, v, scores);
    if (s != JACAP_OK) return s;
  } else {
    JACAP_PHASE(JACAP_PHASE_INIT, launch_init(L));
  }
  if (L.cfg->budget_k == 0) return JACAP_OK;
  JACAP_PHASE(JACAP_PHASE_SELECT, launch_select(L, scores, idx));
  JACAP_PHASE(JACAP_PHASE_COMPACT, launch_compact(L, idx, k, v, k_out, v_out));
  return JACAP_OK;
}

}  // namespace jacap

extern "C" {

jacap_status jacap_workspace_size(const jacap_config* cfg, const jacap_batch* batch, size_t* bytes) {
  if (!bytes) return JACAP_ERR_INVALID_ARG;
  jacap_status s = check_config(cfg);
  if (s != JACAP_OK) return s;
  s = check_batch(cfg, batch);
  if (s != JACAP_OK) return s;
  *bytes = layout(cfg, batch).total;
  return JACAP_OK;
}

jacap_status jacap_score(const jacap_config* cfg, const jacap_batch* batch, const void* q_win,
                         const void* k, const void* v, float* scores, void* ws, size_t ws_bytes,
                         void* stream) {
  Launch L;
  if (!ws) return JACAP_ERR_INVALID_ARG;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L);
  if (s != JACAP_OK) return s;
  if (!score_ptrs_ok(batch, q_win, k, v, scores)) return JACAP_ERR_INVALID_ARG;
  if (batch->total_tokens == 0) {
    TimedPhase tp(L.stream, JACAP_PHASE_INIT);
    return launch_init(L) == hipSuccess ? JACAP_OK : JACAP_ERR_HIP;
  }
  return run_score(L, q_win, k, v, scores);
}

jacap_status jacap_score_from_stats(const jacap_config* cfg, const jacap_batch* batch,
                                    const double* mu, const double* lambda, const void* k,
                                    const void* v, float* scores, void* ws, size_t ws_bytes,
                                    void* stream) {
  Launch L;
  if (!ws) return JACAP_ERR_INVALID_ARG;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L);
  if (s != JACAP_OK) return s;
  if (cfg->gqa_mode == JACAP_GQA_PER_HEAD && cfg->num_q_heads > cfg->num_kv_heads)
    return JACAP_ERR_UNSUPPORTED;
  if (!mu || !lambda || (reinterpret_cast<uintptr_t>(mu) & 7u) ||
      (reinterpret_cast<uintptr_t>(lambda) & 7u))
    return JACAP_ERR_INVALID_ARG;
  if (!data_ptr_ok(k, batch) || !data_ptr_ok(v, batch) || !data_ptr_ok(scores, batch))
    return JACAP_ERR_INVALID_ARG;
  if (batch->total_tokens == 0) {
    TimedPhase tp(L.stream, JACAP_PHASE_INIT);
    return launch_init(L) == hipSuccess ? JACAP_OK : JACAP_ERR_HIP;
  }
  return score_pass(L, nullptr, k, v, scores, mu, lambda);
}

jacap_status jacap_select(const jacap_config* cfg, const jacap_batch* batch, const float* scores,
                          int32_t* idx, void* ws, size_t ws_bytes, void* stream) {
  Launch L;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L);
  if (s != JACAP_OK) return s;
  if (cfg->budget_k == 0) return JACAP_OK;
  if (!idx || (!scores && batch->total_tokens > 0)) return JACAP_ERR_INVALID_ARG;
  if (!aligned16(idx) || (scores && !aligned16(scores))) return JACAP_ERR_INVALID_ARG;
  TimedPhase tp(L.stream, JACAP_PHASE_SELECT);
  return launch_select(L, scores, idx) == hipSuccess ? JACAP_OK : JACAP_ERR_HIP;
}

jacap_status jacap_select_evicted(const jacap_config* cfg, const jacap_batch* batch,
                                  const float* scores, int32_t* slots, int32_t slot_cap, void* ws,
                                  size_t ws_bytes, void* stream) {
  Launch L;
  if (!ws) return JACAP_ERR_INVALID_ARG;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L);
  if (s != JACAP_OK) return s;
  if (!slots_ok(cfg, batch, scores, slots, slot_cap)) return JACAP_ERR_INVALID_ARG;
  TimedPhase tp(L.stream, JACAP_PHASE_SELECT);
  return launch_select_evicted(L, scores, slots, slot_cap) == hipSuccess ? JACAP_OK : JACAP_ERR_HIP;
}

jacap_status jacap_compact(const jacap_config* cfg, const jacap_batch* batch, const int32_t* idx,
                           const void* k, const void* v, void* k_out, void* v_out, void* stream) {
  Launch L;
  jacap_status s = prepare(cfg, batch, nullptr, 0, stream, &L);
  if (s != JACAP_OK) return s;
  if (cfg->budget_k == 0) return JACAP_OK;
  if (!idx || !aligned16(idx)) return JACAP_ERR_INVALID_ARG;
  if (!data_ptr_ok(k, batch) || !data_ptr_ok(v, batch) || !data_ptr_ok(k_out, batch) ||
      !data_ptr_ok(v_out, batch))
    return JACAP_ERR_INVALID_ARG;
  TimedPhase tp(L.stream, JACAP_PHASE_COMPACT);
  return launch_compact(L, idx, k, v, k_out, v_out) == hipSuccess ? JACAP_OK : JACAP_ERR_HIP;
}

jacap_status jacap_evict(const jacap_config* cfg, const jacap_batch* batch, const void* q_win,
                         const void* k, const void* v, float* scores, int32_t* idx, void* k_out,
                         void* v_out, void* ws, size_t ws_bytes, void* stream) {
  Launch L;
  if (!ws) return JACAP_ERR_INVALID_ARG;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L);
  if (s != JACAP_OK) return s;
  s = jacap::check_evict_ptrs(cfg, batch, q_win, k, v, scores, idx, k_out, v_out);
  if (s != JACAP_OK) return s;
  return jacap::evict_prepared(L, q_win, k, v, scores, idx, k_out, v_out);
}

jacap_status jacap_evict_slots(const jacap_config* cfg, const jacap_batch* batch, const void* q_win,
                               const void* k, const void* v, float* scores, int32_t* slots,
                               int32_t slot_cap, void* ws, size_t ws_bytes, void* stream) {
  Launch L;
  if (!ws) return JACAP_ERR_INVALID_ARG;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L);
  if (s != JACAP_OK) return s;
  if (!score_ptrs_ok(batch, q_win, k, v, scores)) return JACAP_ERR_INVALID_ARG;
  if (!slots_ok(cfg, batch, scores, slots, slot_cap)) return JACAP_ERR_INVALID_ARG;
  if (batch->total_tokens > 0) {
    s = run_score(L, q_win, k, v, scores);
    if (s != JACAP_OK) return s;
  } else {
    JACAP_PHASE(JACAP_PHASE_INIT, launch_init(L));
  }
  JACAP_PHASE(JACAP_PHASE_SELECT, launch_select_evicted(L, scores, slots, slot_cap));
  return JACAP_OK;
}

jacap_status jacap_greedy_workspace_size(const jacap_config* cfg, const jacap_batch* batch,
                                         size_t* bytes) {
  if (!bytes) return JACAP_ERR_INVALID_ARG;
  jacap_status s = check_config(cfg);
  if (s != JACAP_OK) return s;
  s = check_batch(cfg, batch);
  if (s != JACAP_OK) return s;
  s = check_greedy(cfg, batch);
  if (s != JACAP_OK) return s;
  *bytes = layout(cfg, batch, true).total;
  return JACAP_OK;
}

jacap_status jacap_greedy(const jacap_config* cfg, const jacap_batch* batch, const void* q_win,
                          const void* k, const void* v, int32_t* idx, int32_t* order,
                          double* logdet, void* ws, size_t ws_bytes, void* stream) {
  Launch L;
  if (!ws) return JACAP_ERR_INVALID_ARG;
  jacap_status s = prepare(cfg, batch, ws, ws_bytes, stream, &L, true);
  if (s != JACAP_OK) return s;
  if (!data_ptr_ok(q_win, batch) || !data_ptr_ok(k, batch) || !data_ptr_ok(v, batch))
    return JACAP_ERR_INVALID_ARG;
  if (cfg->budget_k > 0 && (!idx || !aligned16(idx))) return JACAP_ERR_INVALID_ARG;
  if (order && !aligned16(order)) return JACAP_ERR_INVALID_ARG;
  if (logdet && (reinterpret_cast<uintptr_t>(logdet) & 7u)) return JACAP_ERR_INVALID_ARG;
  JACAP_PHASE(JACAP_PHASE_INIT, launch_init(L));
  if (batch->total_tokens > 0) {
    JACAP_PHASE(JACAP_PHASE_QSTATS, launch_qstats(L, q_win));
    JACAP_PHASE(JACAP_PHASE_KPASS, launch_kpass(L, k, q_win));
    JACAP_PHASE(JACAP_PHASE_WEIGHTS, launch_softmax_weights(L));
  }
  if (cfg->budget_k == 0 && !logdet) return JACAP_OK;
  JACAP_TRY(launch_greedy(L, v, idx, order, logdet));
  return JACAP_OK;
}

jacap_status jacap_read_status(const void* ws, void* stream, uint32_t* flags) {
  if (!ws || !flags || (reinterpret_cast<uintptr_t>(ws) & 255u)) return JACAP_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t host = 0;
  if (hipMemcpyAsync(&host, ws, sizeof(uint32_t), hipMemcpyDeviceToHost, st) != hipSuccess)
    return JACAP_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return JACAP_ERR_HIP;
  *flags = host;
  return JACAP_OK;
}

const char* jacap_status_string(jacap_status s) {
  switch (s) {
    case JACAP_OK: return "JACAP_OK";
    case JACAP_ERR_INVALID_ARG: return "JACAP_ERR_INVALID_ARG";
    case JACAP_ERR_UNSUPPORTED: return "JACAP_ERR_UNSUPPORTED";
    case JACAP_ERR_WORKSPACE: return "JACAP_ERR_WORKSPACE";
    case JACAP_ERR_HIP: return "JACAP_ERR_HIP";
  }
  return "JACAP_ERR_UNKNOWN";
}

}  // extern "C"
