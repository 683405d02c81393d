// Per-phase GPU timing with HIP events (the jacap_timing_* entry points).
#include <mutex>
#include <vector>

#include "jacap_internal.hpp"

namespace jacap {
namespace {

struct Record {
  int phase;
  hipEvent_t begin, end;
};

std::mutex g_mu;
uint32_t g_mask = 0;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

TimedPhase::TimedPhase(hipStream_t stream, int phase) : stream_(stream), phase_(phase) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!(g_mask & (1u << phase))) return;
  begin_ = take_event();
  end_ = take_event();
  if (!begin_ || !end_ || hipEventRecord(begin_, stream_) != hipSuccess) {
    if (begin_) g_pool.push_back(begin_);
    if (end_) g_pool.push_back(end_);
    begin_ = end_ = nullptr;
  }
}

TimedPhase::~TimedPhase() {
  if (!begin_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (hipEventRecord(end_, stream_) == hipSuccess) {
    g_records.push_back(Record{phase_, begin_, end_});
  } else {
    g_pool.push_back(begin_);
    g_pool.push_back(end_);
  }
}

}  // namespace jacap

extern "C" {

jacap_status jacap_timing_start(uint32_t phase_mask) {
  if (phase_mask >> JACAP_NUM_PHASES) return JACAP_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(jacap::g_mu);
  for (auto& r : jacap::g_records) {
    jacap::g_pool.push_back(r.begin);
    jacap::g_pool.push_back(r.end);
  }
  jacap::g_records.clear();
  jacap::g_mask = phase_mask;
  return JACAP_OK;
}

jacap_status jacap_timing_stop(double* ms, int32_t* calls) {
  std::lock_guard<std::mutex> lk(jacap::g_mu);
  jacap::g_mask = 0;
  double acc[JACAP_NUM_PHASES] = {};
  int32_t cnt[JACAP_NUM_PHASES] = {};
  bool ok = true;
  for (auto& r : jacap::g_records) {
    float t = 0.f;
    if (hipEventSynchronize(r.end) != hipSuccess || hipEventElapsedTime(&t, r.begin, r.end) != hipSuccess) {
      ok = false;
    } else {
      acc[r.phase] += (double)t;
      cnt[r.phase] += 1;
    }
    jacap::g_pool.push_back(r.begin);
    jacap::g_pool.push_back(r.end);
  }
  jacap::g_records.clear();
  for (int p = 0; p < JACAP_NUM_PHASES; ++p) {
    if (ms) ms[p] = acc[p];
    if (calls) calls[p] = cnt[p];
  }
  return ok ? JACAP_OK : JACAP_ERR_HIP;
}

const char* jacap_phase_name(int32_t phase) {
  static const char* names[JACAP_NUM_PHASES] = {"init", "qstats", "kpass", "weights", "gram",
                                                 "gram_reduce", "factor", "refine", "leverage",
                                                 "select", "compact", "greedy_init",
                                                 "greedy"};
  if (phase < 0 || phase >= JACAP_NUM_PHASES) return "unknown";
  return names[phase];
}

}  // extern "C"
