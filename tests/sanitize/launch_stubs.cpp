// Host-only stand-ins for the kernel launchers, the phase timer and the two
// HIP runtime calls of the C-ABI host layer, so that jacap_host.hip can be
// built with AddressSanitizer / UndefinedBehaviorSanitizer and driven on a
// machine without a GPU. Each launcher records that it was called (and with
// which workspace geometry) instead of enqueueing a kernel.
#include "jacap_internal.hpp"
#include "stub_log.hpp"

namespace stub {
int calls[kNumLaunchers];
Launch last;
}  // namespace stub

namespace jacap {

static hipError_t note(int which, const Launch& L) {
  ++stub::calls[which];
  stub::last = {L.geo.U, L.geo.maxn, L.ws.total, L.ws.gchunks, L.ws.pchunks, L.ws.plchunks};
  return hipSuccess;
}

TimedPhase::TimedPhase(hipStream_t stream, int phase, bool) : stream_(stream), phase_(phase) {}
TimedPhase::~TimedPhase() {}

hipError_t launch_init(const Launch& L) { return note(stub::kInit, L); }
hipError_t launch_qstats(const Launch& L, const void*) { return note(stub::kQstats, L); }
hipError_t launch_stats_in(const Launch& L, const double*, const double*) { return note(stub::kStatsIn, L); }
hipError_t launch_kpass(const Launch& L, const void*, const void*) { return note(stub::kKpass, L); }
hipError_t launch_softmax_weights(const Launch& L) { return note(stub::kWeights, L); }
hipError_t launch_head_mean(const Launch& L, const float*, float*) { return note(stub::kHeadMean, L); }
hipError_t launch_gram(const Launch& L, const void*, bool) { return note(stub::kGram, L); }
hipError_t launch_gram_reduce(const Launch& L) { return note(stub::kGramReduce, L); }
hipError_t launch_factor(const Launch& L, bool) { return note(stub::kFactor, L); }
hipError_t launch_leverage(const Launch& L, const void*, float*) { return note(stub::kLeverage, L); }
hipError_t launch_leverage_precise(const Launch& L, const void*, float*) { return note(stub::kLeveragePrecise, L); }
hipError_t launch_select(const Launch& L, const float*, int32_t*) { return note(stub::kSelect, L); }
hipError_t launch_select_evicted(const Launch& L, const float*, int32_t*, int) { return note(stub::kSelectEvicted, L); }
hipError_t launch_compact(const Launch& L, const int32_t*, const void*, const void*, void*, void*) { return note(stub::kCompact, L); }
hipError_t launch_greedy(const Launch& L, const void*, int32_t*, int32_t*, double*) { return note(stub::kGreedy, L); }

}  // namespace jacap

// The read-back of jacap_read_status: the "device" status word is host memory here.
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind, hipStream_t) {
  memcpy(dst, src, bytes);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
