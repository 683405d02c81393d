// Call records of the launcher stand-ins (launch_stubs.cpp).
#pragma once
#include <stddef.h>
#include <string.h>

namespace stub {
enum {
  kInit, kQstats, kStatsIn, kKpass, kWeights, kHeadMean, kGram, kGramReduce, kFactor, kLeverage,
  kLeveragePrecise, kSelect, kSelectEvicted, kCompact, kGreedy, kNumLaunchers
};
struct Launch {
  int units, maxn;
  size_t ws_total;
  int gchunks, pchunks, plchunks;
};
extern int calls[kNumLaunchers];
extern Launch last;
inline void reset() { memset(calls, 0, sizeof(calls)); }
}  // namespace stub
