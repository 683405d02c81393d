// TOP-B selection (Algorithm 1, last step), its complement (the evicted
// positions, for caches refilled in place) and the retained-cache gather
// Z_C = {(k_i, v_i)}_{i in C} (Sec. 3.1).
//
// Selection is exact integer work on order-preserving 32-bit keys of the fp32
// scores (NaN -> 0, the lowest key; -0 -> +0): the budget-th largest key T,
// then every token with key > T and the lowest-position tokens with key == T,
// written in ascending position order. One workgroup per unit, in one of two
// shapes (1024 threads with 8192-entry lists, or 256 threads with 1024-entry
// lists for batches of many units with small effective budgets).
//
// Fast path (sample select): keys of a fixed sample of the unit (up to 128
// blocks of 64 contiguous tokens, evenly spaced; 32 in the narrow shape)
// bracket T between two sample
// order statistics lo <= T <= hi. One ordered pass over the scores then
// collects, in position order, the tokens with key > hi (kept for sure) and
// the band lo <= key <= hi (candidates) into LDS; T and the emission are
// finished in LDS. The pass checks that the bracket holds (fewer than budget
// tokens above hi, at least budget at or above lo) and that both lists fit;
// otherwise the unit takes the general path: a three-pass radix select over
// the scores (11 + 11 + 10 bits, MSB first) and an ordered emission pass.
// Both paths give the same, deterministic result.
#include <algorithm>

#include "jacap_internal.hpp"


namespace jacap {

// Launch shape of the selection: THREADS per workgroup, CAP entries in each
// LDS list. The wide shape (one unit per CU) serves few long units; the
// narrow one fits several workgroups per CU for many units with small
// effective budgets.
template <int THREADS, int CAP>
struct SelCfg {
  static constexpr int kThreads = THREADS;
  static constexpr int kPer = 8;                   // tokens per thread per staged chunk
  static constexpr int kChunk = kPer * THREADS;    // scores per staged chunk
  static constexpr int kCand = CAP;                // candidate band capacity
  static constexpr int kSure = CAP;                // kept-for-sure list capacity
  static constexpr int kSample = kChunk / 64;      // sample: <= kSample blocks of 64 tokens
};
using SelWide = SelCfg<1024, 8192>;   // 141 KB of LDS: one workgroup per CU
using SelNarrow = SelCfg<256, 1024>;  // 29 KB: five per CU
// Batches of at least this many units take the narrow shape when no unit
// ranks more than half its list capacity.
constexpr int kSelNarrowUnits = 1024;

__device__ __forceinline__ uint32_t score_key(float f) {
  if (f != f) return 0u;          // NaN ranks lowest
  if (f == 0.0f) f = 0.0f;        // -0 == +0
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

template <class C>
struct SelShared {
  // staged chunk keys (one pad word per 8: the per-thread reads of 8
  // consecutive keys are then bank-conflict free) / sample keys / kept
  // candidate positions / evicted positions
  uint32_t stage[C::kChunk + C::kChunk / 8];
  uint32_t ckey[C::kCand];    // candidate keys (position order)
  int32_t cpos[C::kCand];     // candidate positions
  int32_t gpos[C::kSure];     // kept-for-sure positions (position order)
  uint32_t hist[2048];
  uint32_t scan[C::kThreads / 64 + 1];
  uint32_t bc[2];
};

// Exclusive prefix sum over C::kThreads values (one per thread), fixed order:
// a wave scan, then every thread adds the totals of the waves before its own
// (broadcast LDS reads, no serial pass).
template <class C>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* sh, uint32_t& total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint32_t incl = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  __syncthreads();
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < C::kThreads / 64; ++w) {
    const uint32_t t = sh[w];
    before += w < wave ? t : 0u;
    all += t;
  }
  total = all;
  return before + incl - x;
}

// Radix select (11 + 11 + 10 bits, MSB first): the key of rank `rank`
// (1 = largest, rank <= cnt) among key_at(0 .. cnt-1); `need` = how many keys
// equal to it fall within the top `rank`.
template <class C, class KeyAt>
__device__ uint32_t radix_rank(KeyAt key_at, int cnt, uint32_t rank, SelShared<C>& sh,
                               uint32_t& need) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, pmask = 0u, remaining = rank;
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int shf = shifts[pass];
    const uint32_t nb = 1u << widths[pass];
    const uint32_t dmask = nb - 1u;
    for (uint32_t i = tid; i < nb; i += C::kThreads) sh.hist[i] = 0u;
    if (tid == 0) { sh.bc[0] = 0u; sh.bc[1] = 0u; }
    __syncthreads();
    for (int i = tid; i < cnt; i += C::kThreads) {
      const uint32_t key = key_at(i);
      if ((key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shf) & dmask], 1u);
    }
    __syncthreads();
    // Suffix counts from the top digit down: each thread owns a contiguous run
    // of bins (descending digit order), then a block scan.
    const uint32_t per = nb / C::kThreads;  // bins per thread
    uint32_t local = 0;
    for (uint32_t q = 0; q < per; ++q) local += sh.hist[nb - 1 - (tid * per + q)];
    uint32_t tot;
    uint32_t above = block_exclusive_scan<C>(local, sh.scan, tot);
    for (uint32_t q = 0; q < per; ++q) {
      const uint32_t d = nb - 1 - (tid * per + q);
      const uint32_t c = sh.hist[d];
      if (above < remaining && remaining <= above + c) {
        sh.bc[0] = d;
        sh.bc[1] = above;
      }
      above += c;
    }
    __syncthreads();
    prefix |= sh.bc[0] << shf;
    pmask |= dmask << shf;
    remaining -= sh.bc[1];
    __syncthreads();
  }
  need = remaining;
  return prefix;
}

// General path: radix select over the scores, then an ordered emission pass
// over contiguous per-thread segments.
template <class C, class KeyAt>
__device__ void select_general(KeyAt key_at, int n, int kk, int32_t* out, SelShared<C>& sh) {
  const int tid = threadIdx.x;
  uint32_t need;
  const uint32_t T = radix_rank<C>(key_at, n, (uint32_t)kk, sh, need);
  const int seg = (n + C::kThreads - 1) / C::kThreads;
  const int lo = min(n, tid * seg), hi = min(n, lo + seg);
  uint32_t cgt = 0, ceq = 0;
  for (int i = lo; i < hi; ++i) {
    const uint32_t key = key_at(i);
    cgt += key > T;
    ceq += key == T;
  }
  uint32_t tot;
  uint32_t gt_before = block_exclusive_scan<C>(cgt, sh.scan, tot);
  uint32_t eq_before = block_exclusive_scan<C>(ceq, sh.scan, tot);
  for (int i = lo; i < hi; ++i) {
    const uint32_t key = key_at(i);
    if (key > T) {
      const uint32_t pos = gt_before + min(eq_before, need);
      if (pos < (uint32_t)kk) out[pos] = i;
      ++gt_before;
    } else if (key == T) {
      const uint32_t pos = gt_before + eq_before;
      if (eq_before < need && pos < (uint32_t)kk) out[pos] = i;
      ++eq_before;
    }
  }
}

// Number of entries of the ascending list a[0 .. cnt) that are < p.
__device__ __forceinline__ int lower_bound_lds(const int32_t* a, int cnt, int32_t p) {
  int lo = 0, hi = cnt;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < p) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// TOP-kk of key_at(0 .. n-1) by (key desc, position asc), written to out[0 ..
// kk) in ascending position order (0 < kk < n).
template <class C, class KeyAt, class RawAt, class Conv>
__device__ void select_unit(KeyAt key_at, RawAt raw_at, Conv conv, int n, int kk, int32_t* out,
                            SelShared<C>& sh) {
  static_assert(C::kCand <= C::kChunk + C::kChunk / 8, "kept candidates are merged from stage");
  static_assert(C::kSample * 64 <= C::kChunk, "the sample is staged in stage");
  const int tid = threadIdx.x;
  // Bracket [lo, hi] of T from the sample (the whole unit if it fits the band).
  uint32_t lo = 0u, hi = 0xFFFFFFFFu;
  if (n > C::kCand) {
    const int nb64 = (n + 63) / 64;
    const int q = (nb64 + C::kSample - 1) / C::kSample;  // every q-th 64-token block
    const int nsb = (nb64 + q - 1) / q;
    const int last_start = (nsb - 1) * q * 64;
    const int S = (nsb - 1) * 64 + min(64, n - last_start);   // valid samples form a prefix
    for (int j = tid; j < S; j += C::kThreads)
      sh.stage[j] = key_at((j >> 6) * q * 64 + (j & 63));
    __syncthreads();
    const double ks = (double)kk * (double)S / (double)n;
    const int delta = (int)(4.0 * sqrt(ks)) + 16;
    const int kr = max(1, (int)(ks + 0.5));
    const uint32_t r_lo = (uint32_t)min(S, kr + delta);
    uint32_t dummy;
    // When the band reaches the top of the sample there is no upper bound:
    // tokens above the sample maximum are candidates too.
    if (kr - delta >= 1)
      hi = radix_rank<C>([&](int i) { return sh.stage[i]; }, S, (uint32_t)(kr - delta), sh, dummy);
    lo = radix_rank<C>([&](int i) { return sh.stage[i]; }, S, r_lo, sh, dummy);
  }

  // One ordered pass: kept-for-sure (key > hi) and candidates (lo <= key <= hi).
  // Chunks of 8192 scores are loaded coalesced one chunk ahead (kept raw until
  // staged, so that no conversion waits on the loads early), staged in LDS
  // with a pad word per 8 keys, and read back as 8 consecutive keys per
  // thread (bank-conflict free); the block scan orders the threads' lists.
  auto pad = [](int e) { return e + (e >> 3); };
  float nxt[C::kPer];
  auto load_chunk = [&](int base) {
#pragma unroll
    for (int j = 0; j < C::kPer; ++j) nxt[j] = raw_at(min(base + j * C::kThreads + tid, n - 1));
  };
  load_chunk(0);
  uint32_t gcnt = 0, ccnt = 0;
  for (int base = 0; base < n; base += C::kChunk) {
#pragma unroll
    for (int j = 0; j < C::kPer; ++j) {
      const int p = base + j * C::kThreads + tid;
      sh.stage[pad(j * C::kThreads + tid)] = p < n ? conv(nxt[j]) : 0u;
    }
    if (base + C::kChunk < n) load_chunk(base + C::kChunk);  // uniform
    __syncthreads();
    uint32_t k8[C::kPer];
    uint32_t ng = 0, nc = 0;
#pragma unroll
    for (int qd = 0; qd < C::kPer; ++qd) {
      const int p = base + C::kPer * tid + qd;
      k8[qd] = sh.stage[pad(C::kPer * tid + qd)];
      const bool valid = p < n;
      ng += valid && k8[qd] > hi;
      nc += valid && k8[qd] >= lo && k8[qd] <= hi;
    }
    uint32_t tot;
    const uint32_t off = block_exclusive_scan<C>((ng << 16) | nc, sh.scan, tot);
    uint32_t go = gcnt + (off >> 16), co = ccnt + (off & 0xFFFFu);
#pragma unroll
    for (int qd = 0; qd < C::kPer; ++qd) {
      const int p = base + C::kPer * tid + qd;
      if (p >= n) continue;
      if (k8[qd] > hi) {
        if (go < (uint32_t)C::kSure) sh.gpos[go] = p;
        ++go;
      } else if (k8[qd] >= lo) {
        if (co < (uint32_t)C::kCand) { sh.ckey[co] = k8[qd]; sh.cpos[co] = p; }
        ++co;
      }
    }
    gcnt += tot >> 16;
    ccnt += tot & 0xFFFFu;
    __syncthreads();
  }
  const bool ok = gcnt < (uint32_t)kk && gcnt + ccnt >= (uint32_t)kk &&
                  gcnt <= (uint32_t)C::kSure && ccnt <= (uint32_t)C::kCand;
  if (!ok) {  // uniform: every thread holds the same counts
    select_general<C>(key_at, n, kk, out, sh);
    return;
  }

  // T among the candidates: rank kk - gcnt.
  const uint32_t r = (uint32_t)kk - gcnt;
  uint32_t need;
  const uint32_t T = radix_rank<C>([&](int i) { return sh.ckey[i]; }, (int)ccnt, r, sh, need);
  // Kept candidates, in position order, into stage[0 .. r).
  const int per = ((int)ccnt + C::kThreads - 1) / C::kThreads;
  const int c0 = min((int)ccnt, tid * per), c1 = min((int)ccnt, c0 + per);
  uint32_t ceq = 0;
  for (int i = c0; i < c1; ++i) ceq += sh.ckey[i] == T;
  uint32_t tot;
  uint32_t eq_before = block_exclusive_scan<C>(ceq, sh.scan, tot);
  uint32_t csel = 0;
  for (int i = c0, e = eq_before; i < c1; ++i) {
    const uint32_t key = sh.ckey[i];
    if (key > T) ++csel;
    else if (key == T) { csel += (uint32_t)e < need; ++e; }
  }
  uint32_t sel_before = block_exclusive_scan<C>(csel, sh.scan, tot);
  for (int i = c0, e = eq_before; i < c1; ++i) {
    const uint32_t key = sh.ckey[i];
    bool keep = false;
    if (key > T) keep = true;
    else if (key == T) { keep = (uint32_t)e < need; ++e; }
    if (keep) sh.stage[sel_before++] = (uint32_t)sh.cpos[i];
  }
  __syncthreads();
  // Merge the two position-ordered lists into out[0 .. kk).
  const int32_t* kept_c = reinterpret_cast<const int32_t*>(sh.stage);
  for (int a = tid; a < (int)gcnt; a += C::kThreads) {
    const int32_t p = sh.gpos[a];
    out[a + lower_bound_lds(kept_c, (int)r, p)] = p;
  }
  for (int b = tid; b < (int)r; b += C::kThreads) {
    const int32_t p = kept_c[b];
    out[b + lower_bound_lds(sh.gpos, (int)gcnt, p)] = p;
  }
}

template <class C>
__global__ __launch_bounds__(C::kThreads) void select_kernel(Geo g, const float* __restrict__ scores,
                                                             int32_t* __restrict__ idx, int budget,
                                                             int protect) {
  __shared__ SelShared<C> sh;
  const int u = blockIdx.x, tid = threadIdx.x;
  const Unit un = decode_unit(g, u);
  int32_t* out = idx + (int64_t)u * budget;
  const int kk_all = min(budget, un.n);
  const float* s = scores + token_row(g, un);

  for (int j = kk_all + tid; j < budget; j += C::kThreads) out[j] = -1;
  if (kk_all == 0) return;
  // Protected tail: the last p positions are kept; the ranking fills the
  // remaining kk slots from positions 0 .. n-1 (n = n_b - p), whose indices
  // all precede the tail, so the tail simply follows them in idx.
  const int npro = min(protect, kk_all);
  const int n = un.n - npro, kk = kk_all - npro;
  for (int j = tid; j < npro; j += C::kThreads) out[kk + j] = n + j;
  if (kk == 0) return;
  if (kk == n) {
    for (int j = tid; j < n; j += C::kThreads) out[j] = j;
    return;
  }

  // Keeping more than half: select the n - kk tokens to evict instead (the
  // last n - kk of the order (key desc, position asc) are the first n - kk of
  // (~key desc, reversed position asc)), then emit every other position.
  const int m = n - kk;
  if (m < kk && m <= C::kChunk) {
    select_unit<C>([&](int i) { return ~score_key(s[n - 1 - i]); }, [&](int i) { return s[n - 1 - i]; },
                [](float f) { return ~score_key(f); }, n, m, out, sh);
    __syncthreads();  // out[0 .. m): evicted, as reversed positions ascending
    uint32_t* ev = sh.stage;
    for (int j = tid; j < m; j += C::kThreads) ev[j] = (uint32_t)(n - 1 - out[m - 1 - j]);
    __syncthreads();
    const int32_t* evs = reinterpret_cast<const int32_t*>(ev);
    for (int i = tid; i < n; i += C::kThreads) {
      const int c = lower_bound_lds(evs, m, i);
      if (c == m || evs[c] != i) out[i - c] = i;
    }
    return;
  }
  select_unit<C>([&](int i) { return score_key(s[i]); }, [&](int i) { return s[i]; },
              [](float f) { return score_key(f); }, n, kk, out, sh);
}

hipError_t launch_select(const Launch& L, const float* scores, int32_t* idx) {
  const Geo& g = L.geo;
  const int budget = L.cfg->budget_k;
  // The largest number of tokens any unit ranks: min(B, n - B) at the longest n.
  const int kmax = std::min(budget, std::max(0, g.maxn - budget));
  if (g.U >= kSelNarrowUnits && kmax <= SelNarrow::kCand / 2)
    select_kernel<SelNarrow><<<g.U, SelNarrow::kThreads, 0, L.stream>>>(g, scores, idx, budget,
                                                                        L.cfg->protect_last);
  else
    select_kernel<SelWide><<<g.U, SelWide::kThreads, 0, L.stream>>>(g, scores, idx, budget,
                                                                    L.cfg->protect_last);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Evicted slots: the positions of each unit that the selection does not keep,
// ascending, then -1 up to the list's capacity. The kept positions come
// ascending from select_kernel; an evicted position i goes to slot i - r,
// r = the number of kept positions below i. Workgroup (tile, unit) takes the
// positions [p0, p0 + kEvTile): two binary searches of the kept list bound the
// kept positions inside the tile, which are staged in LDS, and each thread
// places the positions p0 + tid, p0 + tid + kThreads, ... (consecutive
// threads write consecutive slots between kept positions). The tile also
// writes the -1 padding of the slots [p0, p0 + kEvTile) at or past n - kept,
// and the last tile every padding slot beyond.
// ---------------------------------------------------------------------------
constexpr int kEvTile = 4096;

__global__ __launch_bounds__(kThreads) void evicted_kernel(Geo g, const int32_t* __restrict__ kept,
                                                           int budget, int32_t* __restrict__ slots,
                                                           int cap) {
  const int u = blockIdx.y, tile = blockIdx.x, tid = threadIdx.x;
  const Unit un = decode_unit(g, u);
  const int n = un.n, kk = min(budget, n), ne = n - kk;
  const int32_t* kp = kept + (int64_t)u * budget;
  int32_t* out = slots + (int64_t)u * cap;
  const int p0 = tile * kEvTile;
  const int pad_hi = tile == (int)gridDim.x - 1 ? cap : min(cap, p0 + kEvTile);
  for (int j = max(ne, p0) + tid; j < pad_hi; j += kThreads) out[j] = -1;
  if (p0 >= n) return;
  const int p1 = min(n, p0 + kEvTile);
  __shared__ int32_t ks[kEvTile];
  __shared__ int bounds[2];
  if (tid < 2) bounds[tid] = lower_bound_lds(kp, kk, tid == 0 ? p0 : p1);
  __syncthreads();
  const int lo = bounds[0], cnt = bounds[1] - bounds[0];  // distinct positions: cnt <= kEvTile
  for (int j = tid; j < cnt; j += kThreads) ks[j] = kp[lo + j];
  __syncthreads();
  for (int i = p0 + tid; i < p1; i += kThreads) {
    const int r = lower_bound_lds(ks, cnt, i);
    if (r < cnt && ks[r] == i) continue;  // kept
    out[i - (lo + r)] = i;                // i - (lo + r) < ne for an evicted i
  }
}

hipError_t launch_select_evicted(const Launch& L, const float* scores, int32_t* slots, int cap) {
  const int budget = L.cfg->budget_k;
  int32_t* kept = ws_ptr<int32_t>(L.wsp, L.ws.kept);
  if (budget > 0) {
    const hipError_t e = launch_select(L, scores, kept);
    if (e != hipSuccess) return e;
  }
  const int tiles = std::max(1, (L.geo.maxn + kEvTile - 1) / kEvTile);
  evicted_kernel<<<dim3(tiles, L.geo.U), kThreads, 0, L.stream>>>(L.geo, kept, budget, slots, cap);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Gather: a workgroup copies `rows` consecutive kept rows of one unit; each
// thread moves one 16-byte piece of UNR rows of K and of V per trip (all
// loads issued before the stores). STREAM: non-temporal loads and stores, for
// copies much larger than the caches.
// ---------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool STREAM>
__device__ __forceinline__ u32x4 copy_load(const char* p) {
  if constexpr (STREAM) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  else return *reinterpret_cast<const u32x4*>(p);
}

template <bool STREAM>
__device__ __forceinline__ void copy_store(char* p, u32x4 x) {
  if constexpr (STREAM) __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(p));
  else *reinterpret_cast<u32x4*>(p) = x;
}

template <int ROWBYTES, bool STREAM>
__global__ __launch_bounds__(kThreads) void compact_kernel(Geo g, const int32_t* __restrict__ idx,
                                                           int budget, int rows, int esize,
                                                           const char* __restrict__ k,
                                                           const char* __restrict__ v,
                                                           char* __restrict__ ko,
                                                           char* __restrict__ vo) {
  constexpr int PIECES = ROWBYTES / 16;
  constexpr int RPT = kThreads / PIECES;  // rows per trip slice
  constexpr int UNR = 4;
  const int u = blockIdx.y;
  const int j0 = blockIdx.x * rows;
  const int jend = min(budget, j0 + rows);
  if (j0 >= jend) return;
  const Unit un = decode_unit(g, u);
  const int rr = threadIdx.x / PIECES, off = (threadIdx.x % PIECES) * 16;
  const char* kb = k + ((int64_t)un.l * g.ksl + (int64_t)un.h * g.ksh + un.t0 * g.kst) * esize + off;
  const char* vb = v + ((int64_t)un.l * g.vsl + (int64_t)un.h * g.vsh + un.t0 * g.vst) * esize + off;
  char* kob = ko + ((int64_t)un.b * g.oss + (int64_t)un.l * g.osl + (int64_t)un.h * g.osh) * esize + off;
  char* vob = vo + ((int64_t)un.b * g.oss + (int64_t)un.l * g.osl + (int64_t)un.h * g.osh) * esize + off;
  const int32_t* ix = idx + (int64_t)u * budget;
  const int64_t kst = g.kst * esize, vst = g.vst * esize, ost = g.osr * esize;
  for (int jb = j0; jb < jend; jb += UNR * RPT) {
    int32_t t[UNR];
#pragma unroll
    for (int q = 0; q < UNR; ++q) {
      const int j = jb + q * RPT + rr;
      t[q] = j < jend ? ix[j] : -1;
      if (t[q] >= un.n) t[q] = -1;  // a position outside the sequence
    }
    u32x4 a[UNR], b[UNR];
#pragma unroll
    for (int q = 0; q < UNR; ++q)
      if (t[q] >= 0) {
        a[q] = copy_load<STREAM>(kb + t[q] * kst);
        b[q] = copy_load<STREAM>(vb + t[q] * vst);
      }
#pragma unroll
    for (int q = 0; q < UNR; ++q)
      if (t[q] >= 0) {
        const int64_t j = jb + q * RPT + rr;
        copy_store<STREAM>(kob + j * ost, a[q]);
        copy_store<STREAM>(vob + j * ost, b[q]);
      }
  }
}

hipError_t launch_compact(const Launch& L, const int32_t* idx, const void* k, const void* v,
                          void* ko, void* vo) {
  const Geo& g = L.geo;
  const int budget = L.cfg->budget_k;
  if (budget == 0) return hipSuccess;
  const int esize = L.cfg->dtype == JACAP_DTYPE_BF16 ? 2 : 4;
  const int rowbytes = g.D * esize;
  // Rows per workgroup: 64 .. 1024, the most that keep >= 8192 workgroups.
  int rows = 64;
  while (rows < 1024 && (int64_t)g.U * ((budget + 2 * rows - 1) / (2 * rows)) >= 8192) rows *= 2;
  const dim3 grid((unsigned)((budget + rows - 1) / rows), g.U);
  auto go = [&](auto kern) {
    kern<<<grid, kThreads, 0, L.stream>>>(g, idx, budget, rows, esize, (const char*)k,
                                          (const char*)v, (char*)ko, (char*)vo);
  };
  // Non-temporal above 1 GiB of kept rows (K and V), far beyond L2 and MALL.
  const bool stream = 2 * (int64_t)g.U * budget * rowbytes > (int64_t(1) << 30);
  switch (rowbytes * 2 + (stream ? 1 : 0)) {
    case 256: go(compact_kernel<128, false>); break;
    case 257: go(compact_kernel<128, true>); break;
    case 512: go(compact_kernel<256, false>); break;
    case 513: go(compact_kernel<256, true>); break;
    case 1024: go(compact_kernel<512, false>); break;
    case 1025: go(compact_kernel<512, true>); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace jacap
