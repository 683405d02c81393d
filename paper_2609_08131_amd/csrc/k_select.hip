// TOP-B selection (Algorithm 1, last step) and the retained-cache gather
// Z_C = {(k_i, v_i)}_{i in C} (Sec. 3.1).
//
// Selection is exact integer work on order-preserving 32-bit keys of the fp32
// scores (NaN -> 0, the lowest key; -0 -> +0). A three-pass LDS radix select
// (11 + 11 + 10 bits, MSB first) finds the budget-th largest key T and how many
// tokens equal to T must be kept; a final ordered pass emits every token with
// key > T and the lowest-position tokens with key == T, in ascending position
// order, using block prefix sums over contiguous per-thread segments.
#include "jacap_internal.hpp"

namespace jacap {

constexpr int kSelThreads = 1024;

__device__ __forceinline__ uint32_t score_key(float f) {
  if (f != f) return 0u;          // NaN ranks lowest
  if (f == 0.0f) f = 0.0f;        // -0 == +0
  const uint32_t b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Exclusive prefix sum over kSelThreads values (one per thread), fixed order.
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
  if (tid == 0) {
    uint32_t run = 0;
    for (int i = 0; i < kSelThreads / 64; ++i) {
      const uint32_t t = sh[i];
      sh[i] = run;
      run += t;
    }
    sh[kSelThreads / 64] = run;
  }
  __syncthreads();
  total = sh[kSelThreads / 64];
  return sh[wave] + incl - x;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(Geo g, const float* __restrict__ scores,
                                                             int32_t* __restrict__ idx, int budget) {
  const int u = blockIdx.x, tid = threadIdx.x;
  const Unit un = decode_unit(g, u);
  int32_t* out = idx + (int64_t)u * budget;
  const int n = un.n;
  const int kk = min(budget, n);
  const float* s = scores + token_row(g, un);

  for (int j = kk + tid; j < budget; j += kSelThreads) out[j] = -1;
  if (kk == 0) return;
  if (kk == n) {
    for (int j = tid; j < n; j += kSelThreads) out[j] = j;
    return;
  }

  __shared__ uint32_t hist[2048];
  __shared__ uint32_t scan_sh[kSelThreads / 64 + 1];
  __shared__ uint32_t sel_digit, sel_above;

  uint32_t prefix = 0u, pmask = 0u;
  uint32_t remaining = (uint32_t)kk;  // rank (1-based) of T among keys matching the prefix
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass];
    const uint32_t nb = 1u << widths[pass];
    const uint32_t dmask = nb - 1u;
    for (uint32_t i = tid; i < nb; i += kSelThreads) hist[i] = 0u;
    if (tid == 0) { sel_digit = 0u; sel_above = 0u; }
    __syncthreads();
    for (int i = tid; i < n; i += kSelThreads) {
      const uint32_t key = score_key(s[i]);
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> sh) & dmask], 1u);
    }
    __syncthreads();
    // Suffix counts from the top digit down: each thread owns a contiguous run
    // of bins (descending digit order), then a block scan.
    const uint32_t per = nb / kSelThreads;  // 2 or 1
    uint32_t local = 0;
    for (uint32_t q = 0; q < per; ++q) local += hist[nb - 1 - (tid * per + q)];
    uint32_t tot;
    uint32_t above = block_exclusive_scan(local, scan_sh, tot);
    for (uint32_t q = 0; q < per; ++q) {
      const uint32_t d = nb - 1 - (tid * per + q);
      const uint32_t c = hist[d];
      if (above < remaining && remaining <= above + c) {
        sel_digit = d;
        sel_above = above;
      }
      above += c;
    }
    __syncthreads();
    prefix |= sel_digit << sh;
    pmask |= dmask << sh;
    remaining -= sel_above;
    __syncthreads();
  }
  const uint32_t T = prefix;
  const uint32_t need = remaining;  // tokens with key == T to keep, lowest positions first

  // Ordered emission over contiguous segments.
  const int seg = (n + kSelThreads - 1) / kSelThreads;
  const int lo = min(n, tid * seg), hi = min(n, lo + seg);
  uint32_t cgt = 0, ceq = 0;
  for (int i = lo; i < hi; ++i) {
    const uint32_t key = score_key(s[i]);
    cgt += key > T;
    ceq += key == T;
  }
  uint32_t tot;
  uint32_t gt_before = block_exclusive_scan(cgt, scan_sh, tot);
  uint32_t eq_before = block_exclusive_scan(ceq, scan_sh, tot);
  for (int i = lo; i < hi; ++i) {
    const uint32_t key = score_key(s[i]);
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

hipError_t launch_select(const Launch& L, const float* scores, int32_t* idx) {
  select_kernel<<<L.geo.U, kSelThreads, 0, L.stream>>>(L.geo, scores, idx, L.cfg->budget_k);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Gather: each thread copies one 16-byte piece of a kept K row and V row.
// ---------------------------------------------------------------------------
template <int ROWBYTES>
__global__ __launch_bounds__(kThreads) void compact_kernel(Geo g, const int32_t* __restrict__ idx,
                                                           int budget, int esize,
                                                           const char* __restrict__ k,
                                                           const char* __restrict__ v,
                                                           char* __restrict__ ko,
                                                           char* __restrict__ vo) {
  constexpr int PIECES = ROWBYTES / 16;
  const int u = blockIdx.y;
  const int e = blockIdx.x * kThreads + threadIdx.x;
  const int j = e / PIECES, piece = e % PIECES;
  if (j >= budget) return;
  const Unit un = decode_unit(g, u);
  const int32_t t = idx[(int64_t)u * budget + j];
  if (t < 0 || t >= un.n) return;  // padding (or a position outside the sequence)
  const int64_t src_k = ((int64_t)un.l * g.ksl + (int64_t)un.h * g.ksh + (un.t0 + t) * g.kst) * esize;
  const int64_t src_v = ((int64_t)un.l * g.vsl + (int64_t)un.h * g.vsh + (un.t0 + t) * g.vst) * esize;
  const int64_t dst = ((int64_t)un.b * g.oss + (int64_t)un.l * g.osl + (int64_t)un.h * g.osh +
                       (int64_t)j * g.osr) * esize;
  const int64_t off = piece * 16;
  *reinterpret_cast<uint4*>(ko + dst + off) = *reinterpret_cast<const uint4*>(k + src_k + off);
  *reinterpret_cast<uint4*>(vo + dst + off) = *reinterpret_cast<const uint4*>(v + src_v + off);
}

hipError_t launch_compact(const Launch& L, const int32_t* idx, const void* k, const void* v,
                          void* ko, void* vo) {
  const Geo& g = L.geo;
  const int budget = L.cfg->budget_k;
  if (budget == 0) return hipSuccess;
  const int esize = L.cfg->dtype == JACAP_DTYPE_BF16 ? 2 : 4;
  const int rowbytes = g.D * esize;
  const int64_t pieces = (int64_t)budget * (rowbytes / 16);
  const dim3 grid((unsigned)((pieces + kThreads - 1) / kThreads), g.U);
  auto go = [&](auto kern) {
    kern<<<grid, kThreads, 0, L.stream>>>(g, idx, budget, esize, (const char*)k, (const char*)v,
                                          (char*)ko, (char*)vo);
  };
  switch (rowbytes) {
    case 128: go(compact_kernel<128>); break;
    case 256: go(compact_kernel<256>); break;
    case 512: go(compact_kernel<512>); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace jacap
