// Query statistics, centre-attention logits, query response and the global
// softmax normaliser (Algorithm 1, first two steps; Sec. 3.4).
#include <type_traits>

#include <algorithm>

#include "jacap_internal.hpp"

namespace jacap {

// Clears the sticky status word and the per-unit flags. A fill kernel rather
// than hipMemsetAsync so that the launch sequence can be captured in a graph.
__global__ void init_kernel(uint32_t* __restrict__ status, uint32_t* __restrict__ uflags, int U) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) status[0] = 0u;
  if (i < U) uflags[i] = 0u;
}

hipError_t launch_init(const Launch& L) {
  const int U = L.geo.U;
  init_kernel<<<(U + kThreads - 1) / kThreads, kThreads, 0, L.stream>>>(
      ws_ptr<uint32_t>(L.wsp, L.ws.status), ws_ptr<uint32_t>(L.wsp, L.ws.uflags), U);
  return hipGetLastError();
}

// Per-head GQA (the paper is single-head; each query head of a group is scored
// alone and a token's score is the mean over the group):
// scores[l][h][t] = (((s_0 + s_1) + s_2) + ... + s_{G-1}) / G in fp32, in head
// order, from the per-head rows hs[l][h][g][t].
__global__ void head_mean_kernel(const float* __restrict__ hs, float* __restrict__ out, int64_t T,
                                 int G, float inv) {
  const float* src = hs + (int64_t)blockIdx.y * G * T;
  float* dst = out + (int64_t)blockIdx.y * T;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < T; t += stride) {
    float acc = src[t];
    for (int g = 1; g < G; ++g) acc += src[(int64_t)g * T + t];
    dst[t] = acc * inv;
  }
}

hipError_t launch_head_mean(const Launch& L, const float* hs, float* scores) {
  const Geo& g = L.geo;
  const int lh = g.L * g.H;
  if (g.T == 0 || lh == 0) return hipSuccess;
  const int64_t xb = std::min<int64_t>((g.T + kThreads - 1) / kThreads, std::max(1, 8192 / lh));
  head_mean_kernel<<<dim3((unsigned)xb, lh), kThreads, 0, L.stream>>>(hs, scores, g.T, g.G,
                                                                      1.0f / (float)g.G);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// mu_Q and Lambda_Q of the pooled window (G query heads x w positions):
// sample mean and 1/N covariance, accumulated in fp64 in a fixed order.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void qstats_kernel(Geo g, const T* __restrict__ q,
                                                          double* __restrict__ mu_out,
                                                          double* __restrict__ lam_out,
                                                          float* __restrict__ lamfull, int full,
                                                          uint32_t* status, uint32_t* uflags) {
  const int u = blockIdx.x;
  const int tid = threadIdx.x;
  const Unit un = decode_unit(g, u);
  if (tid == 0 && un.n == 0 &&
      !offsets_ok(g, g.seq_off[un.b], g.seq_off[un.b + 1]))
    atomicOr(status, (uint32_t)JACAP_FLAG_BAD_OFFSETS);
  const int Ns = g.G * g.w;
  const T* qb = q + un.b * g.qss + un.l * g.qsl + (int64_t)(un.h * g.V + un.s) * g.G * g.qsh;
  // Thread (cl, rp): 16-byte piece cl of rows rp, rp + RP, ...; partial sums
  // are combined over rp in a fixed order through LDS (fp64).
  constexpr int VEC = 16 / sizeof(T);
  constexpr int CL = D / VEC;           // lanes per row
  constexpr int RP = kThreads / CL;     // row parts
  const int cl = tid % CL, rp = tid / CL;
  __shared__ double smu[D];
  __shared__ double part[RP][D];
  auto row_piece = [&](int r, double (&x)[VEC]) {
    const int gq = r / g.w, p = r - gq * g.w;
    const uint4 raw = *reinterpret_cast<const uint4*>(qb + gq * g.qsh + p * g.qsp + cl * VEC);
    const T* xv = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int e = 0; e < VEC; ++e) x[e] = (double)to_f32(xv[e]);
  };
  auto combine = [&](const double (&acc)[VEC], double* out) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) part[rp][cl * VEC + e] = acc[e];
    __syncthreads();
    if (tid < D) {
      double t = 0.0;
      for (int k = 0; k < RP; ++k) t += part[k][tid];
      out[tid] = t / Ns;
    }
    __syncthreads();
  };
  double acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.0;
  for (int r = rp; r < Ns; r += RP) {
    double x[VEC];
    row_piece(r, x);
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] += x[e];
  }
  combine(acc, smu);
  double m[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) { m[e] = smu[cl * VEC + e]; acc[e] = 0.0; }
  for (int r = rp; r < Ns; r += RP) {
    double x[VEC];
    row_piece(r, x);
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] += (x[e] - m[e]) * (x[e] - m[e]);
  }
  __shared__ double svar[D];
  combine(acc, svar);
  if (tid < D) {
    const double mm = smu[tid], v = svar[tid];
    mu_out[(int64_t)u * D + tid] = mm;
    lam_out[(int64_t)u * D + tid] = v;
    if (!isfinite(mm) || !isfinite(v)) raise_flags(status, uflags, u, kUnitNonfinite);
  }
  if (!full) return;
  // Full covariance: each thread owns D*D/kThreads entries; rows are staged,
  // centred, 32 at a time in LDS.
  constexpr int PER = D * D / kThreads;
  __shared__ double qt[32][D];
  double cacc[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) cacc[k] = 0.0;
  for (int r0 = 0; r0 < Ns; r0 += 32) {
    __syncthreads();
    for (int e = tid; e < 32 * D; e += kThreads) {
      const int rr = e / D, c = e - rr * D, r = r0 + rr;
      double x = 0.0;
      if (r < Ns) {
        const int gq = r / g.w, p = r - gq * g.w;
        x = (double)to_f32(qb[gq * g.qsh + p * g.qsp + c]) - smu[c];
      }
      qt[rr][c] = x;
    }
    __syncthreads();
    const int nr = min(32, Ns - r0);
    for (int rr = 0; rr < nr; ++rr) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int e = tid + k * kThreads;
        cacc[k] += qt[rr][e / D] * qt[rr][e % D];
      }
    }
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * kThreads;
    lamfull[(int64_t)u * D * D + e] = (float)(cacc[k] / Ns);
  }
}

hipError_t launch_qstats(const Launch& L, const void* q) {
  const Geo& g = L.geo;
  const int full = L.cfg->cov_mode == JACAP_COV_FULL && !full_kpass_on_mfma(L, q);
  double* mu = ws_ptr<double>(L.wsp, L.ws.mu);
  double* lam = ws_ptr<double>(L.wsp, L.ws.lam);
  float* lf = ws_ptr<float>(L.wsp, L.ws.lamfull);
  uint32_t* st = ws_ptr<uint32_t>(L.wsp, L.ws.status);
  uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  const bool bf = L.cfg->dtype == JACAP_DTYPE_BF16;
  if (g.D == 128) {
    if (bf)
      qstats_kernel<uint16_t, 128><<<g.U, kThreads, 0, L.stream>>>(g, (const uint16_t*)q, mu, lam, lf, full, st, uf);
    else
      qstats_kernel<float, 128><<<g.U, kThreads, 0, L.stream>>>(g, (const float*)q, mu, lam, lf, full, st, uf);
  } else {
    if (bf)
      qstats_kernel<uint16_t, 64><<<g.U, kThreads, 0, L.stream>>>(g, (const uint16_t*)q, mu, lam, lf, full, st, uf);
    else
      qstats_kernel<float, 64><<<g.U, kThreads, 0, L.stream>>>(g, (const float*)q, mu, lam, lf, full, st, uf);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess || !full_kpass_tri(L, q)) return e;
  return launch_qfactor(L, q);  // Lambda_Q and its factor for the K pass
}

// ---------------------------------------------------------------------------
// Caller-supplied (mu_Q, Lambda_Q) (Algorithm 1's inputs) into the places
// the window statistics take: mu and the diagonal in fp64, the full matrix
// rounded to fp32 for the K pass. One workgroup per unit.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void stats_in_kernel(Geo g, const double* __restrict__ mu,
                                                            const double* __restrict__ lambda,
                                                            int full, double* __restrict__ mu_out,
                                                            double* __restrict__ lam_out,
                                                            float* __restrict__ lamfull,
                                                            uint32_t* status, uint32_t* uflags) {
  const int u = blockIdx.x, tid = threadIdx.x, D = g.D;
  const Unit un = decode_unit(g, u);
  if (tid == 0 && un.n == 0 && !offsets_ok(g, g.seq_off[un.b], g.seq_off[un.b + 1]))
    atomicOr(status, (uint32_t)JACAP_FLAG_BAD_OFFSETS);
  bool bad = false;
  for (int c = tid; c < D; c += kThreads) {
    const double m = mu[(int64_t)u * D + c];
    const double l = full ? lambda[((int64_t)u * D + c) * D + c] : lambda[(int64_t)u * D + c];
    mu_out[(int64_t)u * D + c] = m;
    lam_out[(int64_t)u * D + c] = l;
    bad |= !isfinite(m) || !isfinite(l);
  }
  if (full)
    for (int e = tid; e < D * D; e += kThreads) {
      const double x = lambda[(int64_t)u * D * D + e];
      lamfull[(int64_t)u * D * D + e] = (float)x;
      bad |= !isfinite(x);
    }
  if (__any(bad) && (tid & 63) == 0) raise_flags(status, uflags, u, kUnitNonfinite);
}

hipError_t launch_stats_in(const Launch& L, const double* mu, const double* lambda) {
  const Geo& g = L.geo;
  stats_in_kernel<<<g.U, kThreads, 0, L.stream>>>(
      g, mu, lambda, L.cfg->cov_mode == JACAP_COV_FULL, ws_ptr<double>(L.wsp, L.ws.mu),
      ws_ptr<double>(L.wsp, L.ws.lam), ws_ptr<float>(L.wsp, L.ws.lamfull),
      ws_ptr<uint32_t>(L.wsp, L.ws.status), ws_ptr<uint32_t>(L.wsp, L.ws.uflags));
  return hipGetLastError();
}

// Sum over aligned groups of G lanes (G = 8, 16 or 32); every lane of a group
// ends with the same value. Within a 16-lane row the partners come from DPP
// (quad swaps, then the half-row and row mirrors: one VALU instruction per
// level); groups of 32 add one cross-row exchange.
template <int G, typename F>
__device__ __forceinline__ F group_sum(F v) {
  static_assert(G == 8 || G == 16 || G == 32, "group of 8, 16 or 32 lanes");
  if constexpr (sizeof(F) == 4) {
    v += dpp_f32<kDppQuadXor1>(v);
    v += dpp_f32<kDppQuadXor2>(v);
    v += dpp_f32<kDppHalfMirror>(v);
    if constexpr (G >= 16) v += dpp_f32<kDppMirror>(v);
  } else {
    v += dpp_f64<kDppQuadXor1>(v);
    v += dpp_f64<kDppQuadXor2>(v);
    v += dpp_f64<kDppHalfMirror>(v);
    if constexpr (G >= 16) v += dpp_f64<kDppMirror>(v);
  }
  if constexpr (G == 32) v += __shfl_xor(v, 16);
  return v;
}

// Chunk epilogue of the K pass: z and kappa of the chunk (staged in LDS) stored
// coalesced with one non-finite check, then the chunk's (max z, rest), rest =
// sum of exp(z - max + kRestShift) over every token but the first one holding
// the max (whose term is exactly 1). Kept apart from that 1, the rest keeps its
// own relative precision when one token dominates the softmax, which
// 1 - alpha of that token needs (it is the rest of Z over Z); the shift keeps
// its terms out of fp32's subnormal range.
__device__ __forceinline__ void kpass_epilogue(const Unit& un, int u, int base, int64_t trow,
                                               const float* zsh, const float* ksq, float* red,
                                               float* __restrict__ zout,
                                               float* __restrict__ kout,
                                               float2* __restrict__ cstat, int kchunks,
                                               uint32_t* status, uint32_t* uflags, int chunk) {
  const int tid = threadIdx.x;
  __syncthreads();
  bool bad = false;
  for (int tl = tid; tl < kKChunk; tl += kThreads) {
    const int i = base + tl;
    if (i < un.n) {
      const float z = zsh[tl], kq = ksq[tl];
      zout[trow + i] = z;
      kout[trow + i] = kq;
      bad |= !isfinite(z) || !isfinite(kq);
    }
  }
  if (__any(bad) && (threadIdx.x & 63) == 0) raise_flags(status, uflags, u, kUnitNonfinite);
  __syncthreads();
  static_assert(kKChunk % kThreads == 0, "whole logits per thread in the chunk reduction");
  constexpr int ZPT = kKChunk / kThreads;
  float zv[ZPT];
  float mloc = -INFINITY;
#pragma unroll
  for (int q = 0; q < ZPT; ++q) {
    zv[q] = zsh[q * kThreads + tid];
    mloc = fmaxf(mloc, zv[q]);
  }
  const float m = block_combine(wave_max(mloc), red, [](float a, float b) { return fmaxf(a, b); });
  int first = kKChunk;
#pragma unroll
  for (int q = ZPT - 1; q >= 0; --q)
    if (zv[q] == m) first = q * kThreads + tid;
  __shared__ int redi[kThreads / 64];
  first = block_combine(wave_min(first), redi, [](int a, int b) { return min(a, b); });
  float ex = 0.0f;
#pragma unroll
  for (int q = 0; q < ZPT; ++q)
    ex += (zv[q] == -INFINITY || q * kThreads + tid == first) ? 0.0f
                                                               : expf(zv[q] - m + kRestShift);
  const float s = block_combine(wave_sum(ex), red, [](float a, float b) { return a + b; });
  if (tid == 0) cstat[(int64_t)u * kchunks + chunk] = make_float2(m, s);
}

// ---------------------------------------------------------------------------
// K pass: z_i = k_i . mu / (tau sqrt d) and kappa_i = k_i^T Lambda k_i for a
// chunk of kKChunk tokens, then the chunk's (max z, sum exp(z - max)).
// One 16-byte load per lane: a token row is spread over LPT lanes.
// ---------------------------------------------------------------------------
template <typename T, int D, bool FULL>
__global__ __launch_bounds__(kThreads) void kpass_kernel(
    Geo g, const T* __restrict__ k, const double* __restrict__ mu, const double* __restrict__ lam,
    const float* __restrict__ lamfull, float* __restrict__ zout, float* __restrict__ kout,
    float2* __restrict__ cstat, int kchunks, double inv_scale, uint32_t* status,
    uint32_t* uflags) {
  int u, chunk;
  if (!grid_unit_chunk<false>(g, kchunks, u, chunk)) return;
  const Unit un = decode_unit(g, u);
  const int base = chunk * kKChunk;
  if (base >= un.n) return;

  constexpr int VEC = 16 / sizeof(T);
  constexpr int LPT = D / VEC;
  constexpr int TPW = 64 / LPT;
  constexpr int TPB = TPW * (kThreads / 64);
  using Acc = typename std::conditional<std::is_same<T, float>::value, double, float>::type;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane % LPT, tiw = lane / LPT;

  Acc muv[VEC], lamv[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    muv[e] = (Acc)mu[(int64_t)u * D + sub * VEC + e];
    lamv[e] = (Acc)lam[(int64_t)u * D + sub * VEC + e];
  }
  drain_vmem();  // keep these prologue loads out of the loop's wait counts

  __shared__ float zsh[kKChunk];
  __shared__ float ksq[kKChunk];
  __shared__ float red[kThreads / 64];
  __shared__ float lamsh[FULL ? D * (D + 1) : 1];
  __shared__ float ksh[FULL ? TPB : 1][FULL ? D : 1];
  if constexpr (FULL) {
    for (int e = tid; e < D * D; e += kThreads)
      lamsh[(e / D) * (D + 1) + (e % D)] = lamfull[(int64_t)u * D * D + e];
  }

  const T* kb = k + un.l * g.ksl + un.h * g.ksh;
  const int64_t trow = token_row(g, un);

  // UNR iterations per loop trip, their loads issued first (FULL mode keeps
  // one: it stages each token row in LDS between barriers).
  constexpr int UNR = FULL ? 1 : 4;
  static_assert(kKChunk % (UNR * TPB) == 0, "chunk must be whole unrolled trips");
  // Rows are loaded one trip ahead (double buffer); every load is
  // unconditional (past-the-end rows clamped, discarded) so the compiler's
  // wait counts stay static.
  auto load_trip = [&](int it0, uint4 (&raw)[UNR]) {
#pragma unroll
    for (int j = 0; j < UNR; ++j) {
      const int i = base + it0 + j * TPB + wave * TPW + tiw;
      const int ic = min(i, un.n - 1);
      raw[j] = *reinterpret_cast<const uint4*>(kb + (un.t0 + ic) * g.kst + sub * VEC);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  uint4 nxt[UNR];
  load_trip(0, nxt);
  for (int it0 = 0; it0 < kKChunk; it0 += UNR * TPB) {
    uint4 raw[UNR];
#pragma unroll
    for (int j = 0; j < UNR; ++j) raw[j] = nxt[j];
    load_trip(min(it0 + UNR * TPB, kKChunk - UNR * TPB), nxt);
#pragma unroll
    for (int j = 0; j < UNR; ++j) {
      const int tl = it0 + j * TPB + wave * TPW + tiw;
      const int i = base + tl;
      const bool valid = i < un.n;  // rows past the end were loaded clamped: finite, discarded
      Acc x[VEC];
      const T* xv = reinterpret_cast<const T*>(&raw[j]);
#pragma unroll
      for (int e = 0; e < VEC; ++e) x[e] = (Acc)to_f32(xv[e]);
      Acc dot = 0, kap = 0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) dot += muv[e] * x[e];
      if constexpr (!FULL) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) kap += lamv[e] * x[e] * x[e];
      } else {
        __syncthreads();
#pragma unroll
        for (int e = 0; e < VEC; ++e) ksh[wave * TPW + tiw][sub * VEC + e] = (float)x[e];
        __syncthreads();
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const float* row = lamsh + (sub * VEC + e) * (D + 1);
          Acc t = 0;
          for (int bb = 0; bb < D; ++bb) t += (Acc)row[bb] * (Acc)ksh[wave * TPW + tiw][bb];
          kap += x[e] * t;
        }
      }
      dot = group_sum<LPT>(dot);
      kap = group_sum<LPT>(kap);
      if (sub == 0) {
        zsh[tl] = valid ? (float)((double)dot * inv_scale) : -INFINITY;
        ksq[tl] = (float)kap;
      }
    }
  }
  kpass_epilogue(un, u, base, trow, zsh, ksq, red, zout, kout, cstat, kchunks, status, uflags,
                 chunk);
}

// K pass for bf16 keys, diagonal Lambda: four lanes per key row, each lane
// reading D/32 16-byte pieces (the four lanes of a row read 64 contiguous
// bytes per load), so a row's two sums need two quad DPP levels instead of
// four row levels per 16-byte load.
template <int D>
__global__ __launch_bounds__(kThreads) void kpass_quad_kernel(
    Geo g, const uint16_t* __restrict__ k, const double* __restrict__ mu,
    const double* __restrict__ lam, float* __restrict__ zout, float* __restrict__ kout,
    float2* __restrict__ cstat, int kchunks, double inv_scale, uint32_t* status,
    uint32_t* uflags) {
  int u, chunk;
  if (!grid_unit_chunk<false>(g, kchunks, u, chunk)) return;
  const Unit un = decode_unit(g, u);
  const int base = chunk * kKChunk;
  if (base >= un.n) return;

  constexpr int VEC = 8;                 // bf16 per 16-byte piece
  constexpr int LPT = 4;                 // lanes per token row
  constexpr int PIECES = D / (LPT * VEC);
  constexpr int TPW = 64 / LPT;          // 16 rows per wave per load
  constexpr int TPB = TPW * (kThreads / 64);
  constexpr int UNR = 2;                 // rows per lane per loop trip

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int sub = lane % LPT, tiw = lane / LPT;

  // channel of (piece p, element e): p * 32 + sub * 8 + e
  float muv[PIECES][VEC], lamv[PIECES][VEC];
#pragma unroll
  for (int p = 0; p < PIECES; ++p)
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      muv[p][e] = (float)mu[(int64_t)u * D + p * LPT * VEC + sub * VEC + e];
      lamv[p][e] = (float)lam[(int64_t)u * D + p * LPT * VEC + sub * VEC + e];
    }
  drain_vmem();

  __shared__ float zsh[kKChunk];
  __shared__ float ksq[kKChunk];
  __shared__ float red[kThreads / 64];

  const uint16_t* kb = k + un.l * g.ksl + un.h * g.ksh + un.t0 * g.kst;
  const int64_t trow = token_row(g, un);
  static_assert(kKChunk % (UNR * TPB) == 0, "chunk must be whole unrolled trips");

  // Each load reads the wave's 16 rows through a buffer range that ends at
  // the unit's last row (rows past it load as zeros and are discarded), with
  // fixed per-lane offsets.
  const int32_t kstb = (int32_t)g.kst * 2;
  int32_t koff[PIECES];
#pragma unroll
  for (int p = 0; p < PIECES; ++p) koff[p] = tiw * kstb + sub * 16 + p * LPT * 16;
  auto load_trip = [&](int it0, uint4 (&raw)[UNR][PIECES]) {
#pragma unroll
    for (int j = 0; j < UNR; ++j) {
      const int r0 = base + it0 + j * TPB + wave * TPW;  // first row of the wave
      const int32_t rows = min(un.n - r0, TPW);
      const auto kr = buffer_range(kb + (int64_t)r0 * g.kst, rows_bytes(rows, kstb, D * 2));
#pragma unroll
      for (int p = 0; p < PIECES; ++p) raw[j][p] = buffer_load16(kr, koff[p]);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Two register buffers, swapped by unrolling the trip loop by two (a copy
  // between them would make the compiler wait for the prefetched loads).
  auto process = [&](int it0, const uint4 (&raw)[UNR][PIECES]) {
#pragma unroll
    for (int j = 0; j < UNR; ++j) {
      const int tl = it0 + j * TPB + wave * TPW + tiw;
      const bool valid = base + tl < un.n;
      float dot = 0.0f, kap = 0.0f;
#pragma unroll
      for (int p = 0; p < PIECES; ++p) {
        const uint32_t wd[4] = {raw[j][p].x, raw[j][p].y, raw[j][p].z, raw[j][p].w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const float x0 = __uint_as_float(wd[h] << 16);
          const float x1 = __uint_as_float(wd[h] & 0xFFFF0000u);
          dot = fmaf(muv[p][2 * h], x0, dot);
          dot = fmaf(muv[p][2 * h + 1], x1, dot);
          kap = fmaf(lamv[p][2 * h] * x0, x0, kap);
          kap = fmaf(lamv[p][2 * h + 1] * x1, x1, kap);
        }
      }
      dot += dpp_f32<kDppQuadXor1>(dot);
      kap += dpp_f32<kDppQuadXor1>(kap);
      dot += dpp_f32<kDppQuadXor2>(dot);
      kap += dpp_f32<kDppQuadXor2>(kap);
      if (sub == 0) {
        zsh[tl] = valid ? (float)((double)dot * inv_scale) : -INFINITY;
        ksq[tl] = kap;
      }
    }
  };
  constexpr int TRIP = UNR * TPB;
  static_assert(kKChunk % (2 * TRIP) == 0, "chunk must be whole pairs of trips");
  uint4 ba[UNR][PIECES], bb[UNR][PIECES];
  load_trip(0, ba);
  for (int it0 = 0; it0 < kKChunk; it0 += 2 * TRIP) {
    load_trip(it0 + TRIP, bb);
    process(it0, ba);
    load_trip(min(it0 + 2 * TRIP, kKChunk - TRIP), ba);
    process(it0 + TRIP, bb);
  }
  kpass_epilogue(un, u, base, trow, zsh, ksq, red, zout, kout, cstat, kchunks, status, uflags,
                 chunk);
}

// ---------------------------------------------------------------------------
// K pass for bf16 keys with the FULL window covariance, on the MFMA: the tile
// L = K Q^T of a chunk's tokens against the unit's N_s window queries (both
// exact in bf16, fp32 accumulation), kappa_i = the 1/N_s variance of row i of
// L, which equals k_i^T Lambda_Q k_i. It is taken about c_i = mu . k_i (from
// the VALU, also giving z_i): each MFMA chain starts from -c_i, so it yields
// l - c directly, and kappa = mean((l - c)^2), without the large mean ever
// being subtracted; the omitted (mean(l) - c)^2 is rounding-sized. The
// window (N_s <= kFullMaxQ rows) is staged in LDS;
// each wave takes 16-token tiles of the chunk, two per pass (rows loaded one
// pass ahead), and reads the query fragments one 16-query tile ahead.
// ---------------------------------------------------------------------------
typedef __bf16 kbf16x8 __attribute__((ext_vector_type(8)));
typedef float kfloatx4 __attribute__((ext_vector_type(4)));

// Sum over each 16-lane row; every lane of the row ends with the sum.
__device__ __forceinline__ float row_sum16_f32(float v) {
  v += dpp_f32<kDppQuadXor1>(v);
  v += dpp_f32<kDppQuadXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  return v;
}

// LDS of the window tile: the staged window (u16 rows of QP = d + 8).
template <int D>
constexpr int kWindowLds = kFullMaxQ * (D + 8);

// One chunk (unit u, tokens base ..) of the window-tile K pass; LDS from the
// caller (qsh: kWindowLds<D> u16; zsh, ksq: kKChunk floats; red).
template <int D>
__device__ __forceinline__ void kpass_tile_chunk(
    const Geo& g, int u, const Unit& un, int chunk, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ q, const double* __restrict__ mu, float* __restrict__ zout,
    float* __restrict__ kout, float2* __restrict__ cstat, int kchunks, double inv_scale,
    uint32_t* status, uint32_t* uflags, uint16_t* qsh, float* zsh, float* ksq, float* red) {
  constexpr int NK = D / 32;            // K-blocks of 32 channels
  constexpr int QP = D + 8;             // u16 per staged query row
  constexpr int TT = 2;                 // 16-token tiles per wave pass
  constexpr int WT = kKChunk / (kThreads / 64);  // tokens per wave per chunk
  static_assert(WT % (2 * 16 * TT) == 0, "whole pairs of passes per wave");
  const int base = chunk * kKChunk;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ch = lane & 15, kg = lane >> 4;
  const int Ns = g.G * g.w, nqt = (Ns + 15) / 16;

  // The pooled window: row r = gq * w + p (query head gq of the group,
  // position p); rows N_s .. 16 nqt - 1 are zero and masked below.
  const uint16_t* qb = q + un.b * g.qss + un.l * g.qsl + (int64_t)(un.h * g.V + un.s) * g.G * g.qsh;
  for (int e = tid; e < nqt * 16 * (D / 8); e += kThreads) {
    const int r = e / (D / 8), pc = e % (D / 8);
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (r < Ns) {
      const int gq = r / g.w, p = r - gq * g.w;
      x = *reinterpret_cast<const uint4*>(qb + gq * g.qsh + p * g.qsp + pc * 8);
    }
    *reinterpret_cast<uint4*>(qsh + r * QP + pc * 8) = x;
  }
  // mu on this lane's A-operand channels 32 kb + 8 kg + j
  float muv[NK][8];
#pragma unroll
  for (int kb = 0; kb < NK; ++kb)
#pragma unroll
    for (int j = 0; j < 8; ++j) muv[kb][j] = (float)mu[(int64_t)u * D + 32 * kb + 8 * kg + j];
  drain_vmem();
  __syncthreads();

  const uint16_t* kbase = k + un.l * g.ksl + un.h * g.ksh + un.t0 * g.kst;
  const int64_t trow = token_row(g, un);
  const int32_t kstb = (int32_t)g.kst * 2;
  // A fragments of a pass: tile tt, token 16 tt + ch, channels 32 kb + 8 kg ..
  // + 7 (16-byte loads through ranges ending at the unit's last row: rows past
  // it read as zeros and are discarded).
  struct Pass { uint4 a[TT][NK]; };
  // One range per 16-row tile keeps the byte offsets below 16 rows.
  auto load = [&](int t0, Pass& ps) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      const int r0 = base + t0 + 16 * tt;
      const auto kr = buffer_range(kbase + (int64_t)r0 * g.kst, rows_bytes(min(un.n - r0, 16), kstb, D * 2));
#pragma unroll
      for (int kb = 0; kb < NK; ++kb)
        ps.a[tt][kb] = buffer_load16(kr, ch * kstb + (32 * kb + 8 * kg) * 2);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto compute = [&](int t0, const Pass& ps) {
    // c = mu . k for token 16 tt + ch: the lane's 32 channels, then the 4
    // lanes (kg) of the token
    float c[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      float d = 0.0f;
#pragma unroll
      for (int kb = 0; kb < NK; ++kb) {
        const uint32_t wd[4] = {ps.a[tt][kb].x, ps.a[tt][kb].y, ps.a[tt][kb].z, ps.a[tt][kb].w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          d = fmaf(muv[kb][2 * h], __uint_as_float(wd[h] << 16), d);
          d = fmaf(muv[kb][2 * h + 1], __uint_as_float(wd[h] & 0xFFFF0000u), d);
        }
      }
      d += __shfl_xor(d, 16);
      d += __shfl_xor(d, 32);
      c[tt] = d;
    }
    // the shift of output element (token 4 kg + r of tile tt, query ch),
    // negated: the MFMA chain starts from it, so it ends with l - c
    kfloatx4 negc[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) negc[tt][r] = -__shfl(c[tt], 4 * kg + r);
    float s2[TT][4];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) s2[tt][r] = 0.0f;
    // B fragments (query tile qt, K-block kb) are read one tile ahead.
    auto bload = [&](int qt, kbf16x8 (&b)[NK]) {
#pragma unroll
      for (int kb = 0; kb < NK; ++kb)
        b[kb] = *reinterpret_cast<const kbf16x8*>(qsh + (qt * 16 + ch) * QP + 32 * kb + 8 * kg);
    };
    kbf16x8 bcur[NK], bnxt[NK];
    bload(0, bcur);
    auto qtile = [&](int qt, auto maskc) {
      constexpr bool MASK = decltype(maskc)::value;
      if (!MASK) bload(qt + 1, bnxt);
      kfloatx4 acc[TT];
#pragma unroll
      for (int kb = 0; kb < NK; ++kb) {
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
          acc[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(kbf16x8, ps.a[tt][kb]), bcur[kb], kb == 0 ? negc[tt] : acc[tt],
              0, 0, 0);
      }
      // the last tile's padding queries (rows >= N_s) add nothing
      const float m = (!MASK || qt * 16 + ch < Ns) ? 1.0f : 0.0f;
#pragma unroll
      for (int tt = 0; tt < TT; ++tt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float e = MASK ? acc[tt][r] * m : acc[tt][r];
          s2[tt][r] = fmaf(e, e, s2[tt][r]);
        }
      if (!MASK)
#pragma unroll
        for (int kb = 0; kb < NK; ++kb) bcur[kb] = bnxt[kb];
    };
    for (int qt = 0; qt < nqt - 1; ++qt) qtile(qt, std::false_type{});
    qtile(nqt - 1, std::true_type{});
    // kappa = mean((l - c)^2); the omitted (mean(l) - c)^2 is the square of
    // a rounding difference (c and the mean of l are the same dot product
    // summed in two orders). One window query: exactly zero.
    const float invn = 1.0f / (float)Ns;
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float a2 = Ns > 1 ? row_sum16_f32(s2[tt][r]) * invn : 0.0f;
        const int tl = t0 + 16 * tt + 4 * kg + r;  // chunk-local token
        if (ch == 0) {
          ksq[tl] = a2;
          zsh[tl] = base + tl < un.n ? (float)((double)(-negc[tt][r]) * inv_scale) : -INFINITY;
        }
      }
  };
  Pass pa, pb;
  const int w0 = wave * WT;
  load(w0, pa);
  for (int p0 = 0; p0 < WT; p0 += 2 * 16 * TT) {
    load(w0 + p0 + 16 * TT, pb);
    compute(w0 + p0, pa);
    load(min(w0 + p0 + 2 * 16 * TT, w0 + WT - 16 * TT), pa);
    compute(w0 + p0 + 16 * TT, pb);
  }
  kpass_epilogue(un, u, base, trow, zsh, ksq, red, zout, kout, cstat, kchunks, status, uflags,
                 chunk);
}


template <int D>
__global__ __launch_bounds__(kThreads, 2) void kpass_full_mfma_kernel(
    Geo g, const uint16_t* __restrict__ k, const uint16_t* __restrict__ q,
    const double* __restrict__ mu, float* __restrict__ zout, float* __restrict__ kout,
    float2* __restrict__ cstat, int kchunks, double inv_scale, uint32_t* status,
    uint32_t* uflags) {
  __shared__ __attribute__((aligned(16))) uint16_t qsh[kWindowLds<D>];
  __shared__ float zsh[kKChunk];
  __shared__ float ksq[kKChunk];
  __shared__ float red[kThreads / 64];
  int u, chunk;
  if (!grid_unit_chunk<false>(g, kchunks, u, chunk)) return;
  const Unit un = decode_unit(g, u);
  if (chunk * kKChunk >= un.n) return;
  kpass_tile_chunk<D>(g, u, un, chunk, k, q, mu, zout, kout, cstat, kchunks, inv_scale, status,
                      uflags, qsh, zsh, ksq, red);
}

// ---------------------------------------------------------------------------
// K pass for bf16 keys with the FULL window covariance, triangular path
// (full_kpass_tri): kappa_i = ||X k_i||^2 with Lambda_Q = X^T X, X lower
// triangular in two-term bf16 B fragments from launch_qfactor, on MFMA
// 16x16x32 as in the leverage pass (tokens are the MFMA rows; only the
// K-blocks of the lower triangle). z_i = mu . k_i / (tau sqrt d) comes from
// one more MFMA chain, whose B columns 0, 1 and 2 hold mu (rounded to fp32)
// split exactly into three bf16 terms: the three column sums add to the
// fp32-accumulated dot product. Units marked kUnitKTile take the window tile
// inside the same launch (the two paths share the LDS).
//
// Each wave takes 16-token steps of the chunk (rows read whole, non-temporal
// or cached per POL, two steps ahead in three rotating buffers), as the
// leverage pass does; the rows pass through a wave-private LDS tile into the
// MFMA operand layout.
// ---------------------------------------------------------------------------
template <int D, int POL>
__global__ __launch_bounds__(kThreads, 2) void kpass_tri_kernel(
    Geo g, const uint16_t* __restrict__ k, const uint16_t* __restrict__ q,
    const double* __restrict__ mu, const uint16_t* __restrict__ xfrag,
    float* __restrict__ zout, float* __restrict__ kout, float2* __restrict__ cstat, int kchunks,
    int sub, double inv_scale, uint32_t* status, uint32_t* uflags) {
  constexpr int NB = D / 16;                    // output blocks of 16 channels
  constexpr int NK = D / 32;                    // K blocks of 32 channels
  constexpr int NLP = (NB / 2) * (NB / 2 + 1);  // lower (j, kb) block pairs
  // bytes per tile row: a 32-byte pad leaves the operand reads (16 rows, four
  // 16-byte pieces each) free of bank conflicts, measured (16 bytes: 16.5 %)
  constexpr int PITCH = D * 2 + 32;
  constexpr int TILE_BYTES = (kThreads / 64) * 16 * PITCH;
  static_assert(TILE_BYTES + NK * 64 * 16 <= kWindowLds<D> * 2, "tri path fits the window LDS");
  __shared__ __attribute__((aligned(16))) uint16_t qsh[kWindowLds<D>];
  __shared__ float zsh[kKChunk];
  __shared__ float ksq[kKChunk];
  __shared__ float red[kThreads / 64];
  // `sub` consecutive chunks of one unit per workgroup
  int u, grp;
  if (!grid_unit_chunk<false>(g, (kchunks + sub - 1) / sub, u, grp)) return;
  const Unit un = decode_unit(g, u);
  const int chunk0 = grp * sub;
  const int base0 = chunk0 * kKChunk;
  if (base0 >= un.n) return;
  const int nsub = min(sub, (un.n - base0 + kKChunk - 1) / kKChunk);
  if (uflags[u] & kUnitKTile) {
    for (int c = 0; c < nsub; ++c)
      kpass_tile_chunk<D>(g, u, un, chunk0 + c, k, q, mu, zout, kout, cstat, kchunks, inv_scale,
                          status, uflags, qsh, zsh, ksq, red);
    return;
  }
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ch = lane & 15, kg = lane >> 4;
  const int rl = 2 * (ch >> 3) + ((ch >> 2) & 1);  // token (of 4) whose kappa this lane ends with
  const int lim = base0 + nsub * kKChunk;
  const int end = min(un.n, lim);
  const int64_t trow = token_row(g, un);

  const uint16_t* kb0 = k + un.l * g.ksl + un.h * g.ksh + un.t0 * g.kst;
  const int32_t kstb = (int32_t)g.kst * 2;
  constexpr int LPR = D / 8;                    // lanes per whole row (16 bytes each)
  constexpr int RPL = 64 / LPR;                 // rows per wave load
  static_assert(RPL * NK == 16, "a step's 16 rows in NK whole-row loads");
  const int rrow = lane / LPR, rpc = lane % LPR;
  int32_t koff[NK];
#pragma unroll
  for (int i = 0; i < NK; ++i) koff[i] = (RPL * i + rrow) * kstb + rpc * 16;
  struct Buf { uint4 a[NK]; };
  // Rows past the unit's last one read as zeros (the range ends there).
  auto load = [&](int t0, Buf& bf) {
    const int32_t rows = min(end - t0, 16);
    const auto kr = buffer_range(kb0 + (int64_t)t0 * g.kst, rows_bytes(rows, kstb, D * 2));
#pragma unroll
    for (int i = 0; i < NK; ++i) bf.a[i] = buffer_load16<POL>(kr, koff[i]);
    __builtin_amdgcn_sched_barrier(0);
  };
  // The key stream starts first: the prologue's loads below wait behind it.
  constexpr int WSTRIDE = 16 * (kThreads / 64);
  const int t_first = base0 + wave * 16;
  Buf b0, b1, b2;
  load(t_first, b0);
  load(t_first + WSTRIDE, b1);

  char* tile = reinterpret_cast<char*>(qsh) + wave * 16 * PITCH;
  kbf16x8* mub = reinterpret_cast<kbf16x8*>(reinterpret_cast<char*>(qsh) + TILE_BYTES);
  // B fragments of the mu block: lane (c, kg) of K-block kb holds column c,
  // channels 32 kb + 8 kg + t: mu's hi, mid and lo bf16 terms in columns 0,
  // 1, 2 and zeros elsewhere.
  for (int e = tid; e < NK * 64; e += kThreads) {
    const int kb = e >> 6, c = e & 15, g4 = (e >> 4) & 3;
    kbf16x8 f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float m = (float)mu[(int64_t)u * D + 32 * kb + 8 * g4 + t];
      const __bf16 hi = (__bf16)m;
      const __bf16 mid = (__bf16)(m - (float)hi);
      const __bf16 lo = (__bf16)((m - (float)hi) - (float)mid);
      f[t] = c == 0 ? hi : c == 1 ? mid : c == 2 ? lo : (__bf16)0.0f;
    }
    mub[e] = f;
  }
  // X's B fragments, in registers (as the leverage pass holds L^{-1}).
  kbf16x8 bh[NLP], bl[NLP];
  const uint16_t* xf = xfrag + (int64_t)u * NLP * 2 * 64 * 8;
#pragma unroll
  for (int p = 0; p < NLP; ++p) {
    bh[p] = *reinterpret_cast<const kbf16x8*>(xf + ((int64_t)(p * 2 + 0) * 64 + lane) * 8);
    bl[p] = *reinterpret_cast<const kbf16x8*>(xf + ((int64_t)(p * 2 + 1) * 64 + lane) * 8);
  }
  drain_vmem();
  __syncthreads();  // mu fragments visible

  auto step = [&](int t0, const Buf& bf) {
#pragma unroll
    for (int i = 0; i < NK; ++i)
      *reinterpret_cast<uint4*>(tile + (RPL * i + rrow) * PITCH + rpc * 16) = bf.a[i];
    kbf16x8 cur[NK];
#pragma unroll
    for (int kb = 0; kb < NK; ++kb)
      cur[kb] = *reinterpret_cast<const kbf16x8*>(tile + ch * PITCH + kb * 64 + kg * 16);
    kfloatx4 zc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < NK; ++kb)
      zc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur[kb], mub[kb * 64 + lane], zc, 0, 0, 0);
    float ss[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jp = 0; jp < NB / 2; ++jp) {
      kfloatx4 y0 = {0.f, 0.f, 0.f, 0.f}, y1 = {0.f, 0.f, 0.f, 0.f};
      const int q0 = jp * (jp + 1);             // pair index of (2 jp, 0)
      const int q1 = jp * (jp + 1) + (jp + 1);  // pair index of (2 jp + 1, 0)
#pragma unroll
      for (int kb = 0; kb <= jp; ++kb) {
        y0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur[kb], bh[q0 + kb], y0, 0, 0, 0);
        y1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur[kb], bh[q1 + kb], y1, 0, 0, 0);
        y0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur[kb], bl[q0 + kb], y0, 0, 0, 0);
        y1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur[kb], bl[q1 + kb], y1, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) ss[r] += y0[r] * y0[r] + y1[r] * y1[r];
    }
    // The step's place in its chunk (steps never straddle two chunks).
    const int tc = (t0 - base0) & (kKChunk - 1);
    // kappa: ss[r] is this lane's output channel's part of token 4 kg + r;
    // the transposing row reduction of the leverage pass leaves token rl's
    // sum in lane ch (ch % 4 == 0 stores it).
    const bool hi8 = ch >= 8, hi4 = (ch & 4) != 0;
    const float m0 = (hi8 ? ss[2] : ss[0]) + dpp_f32<kDppMirror>(hi8 ? ss[0] : ss[2]);
    const float m1 = (hi8 ? ss[3] : ss[1]) + dpp_f32<kDppMirror>(hi8 ? ss[1] : ss[3]);
    float sv = (hi4 ? m1 : m0) + dpp_f32<kDppHalfMirror>(hi4 ? m0 : m1);
    sv += dpp_f32<kDppQuadXor1>(sv);
    sv += dpp_f32<kDppQuadXor2>(sv);
    if ((ch & 3) == 0) ksq[tc + 4 * kg + rl] = sv;
    // z: columns 0..3 of the mu block sit in lanes ch = 0..3 (column 3 is
    // zero); a quad sum leaves token 4 kg + r's dot product in lane ch = 0.
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float zv = zc[r];
      zv += dpp_f32<kDppQuadXor1>(zv);
      zv += dpp_f32<kDppQuadXor2>(zv);
      if (ch == 0)
        zsh[tc + 4 * kg + r] = t0 + 4 * kg + r < end ? (float)((double)zv * inv_scale) : -INFINITY;
    }
  };
  // Every step of the chunks runs (steps past the unit's end store -inf
  // logits), so that each chunk's epilogue sees the whole chunk; the
  // epilogue follows the chunk's last step (the same step count in every
  // wave), while the loads for the next chunk are already in flight.
  constexpr int SPC = kKChunk / WSTRIDE;  // steps per wave per chunk
  static_assert((kKChunk & (kKChunk - 1)) == 0 && kKChunk % WSTRIDE == 0, "chunks of whole steps");
  int done = 0;
  auto after = [&]() {
    if (++done % SPC == 0) {
      const int c = done / SPC - 1;
      kpass_epilogue(un, u, base0 + c * kKChunk, trow, zsh, ksq, red, zout, kout, cstat, kchunks,
                     status, uflags, chunk0 + c);
    }
  };
  for (int t0 = t_first; t0 < lim; t0 += 3 * WSTRIDE) {
    load(t0 + 2 * WSTRIDE, b2);
    step(t0, b0);
    after();
    if (t0 + WSTRIDE >= lim) break;
    load(t0 + 3 * WSTRIDE, b0);
    step(t0 + WSTRIDE, b1);
    after();
    if (t0 + 2 * WSTRIDE >= lim) break;
    load(t0 + 4 * WSTRIDE, b1);
    step(t0 + 2 * WSTRIDE, b2);
    after();
  }
}

template <typename T, int D>
static void kpass_dispatch(const Launch& L, const void* k, bool full, dim3 grid, double inv_scale) {
  const Geo& g = L.geo;
  auto args = [&](auto kern) {
    kern<<<grid, kThreads, 0, L.stream>>>(
        g, (const T*)k, ws_ptr<double>(L.wsp, L.ws.mu), ws_ptr<double>(L.wsp, L.ws.lam),
        ws_ptr<float>(L.wsp, L.ws.lamfull), ws_ptr<float>(L.wsp, L.ws.z),
        ws_ptr<float>(L.wsp, L.ws.kappa), ws_ptr<float2>(L.wsp, L.ws.cstat), L.ws.kchunks,
        inv_scale, ws_ptr<uint32_t>(L.wsp, L.ws.status), ws_ptr<uint32_t>(L.wsp, L.ws.uflags));
  };
  if (full) {
    args(kpass_kernel<T, D, true>);
  } else if constexpr (std::is_same<T, uint16_t>::value) {
    kpass_quad_kernel<D><<<grid, kThreads, 0, L.stream>>>(
        g, (const uint16_t*)k, ws_ptr<double>(L.wsp, L.ws.mu), ws_ptr<double>(L.wsp, L.ws.lam),
        ws_ptr<float>(L.wsp, L.ws.z), ws_ptr<float>(L.wsp, L.ws.kappa),
        ws_ptr<float2>(L.wsp, L.ws.cstat), L.ws.kchunks, inv_scale,
        ws_ptr<uint32_t>(L.wsp, L.ws.status), ws_ptr<uint32_t>(L.wsp, L.ws.uflags));
  } else {
    args(kpass_kernel<T, D, false>);
  }
}

hipError_t launch_kpass(const Launch& L, const void* k, const void* q) {
  const Geo& g = L.geo;
  const bool full = L.cfg->cov_mode == JACAP_COV_FULL;
  const double inv_scale = 1.0 / ((double)L.cfg->temperature * sqrt((double)g.D));
  const dim3 grid((unsigned)chunked_grid(g, L.ws.kchunks));
  const bool bf = L.cfg->dtype == JACAP_DTYPE_BF16;
  if (full_kpass_tri(L, q)) {  // ||X k||^2 from Lambda_Q's factor (launch_qfactor)
    // up to kTriChunks chunks per workgroup, fewer while the grid would
    // otherwise hold under kLevMinBlocks workgroups
    int sub = kTriChunks;
    while (sub > 1 && (int64_t)(L.ws.kchunks + sub - 1) / sub * (g.U / g.V) < kLevMinBlocks) sub /= 2;
    const dim3 tgrid((unsigned)chunked_grid(g, (L.ws.kchunks + sub - 1) / sub));
    auto go = [&](auto kern) {
      kern<<<tgrid, kThreads, 0, L.stream>>>(
          g, (const uint16_t*)k, (const uint16_t*)q, ws_ptr<double>(L.wsp, L.ws.mu),
          ws_ptr<uint16_t>(L.wsp, L.ws.lfrag), ws_ptr<float>(L.wsp, L.ws.z),
          ws_ptr<float>(L.wsp, L.ws.kappa), ws_ptr<float2>(L.wsp, L.ws.cstat), L.ws.kchunks, sub,
          inv_scale, ws_ptr<uint32_t>(L.wsp, L.ws.status), ws_ptr<uint32_t>(L.wsp, L.ws.uflags));
    };
    // K rows read once (pooled group): streamed; by the V units of a KV head: cached
    if (g.V == 1) {
      if (g.D == 128) go(kpass_tri_kernel<128, kPolicyStream>);
      else go(kpass_tri_kernel<64, kPolicyStream>);
    } else {
      if (g.D == 128) go(kpass_tri_kernel<128, kPolicyShared>);
      else go(kpass_tri_kernel<64, kPolicyShared>);
    }
    return hipGetLastError();
  }
  if (full_kpass_on_mfma(L, q)) {  // window queries at hand: the MFMA tile
    auto go = [&](auto kern) {
      kern<<<grid, kThreads, 0, L.stream>>>(
          g, (const uint16_t*)k, (const uint16_t*)q, ws_ptr<double>(L.wsp, L.ws.mu),
          ws_ptr<float>(L.wsp, L.ws.z), ws_ptr<float>(L.wsp, L.ws.kappa),
          ws_ptr<float2>(L.wsp, L.ws.cstat), L.ws.kchunks, inv_scale,
          ws_ptr<uint32_t>(L.wsp, L.ws.status), ws_ptr<uint32_t>(L.wsp, L.ws.uflags));
    };
    if (g.D == 128) go(kpass_full_mfma_kernel<128>);
    else go(kpass_full_mfma_kernel<64>);
    return hipGetLastError();
  }
  if (g.D == 128) {
    if (bf) kpass_dispatch<uint16_t, 128>(L, k, full, grid, inv_scale);
    else kpass_dispatch<float, 128>(L, k, full, grid, inv_scale);
  } else {
    if (bf) kpass_dispatch<uint16_t, 64>(L, k, full, grid, inv_scale);
    else kpass_dispatch<float, 64>(L, k, full, grid, inv_scale);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Global softmax normaliser per unit, m = max_c m_c and
// Z = sum_c Z_c exp(m_c - m) (fp64, fixed order), then the Eq. 8 importance
// weight of every token of the block's chunk (fp64, stored as fp32).
// wchunks blocks per unit. Every block of a unit merges the chunk statistics
// in the same order, so all of them use bit-identical (m, Z); block 0 stores them.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void softmax_weights_kernel(
    Geo g, const float2* __restrict__ cstat, int kchunks, const float* __restrict__ zbuf,
    const float* __restrict__ kbuf, double inv_d, int wchunks, float* __restrict__ m_out,
    double* __restrict__ z_out, double* __restrict__ scale_out, float* __restrict__ wout) {
  int u, chunk;
  if (!grid_unit_chunk<false>(g, wchunks, u, chunk)) return;
  const int tid = threadIdx.x;
  const Unit un = decode_unit(g, u);
  __shared__ float redf[kThreads / 64];
  __shared__ int redi[kThreads / 64];
  __shared__ double redd[kThreads / 64];
  if (un.n == 0) {
    if (chunk == 0 && tid == 0) { m_out[u] = 0.0f; z_out[u] = 1.0; scale_out[u] = 1.0; }
    return;
  }
  const int base = chunk * kWChunk;
  if (base >= un.n) return;
  const int nch = (un.n + kKChunk - 1) / kKChunk;
  const float2* cs = cstat + (int64_t)u * kchunks;
  float m = -INFINITY;
  for (int c = tid; c < nch; c += kThreads) m = fmaxf(m, cs[c].x);
  m = block_combine(wave_max(m), redf, [](float a, float b) { return fmaxf(a, b); });
  // The first chunk holding the maximum: its rest is the rest of Z; every
  // other chunk adds its whole sum, (1 + rest) exp(m_c - m).
  int cmax = nch;
  for (int c = tid; c < nch; c += kThreads)
    if (cs[c].x == m) cmax = min(cmax, c);
  cmax = block_combine(wave_min(cmax), redi, [](int a, int b) { return min(a, b); });
  double rest = 0.0;
  for (int c = tid; c < nch; c += kThreads) {
    const double dm = (double)cs[c].x - (double)m;
    rest += (c == cmax ? 0.0 : exp(dm)) + (double)cs[c].y * exp(dm - (double)kRestShift);
  }
  rest = block_combine(wave_sum(rest), redd, [](double a, double b) { return a + b; });
  const double s = 1.0 + rest;  // Z
  // Every rho_i = alpha_i (1 - alpha_i) is at most min(1/4, rest / Z). When
  // that bound is tiny (a saturated softmax) the weights are stored times a
  // power of two that lifts its square to [1, 4), so that they stay inside
  // fp32's range; the ridge (or R) is scaled by the same power of two in the
  // factorisation, which leaves every score w_i v_i^T A^{-1} v_i unchanged.
  const double rho_max = fmin(0.25, rest / s);
  const double wscale = rho_max > 0.0 && rho_max < 0x1p-20 ? ldexp(1.0, -2 * ilogb(rho_max)) : 1.0;
  if (chunk == 0 && tid == 0) { m_out[u] = m; z_out[u] = s; scale_out[u] = wscale; }
  const double wfac = wscale * inv_d;
  const int64_t trow = token_row(g, un);
  const int end = min(un.n, base + kWChunk);
  // Eq. 8 per token: e = exp(z - m) from the fp32 exponential of the rounded
  // difference, corrected to first order by the difference's rounding error
  // (relative error ~1e-7), alpha = e / Z and 1 - alpha = (Z - e) / Z in fp64,
  // with Z - e = (1 - e) + rest (exact for the maximum, where e = 1).
  const double invZ = 1.0 / s;
  auto weight = [&](float z, float kap) {
    const double dz = (double)z - (double)m;  // exact
    const float df = (float)dz;
    // far below the maximum the fp32 exponential would be subnormal
    const double e = df > -80.0f ? (double)expf(df) * (1.0 + (dz - (double)df)) : exp(dz);
    const double rho = (e * invZ) * (((1.0 - e) + rest) * invZ);
    return (float)(rho * rho * (double)kap * wfac);
  };
  constexpr int U4 = 4;
  static_assert(kWChunk % (U4 * kThreads) == 0, "whole unrolled trips per chunk");
  for (int t0 = base + tid; t0 < end; t0 += U4 * kThreads) {
    float z[U4], kq[U4];
#pragma unroll
    for (int j = 0; j < U4; ++j) {
      const int t = min(t0 + j * kThreads, end - 1);
      z[j] = zbuf[trow + t];
      kq[j] = kbuf[trow + t];
    }
#pragma unroll
    for (int j = 0; j < U4; ++j)
      if (t0 + j * kThreads < end) wout[trow + t0 + j * kThreads] = weight(z[j], kq[j]);
  }
}

hipError_t launch_softmax_weights(const Launch& L) {
  const int wchunks = L.ws.wchunks > 0 ? L.ws.wchunks : 1;
  const dim3 grid((unsigned)chunked_grid(L.geo, wchunks));
  softmax_weights_kernel<<<grid, kThreads, 0, L.stream>>>(
      L.geo, ws_ptr<float2>(L.wsp, L.ws.cstat), L.ws.kchunks, ws_ptr<float>(L.wsp, L.ws.z),
      ws_ptr<float>(L.wsp, L.ws.kappa), 1.0 / (double)L.geo.D, wchunks,
      ws_ptr<float>(L.wsp, L.ws.smax_m),
      ws_ptr<double>(L.wsp, L.ws.smax_z), ws_ptr<double>(L.wsp, L.ws.wscale),
      ws_ptr<float>(L.wsp, L.ws.wgt));
  return hipGetLastError();
}

}  // namespace jacap
