// Exact greedy log-det selection (App. B.1): the sequential maximisation that
// the one-shot leverage ranking of Eq. 10 approximates, kept as a quality
// comparator for TOP-B.
//
// Per unit, with the Eq. 8 weights w_i and u_i = v_i, the greedy adds B times
// the token with the largest gain w_i c_i, c_i = u_i^T A_C^{-1} u_i, where
// A_C = ridge I + sum_{j in C} w_j u_j u_j^T (by the matrix determinant lemma
// the log-det increase is log(1 + w_i c_i), increasing in w_i c_i); ties go to
// the lowest position. After a pick s, Sherman-Morrison gives
// A^{-1} <- A^{-1} - g g^T with g = A^{-1} u_s sqrt(w_s / (1 + w_s c_s)).
//
// GPU design (one workgroup of 256 threads per unit):
// * A^{-1} (d x d, fp64) is held in registers: thread t owns row t / TPR and a
//   contiguous run of d / TPR columns (TPR = 256 / d). c = u^T A^{-1} u and
//   A^{-1} u cost d^2 FMA spread over the workgroup.
// * Gains never grow as C grows (each pick lowers c_i by (u_i . g)^2), so a
//   c_i computed after fewer picks bounds the current one from above (lazy
//   greedy, after Minoux). Per token the workspace keeps c_i and the number of
//   picks made when it was computed (its stamp; -1 = taken); per block of 256
//   positions an LDS entry keeps the block's best (key w_i c_i, c_i, position,
//   stamp). Each round wave 0 finds the best entry: if its stamp is current
//   the token is taken, else its c is recomputed and the block rescanned. The
//   token taken is the eager greedy's: every other token's current gain is at
//   most its key, and equal keys resolve by position.
// * Token i's workspace state is read and written only by lane i % 64 of wave
//   0 inside the kernel (the initial values come from the previous launch), so
//   every read sees that lane's own earlier writes.
// * The initial pass (c_i = ||u_i||^2 / ridge, stamp 0, and the block
//   entries) streams V once with many workgroups per unit.
#include <float.h>

#include "jacap_internal.hpp"

namespace jacap {

namespace {

constexpr int kGBlock = 256;            // positions per tournament block
constexpr int kGMaxBlocks = kGreedyMaxLen / kGBlock;
constexpr int kGMaxWords = kGreedyMaxLen / 32;
constexpr int kGSlots = kGBlock / 64;   // positions per lane in a block scan

constexpr int kOpStop = 0, kOpRefresh = 1, kOpPick = 2;

// Ordering key of a gain; NaN and -inf (untaken) sort just above a taken
// token's -inf, so the search never returns a taken token while one is left.
__device__ __forceinline__ double gain_key(float w, double c) {
  const double x = (double)w * c;
  return x >= -DBL_MAX ? x : -DBL_MAX;
}

// (key, position) lexicographic: larger key first, then lower position.
__device__ __forceinline__ void take_better(double& k, int& p, double k2, int p2) {
  if (k2 > k || (k2 == k && p2 < p)) {
    k = k2;
    p = p2;
  }
}

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

// Wave64 arg-max of (key, position); every lane ends with the same result.
__device__ __forceinline__ void wave_argmax(double& k, int& p) {
  take_better(k, p, dpp_f64<kDppQuadXor1>(k), dpp_i32<kDppQuadXor1>(p));
  take_better(k, p, dpp_f64<kDppQuadXor2>(k), dpp_i32<kDppQuadXor2>(p));
  take_better(k, p, dpp_f64<kDppHalfMirror>(k), dpp_i32<kDppHalfMirror>(p));
  take_better(k, p, dpp_f64<kDppMirror>(k), dpp_i32<kDppMirror>(p));
  take_better(k, p, __shfl_xor(k, 16), __shfl_xor(p, 16));
  take_better(k, p, __shfl_xor(k, 32), __shfl_xor(p, 32));
}

// Sum over each 16-lane row (every lane of the row ends with the same value).
__device__ __forceinline__ double row_sum16(double v) {
  v += dpp_f64<kDppQuadXor1>(v);
  v += dpp_f64<kDppQuadXor2>(v);
  v += dpp_f64<kDppHalfMirror>(v);
  v += dpp_f64<kDppMirror>(v);
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  v = row_sum16(v);
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

template <typename X>
__device__ __forceinline__ X pick4(const X (&a)[kGSlots], int m) {
  return m == 0 ? a[0] : m == 1 ? a[1] : m == 2 ? a[2] : a[3];
}

// N consecutive elements (16-byte aligned for N * sizeof(T) == 16) as floats.
template <typename T, int N>
__device__ __forceinline__ void load_elems(const T* p, float (&x)[N]) {
  if constexpr (sizeof(T) == 2) {
    static_assert(N == 4 || N == 8, "bf16 chunk");
    if constexpr (N == 8) {
      const uint4 r = *reinterpret_cast<const uint4*>(p);
      const uint32_t wd[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[2 * i] = bf16_to_f32((uint16_t)(wd[i] & 0xFFFFu));
        x[2 * i + 1] = bf16_to_f32((uint16_t)(wd[i] >> 16));
      }
    } else {
      const uint2 r = *reinterpret_cast<const uint2*>(p);
      const uint32_t wd[2] = {r.x, r.y};
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        x[2 * i] = bf16_to_f32((uint16_t)(wd[i] & 0xFFFFu));
        x[2 * i + 1] = bf16_to_f32((uint16_t)(wd[i] >> 16));
      }
    }
  } else {
    static_assert(N % 4 == 0, "fp32 chunk");
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const float4 r = reinterpret_cast<const float4*>(p)[i];
      x[4 * i] = r.x;
      x[4 * i + 1] = r.y;
      x[4 * i + 2] = r.z;
      x[4 * i + 3] = r.w;
    }
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// Initial pass: c_i = ||v_i||^2 / ridge (A_0 = ridge I), stamp 0, and each
// block's best entry. One workgroup per (block of 256 positions, unit); 16
// lanes per token, each summing d/16 squares.
// ---------------------------------------------------------------------------
template <int D, typename T>
__global__ __launch_bounds__(kThreads) void greedy_init_kernel(
    Geo g, const T* __restrict__ v, const float* __restrict__ wgt, float ridge,
    const double* __restrict__ wscale, int budget,
    int protect, double* __restrict__ gc, int32_t* __restrict__ gst,
    GreedyEntry* __restrict__ entries, int nblk_max) {
  constexpr int EPL = D / 16;
  __shared__ double rk[4], rc[4];
  __shared__ int rp[4];
  const int u = blockIdx.y, blk = blockIdx.x;
  const Unit un = decode_unit(g, u);
  const int i0 = blk * kGBlock;
  if (i0 >= un.n) return;
  const int kk = min(budget, un.n), p = min(protect, kk), nfree = un.n - p;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, row = lane >> 4, rl = lane & 15;
  const T* vb = v + (int64_t)un.l * g.vsl + (int64_t)un.h * g.vsh + un.t0 * g.vst;
  const int64_t trow = token_row(g, un);

  // Iteration it handles positions i0 + 64 wave + 4 it + row; lane rl == it
  // keeps that sum, so lane (row, rl) ends with position i0 + 64 wave + 4 rl + row.
  float x[16][EPL];
#pragma unroll
  for (int it = 0; it < 16; ++it) {
    const int i = min(i0 + wave * 64 + it * 4 + row, un.n - 1);
    load_elems<T, EPL>(vb + (int64_t)i * g.vst + rl * EPL, x[it]);
  }
  double mine = 0.0;
#pragma unroll
  for (int it = 0; it < 16; ++it) {
    double s = 0.0;
#pragma unroll
    for (int e = 0; e < EPL; ++e) s = fma((double)x[it][e], (double)x[it][e], s);
    s = row_sum16(s);
    if (rl == it) mine = s;
  }
  const int i = i0 + wave * 64 + rl * 4 + row;
  const double c = mine / ((double)ridge * wscale[u]);  // the stored weights' scale
  double key = -__builtin_inf();
  int pos = INT32_MAX;
  if (i < un.n) {
    gc[trow + i] = c;
    gst[trow + i] = 0;
    if (i < nfree) {
      key = gain_key(wgt[trow + i], c);
      pos = i;
    }
  }
  const double mykey = key;
  const int mypos = pos;
  wave_argmax(key, pos);
  if (pos == INT32_MAX) {
    if (lane == 0) { rk[wave] = key; rc[wave] = 0.0; rp[wave] = INT32_MAX; }
  } else if (mypos == pos && mykey == key) {
    rk[wave] = key; rc[wave] = c; rp[wave] = pos;
  }
  __syncthreads();
  if (tid == 0) {
    double bk = rk[0], bc = rc[0];
    int bp = rp[0];
    for (int j = 1; j < 4; ++j)
      if (rk[j] > bk || (rk[j] == bk && rp[j] < bp)) { bk = rk[j]; bc = rc[j]; bp = rp[j]; }
    GreedyEntry e;
    e.key = bk; e.c = bc; e.pos = bp; e.stamp = 0;
    entries[(int64_t)u * nblk_max + blk] = e;
  }
}

// ---------------------------------------------------------------------------
// The greedy itself: one workgroup per unit.
// ---------------------------------------------------------------------------
struct GreedyShared {
  GreedyEntry ent[kGMaxBlocks];
  uint32_t bits[kGMaxWords];  // taken positions
  double us[kGreedyMaxD];     // the current token's u (fp64)
  double gs[kGreedyMaxD];     // g of the last pick
  double red[4];
  double f;                   // sqrt(w / (1 + w c)) of a pick (or w of a forced pick)
  int op, pos;
  uint32_t scan[5];
};

template <int D, typename T>
__global__ __launch_bounds__(kThreads) void greedy_kernel(
    Geo g, const T* __restrict__ v, const float* __restrict__ wgt, float ridge_f,
    const double* __restrict__ wscale, int budget,
    int protect, double* __restrict__ gc, int32_t* __restrict__ gst,
    const GreedyEntry* __restrict__ entries, int nblk_max, int32_t* __restrict__ idx_out,
    int32_t* __restrict__ order_out, double* __restrict__ logdet_out) {
  constexpr int TPR = kThreads / D;     // threads per row of A^{-1}
  constexpr int NA = D / TPR;           // entries of A^{-1} per thread
  constexpr int EPL = 16 / sizeof(T);   // elements per 16-byte row piece
  constexpr int ROWL = D / EPL;         // lanes fetching one row
  static_assert(TPR == 2 || TPR == 4, "head_dim 64 or 128");
  __shared__ __align__(16) GreedyShared sh;

  const int u = blockIdx.x;
  const Unit un = decode_unit(g, u);
  const int n = un.n;
  const int kk = min(budget, n), p = min(protect, kk), nfree = n - p;
  const int nblk = (n + kGBlock - 1) / kGBlock, words = (n + 31) / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = tid / TPR, q = tid % TPR;
  // A_0 = ridge I times the stored weights' scale (gains are unchanged by it)
  const double ridge = (double)ridge_f * (n > 0 ? wscale[u] : 1.0);
  const T* vb = v + (int64_t)un.l * g.vsl + (int64_t)un.h * g.vsh + un.t0 * g.vst;
  const int64_t trow = token_row(g, un);

  double ainv[NA];
#pragma unroll
  for (int m = 0; m < NA; ++m) ainv[m] = (q * NA + m == r) ? 1.0 / ridge : 0.0;
  for (int j = tid; j < nblk; j += kThreads) sh.ent[j] = entries[(int64_t)u * nblk_max + j];
  for (int j = tid; j < words; j += kThreads) sh.bits[j] = 0u;

  // Row i of V into sh.us (wave 0, lanes < ROWL).
  auto fetch_row = [&](int i) {
    if (lane < ROWL) {
      float x[EPL];
      load_elems<T, EPL>(vb + (int64_t)i * g.vst + lane * EPL, x);
#pragma unroll
      for (int e = 0; e < EPL; ++e) sh.us[lane * EPL + e] = (double)x[e];
    }
  };
  // (A^{-1} u)_r restricted to this thread's columns.
  auto row_partial = [&]() {
    const double2* u2 = reinterpret_cast<const double2*>(sh.us + q * NA);
    double a = 0.0;
#pragma unroll
    for (int m = 0; m < NA / 2; ++m) {
      const double2 x = u2[m];
      a = fma(ainv[2 * m], x.x, a);
      a = fma(ainv[2 * m + 1], x.y, a);
    }
    return a;
  };
  // c = u^T A^{-1} u over the workgroup (one barrier).
  auto quad_form = [&](double partial) {
    const double s = wave_sum_f64(sh.us[r] * partial);
    if (lane == 0) sh.red[wave] = s;
    __syncthreads();
    return ((sh.red[0] + sh.red[1]) + sh.red[2]) + sh.red[3];
  };
  // A^{-1} <- A^{-1} - g g^T, g = (A^{-1} u) f (one barrier).
  auto downdate = [&](double partial, double f) {
    double h = partial + dpp_f64<kDppQuadXor1>(partial);
    if constexpr (TPR == 4) h += dpp_f64<kDppQuadXor2>(h);
    const double gr = h * f;
    if (q == 0) sh.gs[r] = gr;
    __syncthreads();
    const double2* g2 = reinterpret_cast<const double2*>(sh.gs + q * NA);
#pragma unroll
    for (int m = 0; m < NA / 2; ++m) {
      const double2 x = g2[m];
      ainv[2 * m] = fma(-gr, x.x, ainv[2 * m]);
      ainv[2 * m + 1] = fma(-gr, x.y, ainv[2 * m + 1]);
    }
  };

  int32_t* order = order_out ? order_out + (int64_t)u * budget : nullptr;
  double logdet = 0.0;  // sum of log(1 + w c) over the picks (wave 0)
  int t = 0;
  __syncthreads();

  // Protected positions: taken first, in position order (outside the search).
  for (; t < p; ++t) {
    const int s = nfree + t;
    if (wave == 0) {
      fetch_row(s);
      if (lane == 0) sh.f = (double)wgt[trow + s];
    }
    __syncthreads();
    const double partial = row_partial();
    const double w = sh.f;
    const double c = quad_form(partial);
    downdate(partial, sqrt(w / (1.0 + w * c)));
    if (tid == 0) {
      logdet += log1p(w * c);
      sh.bits[s >> 5] |= 1u << (s & 31);
      if (order) order[t] = s;
    }
  }

  // Lazy greedy over positions [0, nfree).
  int cblk = -1, utok = -1;
  double bc[kGSlots];
  int bst[kGSlots];
  float bw[kGSlots];
#pragma unroll
  for (int j = 0; j < kGSlots; ++j) { bc[j] = 0.0; bst[j] = -1; bw[j] = 0.0f; }
  double pick_gain = 0.0;

  // Best entry of block cblk from the registers (wave 0).
  auto rescan = [&]() {
    double bk = -__builtin_inf();
    int bp = INT32_MAX;
#pragma unroll
    for (int j = 0; j < kGSlots; ++j) {
      const int i = cblk * kGBlock + j * 64 + lane;
      if (i < nfree && bst[j] >= 0) take_better(bk, bp, gain_key(bw[j], bc[j]), i);
    }
    wave_argmax(bk, bp);
    if (bp == INT32_MAX) {
      if (lane == 0) {
        GreedyEntry e;
        e.key = bk; e.c = 0.0; e.pos = INT32_MAX; e.stamp = 0;
        sh.ent[cblk] = e;
      }
    } else if (lane == (bp & 63)) {
      const int j = (bp & (kGBlock - 1)) >> 6;
      GreedyEntry e;
      e.key = bk; e.c = pick4(bc, j); e.pos = bp; e.stamp = pick4(bst, j);
      sh.ent[cblk] = e;
    }
  };

  while (t < kk) {
    if (wave == 0) {
      double bk = -__builtin_inf();
      int bp = INT32_MAX;
      for (int j = lane; j < nblk; j += 64) take_better(bk, bp, sh.ent[j].key, sh.ent[j].pos);
      wave_argmax(bk, bp);
      int op = kOpStop;
      if (bp < nfree) {
        const int b = bp / kGBlock;
        const GreedyEntry e = sh.ent[b];
        op = e.stamp == t ? kOpPick : kOpRefresh;
        if (b != cblk) {
#pragma unroll
          for (int j = 0; j < kGSlots; ++j) {
            const int i = b * kGBlock + j * 64 + lane;
            if (i < n) {
              bc[j] = gc[trow + i];
              bst[j] = gst[trow + i];
              bw[j] = wgt[trow + i];
            } else {
              bc[j] = 0.0; bst[j] = -1; bw[j] = 0.0f;
            }
          }
          cblk = b;
        }
        if (bp != utok) {
          fetch_row(bp);
          utok = bp;
        }
        if (op == kOpPick) {
          const int j = (bp & (kGBlock - 1)) >> 6;
          const double w = (double)__shfl(pick4(bw, j), bp & 63);
          pick_gain = w * e.c;
          if (lane == 0) sh.f = sqrt(w / (1.0 + pick_gain));
        }
      }
      if (lane == 0) { sh.op = op; sh.pos = bp; }
    }
    __syncthreads();
    const int op = sh.op, s = sh.pos;
    if (op == kOpStop) break;  // unreachable: an untaken position always remains
    const double partial = row_partial();
    if (op == kOpRefresh) {
      const double c = quad_form(partial);
      if (wave == 0) {
        const int j = (s & (kGBlock - 1)) >> 6;
        if (lane == (s & 63)) {
#pragma unroll
          for (int jj = 0; jj < kGSlots; ++jj)
            if (jj == j) { bc[jj] = c; bst[jj] = t; }
          gc[trow + s] = c;
          gst[trow + s] = t;
        }
        rescan();
      }
    } else {
      downdate(partial, sh.f);
      if (wave == 0) {
        const int j = (s & (kGBlock - 1)) >> 6;
        if (lane == (s & 63)) {
#pragma unroll
          for (int jj = 0; jj < kGSlots; ++jj)
            if (jj == j) bst[jj] = -1;
          gst[trow + s] = -1;
        }
        rescan();
        if (lane == 0) {
          logdet += log1p(pick_gain);
          sh.bits[s >> 5] |= 1u << (s & 31);
          if (order) order[t] = s;
        }
      }
      ++t;
    }
  }
  __syncthreads();

  // Kept positions in ascending order from the bitmap.
  const int per = (words + kThreads - 1) / kThreads;
  const int w0 = min(tid * per, words), w1 = min(w0 + per, words);
  uint32_t cnt = 0;
  for (int j = w0; j < w1; ++j) cnt += __popc(sh.bits[j]);
  uint32_t incl = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) sh.scan[wave] = incl;
  __syncthreads();
  uint32_t off = incl - cnt;
  for (int j = 0; j < wave; ++j) off += sh.scan[j];
  int32_t* out = idx_out + (int64_t)u * budget;
  for (int j = w0; j < w1; ++j) {
    uint32_t x = sh.bits[j];
    while (x) {
      const int bit = __ffs(x) - 1;
      out[off++] = j * 32 + bit;
      x &= x - 1u;
    }
  }
  for (int j = t + tid; j < budget; j += kThreads) {
    out[j] = -1;
    if (order) order[j] = -1;
  }
  if (logdet_out && tid == 0) logdet_out[u] = (double)D * log((double)ridge_f) + logdet;
}

hipError_t launch_greedy(const Launch& L, const void* v, int32_t* idx, int32_t* order,
                         double* logdet) {
  const Geo& g = L.geo;
  const int budget = L.cfg->budget_k;
  const int nblk_max = (g.maxn + kGBlock - 1) / kGBlock;
  const float* wb = ws_ptr<float>(L.wsp, L.ws.wgt);
  double* gc = ws_ptr<double>(L.wsp, L.ws.gc);
  int32_t* gst = ws_ptr<int32_t>(L.wsp, L.ws.gst);
  GreedyEntry* ent = ws_ptr<GreedyEntry>(L.wsp, L.ws.gent);
  const float ridge = L.cfg->ridge;
  const double* wsc = ws_ptr<double>(L.wsp, L.ws.wscale);
  const int protect = L.cfg->protect_last;
  const bool bf16 = L.cfg->dtype == JACAP_DTYPE_BF16;
  {
    TimedPhase tp(L.stream, JACAP_PHASE_GREEDY_INIT);
    if (nblk_max > 0) {
      const dim3 grid(nblk_max, g.U);
      auto go = [&](auto kern, auto vp) {
        kern<<<grid, kThreads, 0, L.stream>>>(g, vp, wb, ridge, wsc, budget, protect, gc, gst,
                                              ent, nblk_max);
      };
      if (bf16) {
        if (g.D == 128) go(greedy_init_kernel<128, uint16_t>, (const uint16_t*)v);
        else go(greedy_init_kernel<64, uint16_t>, (const uint16_t*)v);
      } else {
        if (g.D == 128) go(greedy_init_kernel<128, float>, (const float*)v);
        else go(greedy_init_kernel<64, float>, (const float*)v);
      }
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  TimedPhase tp(L.stream, JACAP_PHASE_GREEDY);
  auto go = [&](auto kern, auto vp) {
    kern<<<g.U, kThreads, 0, L.stream>>>(g, vp, wb, ridge, wsc, budget, protect, gc, gst, ent,
                                         nblk_max, idx, order, logdet);
  };
  if (bf16) {
    if (g.D == 128) go(greedy_kernel<128, uint16_t>, (const uint16_t*)v);
    else go(greedy_kernel<64, uint16_t>, (const uint16_t*)v);
  } else {
    if (g.D == 128) go(greedy_kernel<128, float>, (const float*)v);
    else go(greedy_kernel<64, float>, (const float*)v);
  }
  return hipGetLastError();
}

}  // namespace jacap
