// Capacity matrix A = ridge I + M (Eq. 9), its Cholesky factor A = L L^T and
// the triangular inverse L^{-1}, one workgroup per unit, in fp64 in LDS.
// ||L^{-1} v||^2 = v^T A^{-1} v is what the leverage score of Eq. 10 needs.
//
// Input: the reduced Gram in block-lane layout (upper 16x16 blocks, see
// k_gram.hip). Output: L^{-1} in fp64 (fp32-input path), or, for the bf16
// MFMA leverage pass, L^{-1} rounded to fp32 and split into bf16 hi + lo
// terms, stored directly in the per-lane B-fragment order of the
// 16x16x32 MFMA (only the K-blocks that touch the lower triangle).
#include "jacap_internal.hpp"

namespace jacap {

// y = op(x) for the matrix held in LDS (row pitch D + 1). MODE 0: the
// symmetric A stored in its lower triangle; MODE 1: the lower-triangular X
// itself; MODE 2: its transpose X^T.
template <int D, int MODE>
__device__ __forceinline__ void sym_matvec(const double* A, const double* x, double* y) {
  constexpr int LD = D + 1;
  constexpr int TPR = kThreads / D;  // threads per output entry
  const int tid = threadIdx.x, row = tid / TPR, part = tid % TPR;
  double s = 0.0;
  for (int b = part; b < D; b += TPR) {
    double a;
    if constexpr (MODE == 0) a = (b <= row) ? A[row * LD + b] : A[b * LD + row];
    else if constexpr (MODE == 1) a = (b <= row) ? A[row * LD + b] : 0.0;
    else a = (b >= row) ? A[b * LD + row] : 0.0;
    s += a * x[b];
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o);
  if (part == 0) y[row] = s;
  __syncthreads();
}

// x <- y / ||y||; returns ||y|| (uniform).
template <int D>
__device__ __forceinline__ double normalize(double* x, const double* y, double* red) {
  const int tid = threadIdx.x;
  const double v = tid < D ? y[tid] * y[tid] : 0.0;
  const double nrm = sqrt(block_combine(wave_sum(v), red, [](double a, double b) { return a + b; }));
  if (tid < D) x[tid] = nrm > 0.0 ? y[tid] / nrm : 0.0;
  __syncthreads();
  return nrm;
}

constexpr int kPowerIters = 8;
// cond(A) estimate above which the bf16 path recomputes the unit's Gram with
// the exact three-term split (its two-term error grows like ~1e-8 cond(A)).
constexpr double kRefineCond = 2e3;

// PASS 0: first factorisation (all units). PASS 1: refinement of the units
// marked kUnitRefine by pass 0 (bf16 path), from their exact-split Gram.
template <int D, bool FRAGS>
__global__ __launch_bounds__(kThreads) void factor_kernel(Geo g, const double* __restrict__ red,
                                                          double ridge, double piv_rel, int pass,
                                                          double* __restrict__ linv64,
                                                          uint16_t* __restrict__ lfrag,
                                                          uint32_t* status, uint32_t* uflags) {
  constexpr int LD = D + 1;
  constexpr int NB = D / 16;
  constexpr int NK = D / 32;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  const int u = blockIdx.x, tid = threadIdx.x;
  if (pass == 1 && !(uflags[u] & kUnitRefine)) return;
  const Unit un = decode_unit(g, u);
  if (un.n == 0) return;
  // The two-term bf16 Gram may be refined later; singularity is decided on
  // the exact one (pass 1) or on the fp64 one (fp32 inputs).
  const bool may_refine = FRAGS && pass == 0;

  __shared__ double A[D * LD];
  __shared__ double dg[D];
  __shared__ double tmp[D];
  __shared__ double px[D], py[D], pred[kThreads / 64];
  __shared__ int bad;

  // 1. Lower triangle of A = ridge I + M from the upper blocks of M.
  const double* R = red + (int64_t)u * (NPAIR * 256);
  for (int e = tid; e < NPAIR * 256; e += kThreads) {
    const int p = e / 256, rem = e % 256, lane = rem / 4, r = rem % 4;
    int i = 0, j = 0, q = p;
    for (int ii = 0; ii < NB; ++ii) {
      const int cnt = NB - ii;
      if (q < cnt) { i = ii; j = ii + q; break; }
      q -= cnt;
    }
    const int row = i * 16 + (lane >> 4) * 4 + r;
    const int col = j * 16 + (lane & 15);
    if (row > col) continue;       // diagonal block: keep the upper half
    A[col * LD + row] = R[e];      // lower-triangle slot (col >= row)
  }
  __syncthreads();
  if (tid == 0) bad = 0;
  __syncthreads();
  for (int a = tid; a < D; a += kThreads) {
    A[a * LD + a] += ridge;
    dg[a] = A[a * LD + a];
    if (!isfinite(dg[a])) atomicOr(&bad, 1);
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) raise_flags(status, uflags, u, kUnitNonfinite);
    return;
  }

  // lambda_max(A) by power iteration (a lower estimate).
  if (tid < D) px[tid] = 1.0 + 0.01 * tid;
  __syncthreads();
  double lam_max = normalize<D>(px, px, pred);
  for (int it = 0; it < kPowerIters; ++it) {
    sym_matvec<D, 0>(A, px, py);
    lam_max = normalize<D>(px, py, pred);
  }

  // 2. Right-looking Cholesky, A <- L (lower).
  const int ty = tid / 16, tx = tid % 16;
  for (int j = 0; j < D; ++j) {
    const double piv = A[j * LD + j];
    // A pivot that has lost all but piv_rel of its diagonal entry is within the
    // rounding noise of the accumulated Gram: A is numerically singular at the
    // path's working precision (rank-deficient M with ridge 0).
    if (!(piv > piv_rel * dg[j]) || !(piv > 0.0)) {
      if (tid == 0) {
        if (!isfinite(piv)) raise_flags(status, uflags, u, kUnitNonfinite);
        else if (may_refine) atomicOr(uflags + u, kUnitRefine);
        else raise_flags(status, uflags, u, kUnitSingular);
      }
      return;  // uniform: every thread read the same pivot
    }
    const double ljj = sqrt(piv);
    const double inv = 1.0 / ljj;
    __syncthreads();
    for (int i = j + 1 + tid; i < D; i += kThreads) A[i * LD + j] *= inv;
    __syncthreads();
    if (tid == 0) A[j * LD + j] = ljj;
    for (int i = j + 1 + ty; i < D; i += 16) {
      const double lij = A[i * LD + j];
      for (int kk = j + 1 + tx; kk <= i; kk += 16) A[i * LD + kk] -= lij * A[kk * LD + j];
    }
    __syncthreads();
  }

  // 3. In-place inverse of the lower-triangular L (column by column from the
  //    right): column j of L^{-1} is -L^{-1}_{jj} * T * L[j+1:, j], with T the
  //    already-inverted trailing block.
  //    Each row's dot product is split over a 16-lane group (lanes sub, sub+16,
  //    ...) and reduced with butterflies inside the group.
  const int grp = tid >> 4, sub = tid & 15;
  for (int j = D - 1; j >= 0; --j) {
    const double ajj = 1.0 / A[j * LD + j];
    for (int i = j + 1 + tid; i < D; i += kThreads) tmp[i] = A[i * LD + j];
    __syncthreads();
    for (int i0 = j + 1; i0 < D; i0 += kThreads / 16) {
      const int i = i0 + grp;
      double s = 0.0;
      if (i < D)
        for (int kk = j + 1 + sub; kk <= i; kk += 16) s += A[i * LD + kk] * tmp[kk];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o);
      if (i < D && sub == 0) A[i * LD + j] = -ajj * s;
    }
    __syncthreads();
    if (tid == 0) A[j * LD + j] = ajj;
    __syncthreads();
  }

  // 1 / lambda_min(A) = ||L^{-1}||_2^2 by power iteration on L^{-T} L^{-1}.
  if (may_refine) {
    if (tid < D) px[tid] = 1.0 + 0.01 * tid;
    __syncthreads();
    normalize<D>(px, px, pred);
    double inv_min = 0.0;
    for (int it = 0; it < kPowerIters; ++it) {
      sym_matvec<D, 1>(A, px, py);   // py = L^{-1} px
      sym_matvec<D, 2>(A, py, tmp);  // tmp = L^{-T} py
      inv_min = normalize<D>(px, tmp, pred);
    }
    if (lam_max * inv_min > kRefineCond) {
      if (tid == 0) atomicOr(uflags + u, kUnitRefine);
      return;  // pass 1 writes this unit's L^{-1}
    }
  }

  // 4. Store L^{-1}.
  if constexpr (!FRAGS) {
    double* o64 = linv64 + (int64_t)u * D * D;
    for (int e = tid; e < D * D; e += kThreads) {
      const int a = e / D, b = e % D;
      o64[e] = (b <= a) ? A[a * LD + b] : 0.0;
    }
  } else {
    // B fragment of output block j (a = 16 j + ch) and K block kb
    // (b = 32 kb + 8 kg + q): lane (ch, kg) holds 8 bf16; hi then lo.
    constexpr int NLP = (NB / 2) * (NB / 2 + 1);  // lower (j, kb) pairs: sum_j (j/2 + 1)
    uint16_t* out = lfrag + (int64_t)u * NLP * 2 * 64 * 8;
    for (int e = tid; e < NLP * 64; e += kThreads) {
      const int qp = e / 64, lane = e % 64, ch = lane & 15, kg = lane >> 4;
      int j = 0, kb = 0, q = qp;
      for (int jj = 0; jj < NB; ++jj) {
        const int cnt = jj / 2 + 1;
        if (q < cnt) { j = jj; kb = q; break; }
        q -= cnt;
      }
      const int a = 16 * j + ch;
      uint16_t hi[8], lo[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int b = 32 * kb + 8 * kg + t;
        const float x = (b <= a) ? (float)A[a * LD + b] : 0.0f;
        const __bf16 h = (__bf16)x;
        const __bf16 l = (__bf16)(x - (float)h);
        hi[t] = __builtin_bit_cast(uint16_t, h);
        lo[t] = __builtin_bit_cast(uint16_t, l);
      }
      uint16_t* dh = out + ((int64_t)(qp * 2 + 0) * 64 + lane) * 8;
      uint16_t* dl = out + ((int64_t)(qp * 2 + 1) * 64 + lane) * 8;
#pragma unroll
      for (int t = 0; t < 8; ++t) { dh[t] = hi[t]; dl[t] = lo[t]; }
    }
  }
  (void)NK;
}

hipError_t launch_factor(const Launch& L, bool refine) {
  if (refine && !L.ws.mfma) return hipSuccess;
  const int pass = refine ? 1 : 0;
  const Geo& g = L.geo;
  const double* red = ws_ptr<double>(L.wsp, L.ws.gram_red);
  double* l64 = ws_ptr<double>(L.wsp, L.ws.linv64);
  uint16_t* lf = ws_ptr<uint16_t>(L.wsp, L.ws.lfrag);
  uint32_t* st = ws_ptr<uint32_t>(L.wsp, L.ws.status);
  uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  const double ridge = (double)L.cfg->ridge;
  // fp32-accumulated Gram (bf16 path) carries ~1e-6 relative noise; the fp64
  // path ~1e-15.
  const double piv_rel = L.ws.mfma ? 1e-4 : 1e-12;
  if (L.ws.mfma) {
    if (g.D == 128) factor_kernel<128, true><<<g.U, kThreads, 0, L.stream>>>(g, red, ridge, piv_rel, pass, l64, lf, st, uf);
    else factor_kernel<64, true><<<g.U, kThreads, 0, L.stream>>>(g, red, ridge, piv_rel, pass, l64, lf, st, uf);
  } else {
    if (g.D == 128) factor_kernel<128, false><<<g.U, kThreads, 0, L.stream>>>(g, red, ridge, piv_rel, pass, l64, lf, st, uf);
    else factor_kernel<64, false><<<g.U, kThreads, 0, L.stream>>>(g, red, ridge, piv_rel, pass, l64, lf, st, uf);
  }
  return hipGetLastError();
}

}  // namespace jacap
