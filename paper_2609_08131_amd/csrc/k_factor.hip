// Capacity matrix A = ridge I + M (Eq. 9) -- or R + M with a caller-supplied
// SPD matrix R (the output-projection variant) -- its Cholesky factor A = L L^T and
// the triangular inverse L^{-1}, one workgroup per unit, in fp64 in LDS.
// ||L^{-1} v||^2 = v^T A^{-1} v is what the leverage score of Eq. 10 needs.
//
// Input: the unit's Gram in block-lane layout (upper 16x16 blocks, see
// k_gram.hip): its per-chunk partials, summed here in chunk order in fp64, or
// (units of many chunks) the reduce kernel's sum of them. Output, after the
// first factorisation of an fp32-accumulated
// Gram (bf16 inputs): L^{-1} rounded to fp32 and split into bf16 hi + lo
// terms, stored directly in the per-lane B-fragment order of the 16x16x32
// MFMA (only the K-blocks that touch the lower triangle). After a
// factorisation of an fp64 Gram (fp32 inputs; the bf16 units marked for the
// fp64 path): L^{-1} in fp64, over the unit's slot of the reduced-Gram buffer
// in the lower-block layout -- block pair p = pair_index(i, j), i <= j, holds the
// 16x16 block X[16 j + r][16 i + c] at p * 256 + 16 r + c (zero above the
// diagonal of a diagonal block).
//
// Blocked algorithm on 16x16 blocks (the sequential chain is what bounds a
// single workgroup, so the work between barriers is made as wide as possible):
//   Cholesky, for each block column k:
//     1. the diagonal block is factored in registers by 16 lanes of wave 0
//        (lane s holds row s; each pivot's column is broadcast by DPP);
//     2. the panel below it is solved against it by forward substitution,
//        one row per thread;
//     3. the trailing lower triangle takes the rank-16 update, 4x4 register
//        tiles per thread.
//   Inverse X = L^{-1}:
//     4. the diagonal 16x16 blocks are inverted independently (one column per
//        lane);
//     5. block columns J from right to left: X_IJ = -(sum_{M > J} X_IM L_MJ)
//        X_JJ for every I > J at once (16x16 products on the fp64 MFMA).
// LDS holds only the lower 16x16 blocks of A (about 78 KB at d = 128, so two
// workgroups share a compute unit); L replaces A and X replaces L there,
// block by block as each part is consumed.
#include <algorithm>

#include "jacap_internal.hpp"

namespace jacap {

// Bound on cond(A) above which the bf16 path recomputes the unit in fp64: the
// fp32-accumulated two-term Gram and the two-term L^{-1} products carry errors
// that A^{-1} amplifies by up to cond(A) (~1e-8 cond(A) in the scores, so at
// most ~2e-4 below the threshold; the bound itself can exceed cond(A) by one
// or two orders of magnitude).
constexpr double kRefineCond = 2e4;
// Smallest pivot, relative to its diagonal entry, taken as positive. On the
// fp32-accumulated Gram a smaller one sends the unit to the fp64 path. On an
// fp64 Gram it means A is numerically singular at the score tolerance: a
// pivot ratio r implies cond(A) >= 1 / r, and fp64 rounding (any evaluation
// order, ~1e-14 relative in A) then moves the scores by about 5e-15 / r, so
// below 1e-13 / tol (1e-10 for the 1e-3 of bf16 inputs, 1e-8 for the 1e-5 of
// fp32 inputs) the scores are not determined to the tolerance -- at ridge 0,
// a rank-deficient M or a saturated softmax's weights spanning 1e30.
constexpr double kPivRelRefine = 1e-4;
constexpr double kPivRelSingularBf16 = 1e-10;
constexpr double kPivRelSingularFp32 = 1e-8;

// Eight waves: two per SIMD, so that one wave's LDS and fp64 latencies
// overlap the other's work (the capacity factorisation also has a
// four-wave shape, see factor_kernel).
constexpr int kFactorThreads = 512;

// Lane N of each 16-lane row, broadcast to the row (one 64-bit DPP move,
// row_newbcast).
template <int N>
__device__ __forceinline__ double row_bcast_f64(double v) {
  return __builtin_amdgcn_mov_dpp(v, 0x150 + N, 0xF, 0xF, false);
}
// The same for a lane index that is a constant once the caller's loop is
// unrolled.
__device__ __forceinline__ double row_bcast_f64_at(double v, int n) {
  switch (n) {
    case 0: return row_bcast_f64<0>(v);
    case 1: return row_bcast_f64<1>(v);
    case 2: return row_bcast_f64<2>(v);
    case 3: return row_bcast_f64<3>(v);
    case 4: return row_bcast_f64<4>(v);
    case 5: return row_bcast_f64<5>(v);
    case 6: return row_bcast_f64<6>(v);
    case 7: return row_bcast_f64<7>(v);
    case 8: return row_bcast_f64<8>(v);
    case 9: return row_bcast_f64<9>(v);
    case 10: return row_bcast_f64<10>(v);
    case 11: return row_bcast_f64<11>(v);
    case 12: return row_bcast_f64<12>(v);
    case 13: return row_bcast_f64<13>(v);
    case 14: return row_bcast_f64<14>(v);
    default: return row_bcast_f64<15>(v);
  }
}

// 1 / sqrt(x): the hardware estimate (relative error 2^-24.2, measured on
// the device) and Newton steps, one (2^-47.8) or two (2^-51.9, full fp64).
template <bool FULL>
__device__ __forceinline__ double rsqrt_f64(double x) {
  double y = __builtin_amdgcn_rsq(x);
  y = y * (1.5 - 0.5 * x * y * y);
  if constexpr (FULL) y = y * (1.5 - 0.5 * x * y * y);
  return y;
}

typedef double f64x4 __attribute__((ext_vector_type(4)));

// LDS layout of A (and of L, then X = L^{-1}, which replace it): only the
// lower 16x16 blocks (I >= J), packed by rows of blocks; block (I, J) starts
// at (I (I + 1) / 2 + J) * kBlk and holds element (r, c) at r * kBP + c. The
// pitch of 17 doubles puts the 16 rows of a block column in distinct banks.
// Diagonal blocks are stored whole (their upper halves serve as scratch).
constexpr int kBP = 17;
constexpr int kBlk = 16 * kBP;
__device__ __forceinline__ int lidx(int row, int col) {
  const int I = row >> 4, J = col >> 4;
  return (I * (I + 1) / 2 + J) * kBlk + (row & 15) * kBP + (col & 15);
}

// D += A B on the fp64 MFMA (16x16x4): lane l supplies A[l % 16][l / 16] and
// B[l / 16][l % 16]; element i of lane l's result is D[4 i + l / 16][l % 16].
__device__ __forceinline__ f64x4 mfma64(double a, double b, f64x4 acc) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
}

// Lower-triangle index e -> (row i, column j), j <= i (row-major over the triangle).
__device__ __forceinline__ void tri_index(int e, int& i, int& j) {
  int r = (int)((sqrtf(8.0f * (float)e + 1.0f) - 1.0f) * 0.5f);
  while ((r + 1) * (r + 2) / 2 <= e) ++r;
  while (r * (r + 1) / 2 > e) --r;
  i = r;
  j = e - r * (r + 1) / 2;
}

// Elements (u16) of one unit's two-term B fragments of a lower-triangular
// d x d matrix (see store_lower_frags).
__host__ __device__ constexpr int lower_frag_elems(int d) {
  return (d / 32) * (d / 32 + 1) * 2 * 64 * 8;
}

// A lower-triangular matrix X (x(a, b) = X[a][b] for b <= a) rounded to fp32
// and split into bf16 hi + lo terms, stored in the per-lane B-fragment order
// of the 16x16x32 MFMA for Y = V X^T: B fragment of output block j
// (a = 16 j + ch) and K block kb (b = 32 kb + 8 kg + q), only the pairs with
// kb <= j / 2 (the rest of X^T is zero); lane (ch, kg) holds 8 bf16, hi then
// lo.
template <int D, typename F>
__device__ __forceinline__ void store_lower_frags(uint16_t* __restrict__ out, F x) {
  constexpr int NB = D / 16;
  constexpr int NLP = (NB / 2) * (NB / 2 + 1);  // lower (j, kb) pairs: sum_j (j/2 + 1)
  static_assert(NLP * 2 * 64 * 8 == lower_frag_elems(D), "fragment count");
  for (int e = threadIdx.x; e < NLP * 64; e += blockDim.x) {
    const int qp = e / 64, ln = e % 64, ch = ln & 15, kg = ln >> 4;
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
      const float xv = (b <= a) ? (float)x(a, b) : 0.0f;
      const __bf16 h = (__bf16)xv;
      const __bf16 l = (__bf16)(xv - (float)h);
      hi[t] = __builtin_bit_cast(uint16_t, h);
      lo[t] = __builtin_bit_cast(uint16_t, l);
    }
    uint16_t* dh = out + ((int64_t)(qp * 2 + 0) * 64 + ln) * 8;
    uint16_t* dl = out + ((int64_t)(qp * 2 + 1) * 64 + ln) * 8;
#pragma unroll
    for (int t = 0; t < 8; ++t) { dh[t] = hi[t]; dl[t] = lo[t]; }
  }
}

// Blocked Cholesky A = L L^T in place on the lower blocks in LDS (see lidx),
// given dg = diag(A) before factorisation and *bad == 0 (both visible to
// every thread). idg receives 1 / L_rr. Returns 0, or the flag that stopped
// it -- kUnitNonfinite for a non-finite pivot, `fail` for a pivot at or below
// piv_rel times its diagonal entry -- the same value in every thread.
// FULL: the pivots' reciprocal square roots to full fp64 accuracy; else to
// 2^-47.8, for factors that are rounded to two bf16 terms afterwards.
template <int D, int NT, bool FULL>
__device__ __forceinline__ int cholesky_lds(double* A, const double* dg, double* idg, int* bad,
                                            double piv_rel, int fail) {
  constexpr int NB = D / 16;
  constexpr int NW = NT / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // 1. Diagonal block, in registers of wave 0: lane s (mod 16) holds row s.
  //    The chain from one pivot to the next is a broadcast, a reciprocal
  //    square root and one broadcast-FMA; the pivot thresholds are read
  //    before it starts and the checks stay off it.
  auto diag = [&](int kb) {
    const int c = 16 * kb;
    const int s = lane & 15;
    double a[16], thr[16], yv[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) a[q] = (q <= s) ? A[lidx((c + s), c + q)] : 0.0;
    // A pivot that has lost all but piv_rel of its diagonal entry is within
    // the rounding noise of A: A is numerically singular at the working
    // precision (or the caller's fail condition holds).
#pragma unroll
    for (int t = 0; t < 16; ++t) thr[t] = piv_rel * dg[c + t];
    // No early exit (the loop must stay fully unrolled so that a[] lives in
    // registers): after a failed pivot the rest is computed on whatever it
    // produced and discarded; the flag is the first failure's kind.
    bool failed = false, nonfinite = false;
    double piv = row_bcast_f64<0>(a[0]);  // A[t][t], from lane t of the row
    double y = rsqrt_f64<FULL>(piv);
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const bool ok = piv > thr[t] && piv > 0.0;
      if (!ok && !failed) nonfinite = !isfinite(piv);
      failed = failed || !ok;
      yv[t] = y;
      a[t] = (s == t) ? piv * y : a[t] * y;  // column t of L (rows s < t: unused)
      // a[q] -= L[s][t] L[q][t] for q > t; L[q][t] is lane q's a[t]. Entries
      // with q > s are outside row s's lower part and never stored. Row
      // t + 1 goes first, and the next pivot's reciprocal square root is
      // issued before the other rows' updates, which then fill its latency.
      double pn = 0.0, yn = 0.0;
      if (t + 1 < 16) {
        a[t + 1] = fma(-a[t], row_bcast_f64_at(a[t], t + 1), a[t + 1]);
        pn = row_bcast_f64_at(a[t + 1], t + 1);
        yn = rsqrt_f64<FULL>(pn);
      }
#pragma unroll
      for (int q = t + 2; q < 16; ++q) a[q] = fma(-a[t], row_bcast_f64_at(a[t], q), a[q]);
      piv = pn;
      y = yn;
    }
    const int code = failed ? (nonfinite ? (int)kUnitNonfinite : fail) : 0;
    if (code) {
      if (lane == 0) *bad = code;
    } else if (lane < 16) {
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (q <= s) A[lidx((c + s), c + q)] = a[q];
      if (lane == 0) {
#pragma unroll
        for (int t = 0; t < 16; ++t) idg[c + t] = yv[t];
      }
    }
  };
  // 3. Trailing update A_IJ -= L_Ik L_Jk^T of one 16x16 block (I >= J > k,
  //    block e of the trailing lower triangle, row-major) by one wave on the
  //    fp64 MFMA (K = 16 in four slices). Diagonal blocks also update their
  //    upper half, which is unused until the inverse overwrites it.
  auto update = [&](int kb, int e) {
    const int c = 16 * kb, r16 = lane & 15, q4 = lane >> 4;
    int bi, bj;
    tri_index(e, bi, bj);
    const int I = 16 * (kb + 1 + bi), J = 16 * (kb + 1 + bj);
    f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int kq = 0; kq < 4; ++kq) {
      const int t = c + 4 * kq + q4;
      acc = mfma64(A[lidx((I + r16), t)], A[lidx((J + r16), t)], acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) A[lidx((I + 4 * i + q4), J + r16)] -= acc[i];
  };
  if (wave == 0) diag(0);
  __syncthreads();
  if (*bad) return *bad;
  for (int kb = 0; kb < NB; ++kb) {
    const int c = 16 * kb;
    // 2. Panel rows r >= c + 16: L[r, c:c+16] = A[r, c:c+16] L_kk^{-T}.
    for (int r = c + 16 + tid; r < D; r += NT) {
      double x[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) x[t] = A[lidx(r, c + t)];
      // Row t of L_kk (columns < t) and 1 / L_tt are read one row ahead, so
      // that the chain does not wait on LDS.
      double lr[2][16], il[2];
      il[0] = idg[c];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        const int cur = t & 1, nxt = cur ^ 1;
        if (t + 1 < 16) {
#pragma unroll
          for (int q = 0; q <= t; ++q) lr[nxt][q] = A[lidx((c + t + 1), c + q)];
          il[nxt] = idg[c + t + 1];
        }
        // x[t] = (A[r][c+t] - sum_q x[q] L[c+t][c+q]) / L[c+t][c+t]; the sum in
        // four independent chains (latency, not order, bounds this loop)
        double sp[4] = {x[t], 0.0, 0.0, 0.0};
#pragma unroll
        for (int q = 0; q < t; ++q) sp[q & 3] = fma(-x[q], lr[cur][q], sp[q & 3]);
        x[t] = ((sp[0] + sp[1]) + (sp[2] + sp[3])) * il[cur];
      }
#pragma unroll
      for (int t = 0; t < 16; ++t) A[lidx(r, c + t)] = x[t];
    }
    __syncthreads();
    // Look-ahead: wave 0 updates the next diagonal block and factors it at
    // once, while the other waves take the rest of the trailing update, so
    // that the update is hidden behind the pivot chain.
    const int m = NB - kb - 1;
    if (m > 0) {
      if (wave == 0) {
        update(kb, 0);  // block (kb + 1, kb + 1)
        diag(kb + 1);
      } else {
        for (int e = wave; e < m * (m + 1) / 2; e += NW - 1) update(kb, e);
      }
      __syncthreads();
      if (*bad) return *bad;
    }
  }
  return 0;
}

// One unit. Its Gram: PASS 0 (all units) reads the reduced Gram `red` if the
// reduce kernel ran (`reduced`), else sums here, in chunk order, in fp64, the
// fp32 MFMA partials `part32` (bf16 inputs; gchunks per unit of gchunk tokens)
// or the fp64 partials `part` (fp32 inputs; pchunks of pchunk tokens) -- the
// reduce kernel's arithmetic; PASS 1 (the units of bf16 inputs that pass 0
// marked kUnitRefine) sums its fp64 partials. FRAGS: bf16 inputs.
template <int D, bool FRAGS, int NT>
__device__ __forceinline__ void factor_unit(const Geo& g, int u, double* __restrict__ red,
                                            const double* __restrict__ part, int pchunks,
                                            int pchunk, const float* __restrict__ part32,
                                            int gchunks, int gchunk, bool reduced,
                                            double ridge,
                                            const double* __restrict__ wscale, int pass,
                                            uint16_t* __restrict__ lfrag, uint32_t* status,
                                            uint32_t* uflags) {
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const Unit un = decode_unit(g, u);
  if (un.n == 0) return;
  // The fp32-accumulated Gram of bf16 inputs may be redone in fp64 later;
  // singularity is decided on an fp64 Gram only (pass 1, or fp32 inputs).
  const bool may_refine = FRAGS && pass == 0;
  const double piv_rel =
      may_refine ? kPivRelRefine : (FRAGS ? kPivRelSingularBf16 : kPivRelSingularFp32);

  __shared__ double A[NB * (NB + 1) / 2 * kBlk];  // lower 16x16 blocks, see lidx
  __shared__ double dg[D];   // diagonal of A before factorisation
  __shared__ double idg[D];  // 1 / L_rr
  __shared__ double red_sh[NT / 64];
  __shared__ double red_sh2[NT / 64];
  __shared__ int bad;        // 0, or the unit flag that stops the factorisation

  // Lower triangle of A = ridge I + M from the upper blocks of M. Entries
  // (2 e', 2 e' + 1) share a block pair and a lane: each thread loads its
  // pairs first (all loads in flight), then places them.
  constexpr int NE2 = NPAIR * 128;  // entry pairs
  constexpr int PER = (NE2 + NT - 1) / NT;
  double2 rv[PER];
  // Fixed-order sum of the unit's partials (the chunk loop unrolled so that
  // about 18 of a thread's loads are in flight; more spills registers).
  constexpr int CHU = PER <= 9 ? 2 : 1;
#pragma unroll
  for (int k = 0; k < PER; ++k) rv[k] = make_double2(0.0, 0.0);
  if (reduced && pass == 0) {
    const double2* R = reinterpret_cast<const double2*>(red + (int64_t)u * (NPAIR * 256));
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e2 = tid + k * NT;
      if (e2 < NE2) rv[k] = R[e2];
    }
  } else if (may_refine) {  // fp32 MFMA partials
    const int nch = (un.n + gchunk - 1) / gchunk;
    const float2* P = reinterpret_cast<const float2*>(part32 + (int64_t)u * gchunks * (NPAIR * 256));
#pragma unroll CHU
    for (int c = 0; c < nch; ++c) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int e2 = tid + k * NT;
        if (e2 < NE2) {
          const float2 x = P[(int64_t)c * NE2 + e2];
          rv[k].x += (double)x.x;
          rv[k].y += (double)x.y;
        }
      }
    }
  } else {  // fp64 partials
    const int nch = (un.n + pchunk - 1) / pchunk;
    const double2* P = reinterpret_cast<const double2*>(part + (int64_t)u * pchunks * (NPAIR * 256));
#pragma unroll CHU
    for (int c = 0; c < nch; ++c) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int e2 = tid + k * NT;
        if (e2 < NE2) {
          const double2 x = P[(int64_t)c * NE2 + e2];
          rv[k].x += x.x;
          rv[k].y += x.y;
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e2 = tid + k * NT;
    if (e2 < NE2) {
      const int e = 2 * e2;
      int p = e >> 8, bi = 0;  // block pair p -> block (bi, bj), bi <= bj, row-major
#pragma unroll
      for (int q = 0; q < NB; ++q)
        if (p >= NB - bi) { p -= NB - bi; ++bi; }
      const int bj = bi + p;
      const int ln = (e & 255) / 4, r = e % 4;  // r even: entries r and r + 1 of lane ln
      const int row = bi * 16 + (ln >> 4) * 4 + r;
      const int col = bj * 16 + (ln & 15);
      if (row <= col) A[lidx(col, row)] = rv[k].x;  // diagonal block: upper half only
      if (row + 1 <= col) A[lidx(col, row + 1)] = rv[k].y;
    }
  }
  if (tid == 0) bad = 0;
  __syncthreads();
  // The weights of a saturated softmax are stored times a power of two (the
  // weight pass's scale); the ridge term takes the same factor, so that A is
  // the capacity matrix times it and every score is unchanged.
  const double sc = wscale[u];
  if (g.ridge_mat) {  // output-projection variant: A = R + M
    const double* Rm = g.ridge_mat + ((int64_t)un.l * g.H + un.h) * D * D;
    for (int e = tid; e < D * D; e += NT) {
      const int r = e / D, cc = e % D;
      if (cc <= r) A[lidx(r, cc)] += Rm[e] * sc;
    }
    __syncthreads();
  }
  for (int a = tid; a < D; a += NT) {
    if (!g.ridge_mat) A[lidx(a, a)] += ridge * sc;
    dg[a] = A[lidx(a, a)];
    if (!isfinite(dg[a])) atomicOr(&bad, (int)kUnitNonfinite);
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) raise_flags(status, uflags, u, kUnitNonfinite);
    return;
  }

  // max over rows of sum_c |A[r][c]| (>= lambda_max(A), A symmetric with its
  // lower triangle stored); TPR threads per row.
  constexpr int TPR = NT / D;
  const int prow = tid / TPR, ppart = tid % TPR;
  // Row prow's entries and column prow's entries at b = ppart + TPR j: with
  // TPR dividing 16, b's block (TPR j / 16) and offset in it (TPR j mod 16,
  // plus ppart) are constants of j, so each address is a per-thread base plus
  // a constant. row_at(j): entry (prow, b), stored for b <= prow; col_at(j):
  // entry (b, prow), stored for b >= prow (other j give in-range addresses
  // whose values are not used).
  static_assert(16 % TPR == 0, "threads per row divide a block row");
  const int pI = prow >> 4, pr = prow & 15;
  const int rbase = (pI * (pI + 1) / 2) * kBlk + pr * kBP + ppart;
  const int cbase = pI * kBlk + ppart * kBP + pr;
  auto row_at = [&](int j) {
    const int Ib = (TPR * j) >> 4, o = (TPR * j) & 15;
    return rbase + Ib * kBlk + o;
  };
  auto col_at = [&](int j) {
    const int Ib = (TPR * j) >> 4, o = (TPR * j) & 15;
    return cbase + (Ib * (Ib + 1) / 2) * kBlk + o * kBP;
  };
  auto block_max = [&](double v) {
    v = wave_max_f64(v);
    __syncthreads();
    if (lane == 0) red_sh[wave] = v;
    __syncthreads();
    double m = red_sh[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) m = fmax(m, red_sh[w]);
    return m;
  };

  double anorm = 0.0;
  if (may_refine) {
    double sr = 0.0;
#pragma unroll 8
    for (int j = 0; j < D / TPR; ++j) {
      const int b = ppart + TPR * j;
      sr += fabs((b <= prow) ? A[row_at(j)] : A[col_at(j)]);
    }
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) sr += __shfl_xor(sr, o);
    anorm = block_max(sr);
  }

  // ---------------- Cholesky A = L L^T (L overwrites the lower triangle) ----
  // The first factorisation of bf16 inputs ends in two-term bf16 fragments
  // of L^{-1}; the fp64 paths keep full precision.
  const int code =
      may_refine ? cholesky_lds<D, NT, false>(A, dg, idg, &bad, piv_rel, (int)kUnitRefine)
                 : cholesky_lds<D, NT, true>(A, dg, idg, &bad, piv_rel, (int)kUnitSingular);
  if (code) {
    if (tid == 0) {
      if (code == (int)kUnitRefine) atomicOr(uflags + u, kUnitRefine);
      else raise_flags(status, uflags, u, (uint32_t)code);
    }
    return;
  }

  // ---------------- Inverse X = L^{-1} --------------------------------------
  // 4. Diagonal blocks: lane (k, t) computes column t of X_kk by forward
  //    substitution and stores X_kk[i][t] (i > t) at A[c + t][c + i] (the
  //    block's upper half; L_kk is still being read), then the block is
  //    copied down over L_kk with 1 / L_rr on the diagonal.
  if (tid < 16 * NB) {
    const int k = tid >> 4, t = tid & 15, c = 16 * k;
    double x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      double sum = 0.0;
#pragma unroll
      for (int q = 0; q < i; ++q) sum += A[lidx((c + i), c + q)] * x[q];
      x[i] = i < t ? 0.0 : (i == t ? idg[c + i] : -idg[c + i] * sum);
    }
#pragma unroll
    for (int i = 1; i < 16; ++i)
      if (i > t) A[lidx((c + t), c + i)] = x[i];
  }
  __syncthreads();
  for (int e = tid; e < NB * 256; e += NT) {
    const int c = 16 * (e >> 8), i = (e >> 4) & 15, t = e & 15;
    if (i > t) A[lidx((c + i), c + t)] = A[lidx((c + t), c + i)];
    else if (i == t) A[lidx((c + i), c + i)] = idg[c + i];
  }
  __syncthreads();
  // 5. Off-diagonal blocks of X, block column J from right to left, in place:
  //    X_IJ = -(sum_{M=J+1..I} X_IM L_MJ) X_JJ for I > J ((X L)_IJ = 0), where
  //    the blocks X_IM (M > J) are final and L_MJ still in place. One 16x16
  //    output block per wave on the fp64 MFMA; the sum is held in registers
  //    until every wave has read its operands, then stored over L_IJ, and
  //    the wave multiplies its own stored block by X_JJ at once (no other
  //    wave reads it until the next block column). The triangular X blocks
  //    are masked above their diagonal (their upper halves hold the
  //    temporaries of step 4).
  {
    const int r16 = lane & 15, q4 = lane >> 4;
    constexpr int NW = NT / 64;
    constexpr int PW = (NB - 1 + NW - 1) / NW;  // output blocks per wave, at most
    for (int J = NB - 2; J >= 0; --J) {
      // output blocks I = J + 1 + wave + NW p, p < PW
      f64x4 acc[PW];
#pragma unroll
      for (int p = 0; p < PW; ++p) {
        acc[p] = f64x4{0.0, 0.0, 0.0, 0.0};
        const int I = J + 1 + wave + NW * p;
        if (I < NB) {
          for (int M = J + 1; M <= I; ++M) {
            // the block step's operands, all loaded before its MFMAs
            double x[4], l[4];
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) {
              const int t = 4 * kq + q4;
              x[kq] = (M < I || r16 >= t) ? A[lidx(16 * I + r16, 16 * M + t)] : 0.0;
              l[kq] = A[lidx(16 * M + t, 16 * J + r16)];
            }
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) acc[p] = mfma64(x[kq], l[kq], acc[p]);
          }
        }
      }
      __syncthreads();  // every wave's reads of L_.J done
#pragma unroll
      for (int p = 0; p < PW; ++p) {
        const int I = J + 1 + wave + NW * p;
        if (I < NB) {
#pragma unroll
          for (int i = 0; i < 4; ++i) A[lidx(16 * I + 4 * i + q4, 16 * J + r16)] = acc[p][i];
          double tv[4], x[4];
#pragma unroll
          for (int kq = 0; kq < 4; ++kq) {
            const int t = 4 * kq + q4;
            tv[kq] = A[lidx(16 * I + r16, 16 * J + t)];
            x[kq] = t >= r16 ? A[lidx(16 * J + t, 16 * J + r16)] : 0.0;
          }
          f64x4 out = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
          for (int kq = 0; kq < 4; ++kq) out = mfma64(tv[kq], x[kq], out);
#pragma unroll
          for (int i = 0; i < 4; ++i) A[lidx(16 * I + 4 * i + q4, 16 * J + r16)] = -out[i];
        }
      }
      __syncthreads();  // X_.J visible to the next block column's products
    }
  }
  // X[r][c] (zero above the diagonal).
  auto xat = [&](int r, int cc) -> double { return r >= cc ? A[lidx(r, cc)] : 0.0; };

  auto xinv = xat;

  // cond(A) <= ||A||_inf ||L^{-1}||_1 ||L^{-1}||_inf (lambda_max <= ||A||_inf,
  // 1 / lambda_min = ||L^{-1}||_2^2 <= ||L^{-1}||_1 ||L^{-1}||_inf): a bound,
  // so no ill-conditioned unit escapes the refinement.
  if (may_refine) {
    double rs = 0.0, cs = 0.0;  // row prow's and column prow's absolute sums
#pragma unroll 8
    for (int j = 0; j < D / TPR; ++j) {
      const int b = ppart + TPR * j;
      rs += fabs(b <= prow ? A[row_at(j)] : 0.0);
      cs += fabs(b >= prow ? A[col_at(j)] : 0.0);
    }
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) {
      rs += __shfl_xor(rs, o);
      cs += __shfl_xor(cs, o);
    }
    // both maxima in one exchange (red_sh was last read before step 5's
    // barriers)
    const double wr = wave_max_f64(rs), wc = wave_max_f64(cs);
    if (lane == 0) { red_sh[wave] = wr; red_sh2[wave] = wc; }
    __syncthreads();
    double xinf = red_sh[0], x1 = red_sh2[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) {
      xinf = fmax(xinf, red_sh[w]);
      x1 = fmax(x1, red_sh2[w]);
    }
    if (anorm * x1 * xinf > kRefineCond) {
      if (tid == 0) atomicOr(uflags + u, kUnitRefine);
      return;  // pass 1 writes this unit's L^{-1}
    }
  }

  // Store L^{-1}.
  if (!may_refine) {  // fp64, over the unit's slot of the reduced-Gram buffer
    double* o64 = red + (int64_t)u * (NPAIR * 256);
    for (int e = tid; e < NPAIR * 256; e += NT) {
      int p = e >> 8, bi = 0;  // block pair p -> (bi, bj), bi <= bj
#pragma unroll
      for (int q = 0; q < NB; ++q)
        if (p >= NB - bi) { p -= NB - bi; ++bi; }
      const int bj = bi + p;
      o64[e] = xinv(16 * bj + ((e >> 4) & 15), 16 * bi + (e & 15));
    }
  } else {
    store_lower_frags<D>(lfrag + (int64_t)u * lower_frag_elems(D), xinv);
  }
}

// PASS 0: one workgroup per unit. PASS 1: a grid-stride walk over the units
// that skips those not marked kUnitRefine. NT threads: 512 (eight waves)
// when the units fit the compute units in one round; 256 (bounded to 256
// VGPRs, so that two workgroups share a compute unit and one's sequential
// steps overlap the other's) when there are more.
template <int D, bool FRAGS, int NT>
__global__ __launch_bounds__(NT, 512 / NT) void factor_kernel(
    Geo g, double* __restrict__ red, const double* __restrict__ part, int pchunks, int pchunk,
    const float* __restrict__ part32, int gchunks, int gchunk, int reduced, double ridge,
    const double* __restrict__ wscale, int pass, uint16_t* __restrict__ lfrag, uint32_t* status,
    uint32_t* uflags) {
  for (int u = blockIdx.x; u < g.U; u += gridDim.x) {
    if (pass == 1 && !(uflags[u] & kUnitRefine)) continue;
    factor_unit<D, FRAGS, NT>(g, u, red, part, pchunks, pchunk, part32, gchunks, gchunk,
                              reduced != 0, ridge, wscale, pass, lfrag, status, uflags);
    __syncthreads();  // LDS of this unit fully consumed before the next one's loads
  }
}

hipError_t launch_factor(const Launch& L, bool refine) {
  if (refine && !L.ws.mfma) return hipSuccess;
  const int pass = refine ? 1 : 0;
  const Geo& g = L.geo;
  double* red = ws_ptr<double>(L.wsp, L.ws.gram_red);
  uint16_t* lf = ws_ptr<uint16_t>(L.wsp, L.ws.lfrag);
  uint32_t* st = ws_ptr<uint32_t>(L.wsp, L.ws.status);
  uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  const double* wsc = ws_ptr<double>(L.wsp, L.ws.wscale);
  const double ridge = (double)L.cfg->ridge;
  // the Gram partials: fp64 (fp32 inputs, and the refine pass), fp32 (the
  // first pass of bf16 inputs); both in the Gram buffer
  const double* part = ws_ptr<double>(L.wsp, L.ws.gram);
  const float* part32 = ws_ptr<float>(L.wsp, L.ws.gram);
  const int blocks = refine ? std::min(g.U, kRefineBlocks) : g.U;
  const bool pairs = !refine && g.U > kComputeUnits;  // two workgroups per compute unit
  auto go = [&](auto kern, int nt) {
    kern<<<blocks, nt, 0, L.stream>>>(g, red, part, L.ws.pchunks, L.ws.pchunk, part32,
                                      L.ws.gchunks, L.ws.gchunk, gram_reduced(L) ? 1 : 0, ridge,
                                      wsc, pass, lf, st, uf);
  };
  if (L.ws.mfma) {
    if (g.D == 128) pairs ? go(factor_kernel<128, true, 256>, 256) : go(factor_kernel<128, true, 512>, 512);
    else pairs ? go(factor_kernel<64, true, 256>, 256) : go(factor_kernel<64, true, 512>, 512);
  } else {
    if (g.D == 128) pairs ? go(factor_kernel<128, false, 256>, 256) : go(factor_kernel<128, false, 512>, 512);
    else pairs ? go(factor_kernel<64, false, 256>, 256) : go(factor_kernel<64, false, 512>, 512);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// FULL covariance, triangular K pass (full_kpass_tri): per unit, Lambda_Q of
// the pooled window in fp64 and a factor Lambda_Q = X^T X with X lower
// triangular, stored as two-term bf16 B fragments (store_lower_frags) in the
// L^{-1} fragment buffer, which is free until the capacity matrix is factored.
// Then kappa_i = k_i^T Lambda_Q k_i = ||X k_i||^2 (Sec. 3.4, full query
// covariance) takes the leverage pass's triangular MFMA product.
//
// X comes from the Cholesky factorisation of the order-reversed matrix:
// P Lambda_Q P = C C^T (P reverses the channel order, C lower triangular)
// gives Lambda_Q = (P C P)(P C P)^T with P C P upper triangular, so
// X = (P C P)^T, X[i][j] = C[d-1-j][d-1-i].
//
// Lambda_Q = (1/N_s) sum_r (q_r - mu)(q_r - mu)^T: the window (raw bf16, all
// of it in LDS) goes through the fp64 MFMA, each row centred in fp64 as it is
// read, each wave accumulating its share of the 16x16 lower blocks in
// registers; the blocks are then written to the factor's LDS layout already
// reversed.
//
// The unit is marked kUnitKTile (the K pass takes the window tile) if it has
// fewer than kTriMinTokens tokens, non-finite window statistics, or a pivot at
// most kPivRelTri of its diagonal entry: a numerically rank-deficient
// Lambda_Q, whose factor would not carry kappa to the tolerance in two bf16
// terms.
// ---------------------------------------------------------------------------
constexpr double kPivRelTri = 1e-3;

template <int D>
__device__ __forceinline__ void qfactor_unit(const Geo& g, int u, const uint16_t* __restrict__ q,
                                             const double* __restrict__ mu,
                                             uint16_t* __restrict__ xfrag,
                                             uint32_t* __restrict__ uflags) {
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  constexpr int NW = kFactorThreads / 64;
  constexpr int PW = (NPAIR + NW - 1) / NW;  // lower 16x16 blocks of Lambda_Q per wave
  constexpr int QPB = D + 8;  // u16 per staged window row
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, q4 = lane >> 4;
  const Unit un = decode_unit(g, u);
  if (un.n == 0) return;
  if (un.n < kTriMinTokens || (uflags[u] & kUnitNonfinite)) {
    if (tid == 0) atomicOr(uflags + u, kUnitKTile);
    return;
  }
  __shared__ double A[NPAIR * kBlk];  // lower 16x16 blocks, see lidx
  __shared__ double dg[D];
  __shared__ double idg[D];
  __shared__ double smu[D];
  __shared__ __attribute__((aligned(16))) uint16_t qs[kFullMaxQ * QPB];  // the window, raw bf16
  __shared__ int bad;

  const int Ns = g.G * g.w;
  const uint16_t* qb =
      q + un.b * g.qss + un.l * g.qsl + (int64_t)(un.h * g.V + un.s) * g.G * g.qsh;
  for (int c = tid; c < D; c += kFactorThreads) smu[c] = mu[(int64_t)u * D + c];
  if (tid == 0) bad = 0;
  // The whole window in one round of 16-byte loads (N_s <= kFullMaxQ rows),
  // then the products over it with no further barrier. Rows N_s .. N_s4 - 1
  // are padding and masked.
  const int Ns4 = (Ns + 3) & ~3;
  for (int e = tid; e < Ns4 * (D / 8); e += kFactorThreads) {
    const int r = e / (D / 8), pc = e - r * (D / 8);
    uint4 x = make_uint4(0u, 0u, 0u, 0u);
    if (r < Ns) {
      const int gq = r / g.w, p = r - gq * g.w;
      x = *reinterpret_cast<const uint4*>(qb + gq * g.qsh + p * g.qsp + pc * 8);
    }
    *reinterpret_cast<uint4*>(qs + r * QPB + pc * 8) = x;
  }
  __syncthreads();  // window and smu visible
  // block (bi, bj), bi >= bj: sum_r (q_r - mu)[16 bi + i] (q_r - mu)[16 bj + j],
  // four rows per MFMA (lane (r16, q4) supplies row 4 s + q4, column r16 of
  // each), centred in fp64 as they are read; the wave's blocks take turns so
  // that their accumulation chains interleave.
  f64x4 acc[PW];
  int cbi[PW], cbj[PW];
  double mbi[PW], mbj[PW];
  // A wave's slots past the last block repeat that block (no branch in the
  // loop below); their sums are not stored.
#pragma unroll
  for (int p = 0; p < PW; ++p) {
    acc[p] = f64x4{0.0, 0.0, 0.0, 0.0};
    const int e = min(wave + NW * p, NPAIR - 1);
    int bi, bj;
    tri_index(e, bi, bj);
    cbi[p] = 16 * bi + r16;
    cbj[p] = 16 * bj + r16;
    mbi[p] = smu[cbi[p]];
    mbj[p] = smu[cbj[p]];
  }
  // Each row group's raw values are read while the previous group's MFMAs
  // run (the last read repeats the last group and is not used).
  uint16_t na[PW], nb[PW];
#pragma unroll
  for (int p = 0; p < PW; ++p) {
    na[p] = qs[q4 * QPB + cbi[p]];
    nb[p] = qs[q4 * QPB + cbj[p]];
  }
  for (int r = q4; r < Ns4; r += 4) {
    uint16_t ca[PW], cb[PW];
#pragma unroll
    for (int p = 0; p < PW; ++p) { ca[p] = na[p]; cb[p] = nb[p]; }
    const uint16_t* nrow = qs + min(r + 4, Ns4 - 4 + q4) * QPB;
#pragma unroll
    for (int p = 0; p < PW; ++p) {
      na[p] = nrow[cbi[p]];
      nb[p] = nrow[cbj[p]];
    }
    __builtin_amdgcn_sched_barrier(0);  // the next group's reads stay ahead of these MFMAs
    const double live = r < Ns ? 1.0 : 0.0;  // a factor, not a branch
#pragma unroll
    for (int p = 0; p < PW; ++p) {
      const double xa = ((double)bf16_to_f32(ca[p]) - mbi[p]) * live;
      const double xb = (double)bf16_to_f32(cb[p]) - mbj[p];
      acc[p] = mfma64(xa, xb, acc[p]);
    }
  }
  // Lambda_Q[row][col] (row >= col) goes to the reversed matrix at
  // (d-1-col, d-1-row), a lower entry; diagonal blocks are written whole.
  const double invn = 1.0 / (double)Ns;
#pragma unroll
  for (int p = 0; p < PW; ++p) {
    const int e = wave + NW * p;
    if (e < NPAIR) {
      int bi, bj;
      tri_index(e, bi, bj);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * bi + 4 * i + q4, col = 16 * bj + r16;
        A[lidx(D - 1 - col, D - 1 - row)] = acc[p][i] * invn;
      }
    }
  }
  __syncthreads();
  for (int a = tid; a < D; a += kFactorThreads) dg[a] = A[lidx(a, a)];
  __syncthreads();
  if (cholesky_lds<D, kFactorThreads, false>(A, dg, idg, &bad, kPivRelTri, (int)kUnitKTile) != 0) {
    if (tid == 0) atomicOr(uflags + u, kUnitKTile);
    return;
  }
  store_lower_frags<D>(xfrag + (int64_t)u * lower_frag_elems(D),
                       [&](int a, int b) { return A[lidx(D - 1 - b, D - 1 - a)]; });
}

// One workgroup per unit (a grid-stride walk if the grid is smaller).
template <int D>
__global__ __launch_bounds__(kFactorThreads) void qfactor_kernel(Geo g, const uint16_t* __restrict__ q,
                                                                 const double* __restrict__ mu,
                                                                 uint16_t* __restrict__ xfrag,
                                                                 uint32_t* __restrict__ uflags) {
  for (int u = blockIdx.x; u < g.U; u += gridDim.x) {
    qfactor_unit<D>(g, u, q, mu, xfrag, uflags);
    __syncthreads();  // LDS of this unit fully consumed before the next one's
  }
}

hipError_t launch_qfactor(const Launch& L, const void* q) {
  const Geo& g = L.geo;
  if (g.U == 0) return hipSuccess;
  // The fragments go to the L^{-1} fragment section, which every layout that
  // can take this path reserves (offset 0 is the status word's).
  if (L.ws.lfrag == 0) return hipErrorInvalidValue;
  auto go = [&](auto kern) {
    kern<<<g.U, kFactorThreads, 0, L.stream>>>(g, (const uint16_t*)q,
                                                ws_ptr<double>(L.wsp, L.ws.mu),
                                                ws_ptr<uint16_t>(L.wsp, L.ws.lfrag),
                                                ws_ptr<uint32_t>(L.wsp, L.ws.uflags));
  };
  if (g.D == 128) go(qfactor_kernel<128>);
  else go(qfactor_kernel<64>);
  return hipGetLastError();
}

}  // namespace jacap
