// Capacity matrix A = ridge I + M (Eq. 9), its Cholesky factor A = L L^T and
// the triangular inverse L^{-1}, one workgroup per unit, in fp64 in LDS.
// ||L^{-1} v||^2 = v^T A^{-1} v is what the leverage score of Eq. 10 needs.
//
// Input: the reduced Gram in block-lane layout (upper 16x16 blocks, see
// k_gram.hip). Output: L^{-1} in fp64 (fp32-input path), or, for the bf16
// MFMA leverage pass, L^{-1} rounded to fp32 and split into bf16 hi + lo
// terms, stored directly in the per-lane B-fragment order of the
// 16x16x32 MFMA (only the K-blocks that touch the lower triangle).
//
// Blocked algorithm on 16x16 blocks (the sequential chain is what bounds a
// single workgroup, so the work between barriers is made as wide as possible):
//   Cholesky, for each block column k:
//     1. wave 0 factors the diagonal block (16 pivots, wave-synchronous);
//     2. the panel below it is solved against it by forward substitution,
//        one row per thread;
//     3. the trailing lower triangle takes the rank-16 update, 4x4 register
//        tiles per thread.
//   Inverse X = L^{-1}:
//     4. the diagonal blocks are inverted independently (one column per lane);
//     5. off-diagonal blocks follow block diagonal by block diagonal:
//        X_ij = -X_ii (sum_{k=j}^{i-1} L_ik X_kj).
// LDS holds A (pitch D + 1) with L in its lower triangle; X is written
// transposed into the upper triangle (X[r][c] at A[c][r], r > c) and its
// diagonal 1 / L_rr is kept in idg.
#include "jacap_internal.hpp"

namespace jacap {

// Orders LDS accesses of the lanes of one wave (no workgroup barrier).
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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

// Lower-triangle index e -> (row i, column j), j <= i (row-major over the triangle).
__device__ __forceinline__ void tri_index(int e, int& i, int& j) {
  int r = (int)((sqrtf(8.0f * (float)e + 1.0f) - 1.0f) * 0.5f);
  while ((r + 1) * (r + 2) / 2 <= e) ++r;
  while (r * (r + 1) / 2 > e) --r;
  i = r;
  j = e - r * (r + 1) / 2;
}

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
  constexpr int NPAIR = NB * (NB + 1) / 2;
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (pass == 1 && !(uflags[u] & kUnitRefine)) return;
  const Unit un = decode_unit(g, u);
  if (un.n == 0) return;
  // The two-term bf16 Gram may be refined later; singularity is decided on
  // the exact one (pass 1) or on the fp64 one (fp32 inputs).
  const bool may_refine = FRAGS && pass == 0;

  __shared__ double A[D * LD];
  __shared__ double dg[D];   // diagonal of A before factorisation
  __shared__ double idg[D];  // 1 / L_rr
  __shared__ double px[D], py[D], pred[kThreads / 64];
  __shared__ int bad;        // 0, or the unit flag that stops the factorisation

  // Lower triangle of A = ridge I + M from the upper blocks of M.
  const double* R = red + (int64_t)u * (NPAIR * 256);
  for (int e = tid; e < NPAIR * 256; e += kThreads) {
    const int p = e / 256, rem = e % 256, ln = rem / 4, r = rem % 4;
    int i = 0, j = 0, q = p;
    for (int ii = 0; ii < NB; ++ii) {
      const int cnt = NB - ii;
      if (q < cnt) { i = ii; j = ii + q; break; }
      q -= cnt;
    }
    const int row = i * 16 + (ln >> 4) * 4 + r;
    const int col = j * 16 + (ln & 15);
    if (row > col) continue;       // diagonal block: keep the upper half
    A[col * LD + row] = R[e];      // lower-triangle slot (col >= row)
  }
  if (tid == 0) bad = 0;
  __syncthreads();
  for (int a = tid; a < D; a += kThreads) {
    A[a * LD + a] += ridge;
    dg[a] = A[a * LD + a];
    if (!isfinite(dg[a])) atomicOr(&bad, (int)kUnitNonfinite);
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) raise_flags(status, uflags, u, kUnitNonfinite);
    return;
  }

  // lambda_max(A) by power iteration (a lower estimate); A is symmetric with
  // its lower triangle stored.
  constexpr int TPR = kThreads / D;  // threads per row in the matrix-vector products
  const int prow = tid / TPR, ppart = tid % TPR;
  double lam_max = 0.0;
  if (may_refine) {
    if (tid < D) px[tid] = 1.0 + 0.01 * tid;
    __syncthreads();
    normalize<D>(px, px, pred);
    for (int it = 0; it < kPowerIters; ++it) {
      double s = 0.0;
      for (int b = ppart; b < D; b += TPR)
        s += ((b <= prow) ? A[prow * LD + b] : A[b * LD + prow]) * px[b];
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o);
      if (ppart == 0) py[prow] = s;
      __syncthreads();
      lam_max = normalize<D>(px, py, pred);
    }
  }

  // ---------------- Cholesky A = L L^T (L overwrites the lower triangle) ----
  for (int kb = 0; kb < NB; ++kb) {
    const int c = 16 * kb;
    // 1. Diagonal block, by wave 0.
    if (wave == 0) {
      for (int t = 0; t < 16; ++t) {
        const int jj = c + t;
        const double piv = A[jj * LD + jj];
        // A pivot that has lost all but piv_rel of its diagonal entry is within
        // the rounding noise of the accumulated Gram: A is numerically singular
        // at the path's working precision (rank-deficient M with ridge 0).
        if (!(piv > piv_rel * dg[jj]) || !(piv > 0.0)) {
          if (lane == 0) bad = !isfinite(piv) ? (int)kUnitNonfinite
                               : (may_refine ? (int)kUnitRefine : (int)kUnitSingular);
          break;  // uniform: every lane read the same pivot
        }
        const double y = 1.0 / sqrt(piv);
        if (lane < 15 - t) A[(jj + 1 + lane) * LD + jj] *= y;
        if (lane == 0) { A[jj * LD + jj] = piv * y; idg[jj] = y; }
        wave_sync_lds();
        // rank-1 update of the block's trailing lower triangle
        const int m = 15 - t, cnt = m * (m + 1) / 2;
        for (int e = lane; e < cnt; e += 64) {
          int i, j;
          tri_index(e, i, j);
          const int r = jj + 1 + i, s = jj + 1 + j;
          A[r * LD + s] -= A[r * LD + jj] * A[s * LD + jj];
        }
        wave_sync_lds();
      }
    }
    __syncthreads();
    if (bad) {
      if (tid == 0) {
        if (bad == (int)kUnitRefine) atomicOr(uflags + u, kUnitRefine);
        else raise_flags(status, uflags, u, (uint32_t)bad);
      }
      return;
    }
    // 2. Panel rows r >= c + 16: L[r, c:c+16] = A[r, c:c+16] L_kk^{-T}.
    for (int r = c + 16 + tid; r < D; r += kThreads) {
      double x[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) x[t] = A[r * LD + c + t];
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        double s = x[t];
#pragma unroll
        for (int q = 0; q < t; ++q) s -= x[q] * A[(c + t) * LD + c + q];
        x[t] = s * idg[c + t];
      }
#pragma unroll
      for (int t = 0; t < 16; ++t) A[r * LD + c + t] = x[t];
    }
    __syncthreads();
    // 3. Trailing update A[r][s] -= sum_t L[r][c+t] L[s][c+t], r >= s >= c + 16,
    //    in 4x4 tiles (diagonal tiles also touch their upper half, which is
    //    unused until the inverse overwrites it).
    const int m = D - c - 16;
    if (m > 0) {
      const int mt = m / 4, ntile = mt * (mt + 1) / 2;
      for (int e = tid; e < ntile; e += kThreads) {
        int ti, tj;
        tri_index(e, ti, tj);
        const int r0 = c + 16 + 4 * ti, s0 = c + 16 + 4 * tj;
        double acc[4][4] = {};
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          double a[4], b[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) a[i] = A[(r0 + i) * LD + c + t];
#pragma unroll
          for (int j = 0; j < 4; ++j) b[j] = A[(s0 + j) * LD + c + t];
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) A[(r0 + i) * LD + s0 + j] -= acc[i][j];
      }
    }
    __syncthreads();
  }

  // ---------------- Inverse X = L^{-1} (transposed into the upper triangle) --
  // 4. Diagonal blocks: lane (k, t) computes column t of X_kk by forward
  //    substitution and stores X_kk[i][t] (i > t) at A[c + t][c + i].
  if (tid < 16 * NB) {
    const int k = tid >> 4, t = tid & 15, c = 16 * k;
    double x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      double s = 0.0;
#pragma unroll
      for (int q = 0; q < i; ++q) s += A[(c + i) * LD + c + q] * x[q];
      x[i] = i < t ? 0.0 : (i == t ? idg[c + i] : -idg[c + i] * s);
    }
#pragma unroll
    for (int i = 1; i < 16; ++i)
      if (i > t) A[(c + t) * LD + c + i] = x[i];
  }
  __syncthreads();
  // 5. Off-diagonal blocks, diagonal sd = i - j = 1 .. NB-1.
  //    X_kj[m][b] for k > j, or k == j and m > b, sits at A[16j + b][16k + m].
  for (int sd = 1; sd < NB; ++sd) {
    const int nblk = NB - sd;
    // T_j = sum_{k=j}^{j+sd-1} L_{j+sd,k} X_kj, written into X_{j+sd,j}'s slot;
    // 4x4 output tiles (a0..a0+3, b0..b0+3), 16 tiles per block.
    for (int e = tid; e < nblk * 16; e += kThreads) {
      const int j = e >> 4, a0 = 4 * ((e >> 2) & 3), b0 = 4 * (e & 3);
      const int i = j + sd;
      double acc[4][4] = {};
      for (int k = j; k < i; ++k) {
        for (int m = 0; m < 16; ++m) {
          double l[4], x[4];
#pragma unroll
          for (int p = 0; p < 4; ++p) l[p] = A[(16 * i + a0 + p) * LD + 16 * k + m];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int bb = b0 + q;
            double xv;
            if (k > j) xv = A[(16 * j + bb) * LD + 16 * k + m];
            else xv = m > bb ? A[(16 * j + bb) * LD + 16 * j + m] : (m == bb ? idg[16 * j + m] : 0.0);
            x[q] = xv;
          }
#pragma unroll
          for (int p = 0; p < 4; ++p)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[p][q] += l[p] * x[q];
        }
      }
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) A[(16 * j + b0 + q) * LD + 16 * i + a0 + p] = acc[p][q];
    }
    __syncthreads();
    // X_{i,j} = -X_ii T_j, one column b per thread (in place: the column of T
    // is read into registers first).
    for (int e = tid; e < nblk * 16; e += kThreads) {
      const int j = e >> 4, b = e & 15, i = j + sd;
      double tcol[16];
#pragma unroll
      for (int m = 0; m < 16; ++m) tcol[m] = A[(16 * j + b) * LD + 16 * i + m];
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        double s = idg[16 * i + a] * tcol[a];
#pragma unroll
        for (int m = 0; m < a; ++m) s += A[(16 * i + m) * LD + 16 * i + a] * tcol[m];
        A[(16 * j + b) * LD + 16 * i + a] = -s;
      }
    }
    __syncthreads();
  }

  // L^{-1}[r][c] for r >= c.
  auto xinv = [&](int r, int c) -> double { return r == c ? idg[r] : A[c * LD + r]; };

  // 1 / lambda_min(A) = ||L^{-1}||_2^2 by power iteration on L^{-T} L^{-1}.
  if (may_refine) {
    if (tid < D) px[tid] = 1.0 + 0.01 * tid;
    __syncthreads();
    normalize<D>(px, px, pred);
    double inv_min = 0.0;
    for (int it = 0; it < kPowerIters; ++it) {
      double s = 0.0;  // py = X px
      for (int b = ppart; b <= prow; b += TPR) s += xinv(prow, b) * px[b];
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o);
      if (ppart == 0) py[prow] = s;
      __syncthreads();
      double t2 = 0.0;  // X^T py
      for (int b = prow + ppart; b < D; b += TPR) t2 += xinv(b, prow) * py[b];
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) t2 += __shfl_xor(t2, o);
      __syncthreads();
      if (ppart == 0) py[prow] = t2;
      __syncthreads();
      inv_min = normalize<D>(px, py, pred);
    }
    if (lam_max * inv_min > kRefineCond) {
      if (tid == 0) atomicOr(uflags + u, kUnitRefine);
      return;  // pass 1 writes this unit's L^{-1}
    }
  }

  // Store L^{-1}.
  if constexpr (!FRAGS) {
    double* o64 = linv64 + (int64_t)u * D * D;
    for (int e = tid; e < D * D; e += kThreads) {
      const int a = e / D, b = e % D;
      o64[e] = (b <= a) ? xinv(a, b) : 0.0;
    }
  } else {
    // B fragment of output block j (a = 16 j + ch) and K block kb
    // (b = 32 kb + 8 kg + q): lane (ch, kg) holds 8 bf16; hi then lo.
    constexpr int NLP = (NB / 2) * (NB / 2 + 1);  // lower (j, kb) pairs: sum_j (j/2 + 1)
    uint16_t* out = lfrag + (int64_t)u * NLP * 2 * 64 * 8;
    for (int e = tid; e < NLP * 64; e += kThreads) {
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
        const float x = (b <= a) ? (float)xinv(a, b) : 0.0f;
        const __bf16 h = (__bf16)x;
        const __bf16 l = (__bf16)(x - (float)h);
        hi[t] = __builtin_bit_cast(uint16_t, h);
        lo[t] = __builtin_bit_cast(uint16_t, l);
      }
      uint16_t* dh = out + ((int64_t)(qp * 2 + 0) * 64 + ln) * 8;
      uint16_t* dl = out + ((int64_t)(qp * 2 + 1) * 64 + ln) * 8;
#pragma unroll
      for (int t = 0; t < 8; ++t) { dh[t] = hi[t]; dl[t] = lo[t]; }
    }
  }
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
