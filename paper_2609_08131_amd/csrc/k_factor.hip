// Capacity matrix A = ridge I + M (Eq. 9), its Cholesky factor A = L L^T and
// the triangular inverse L^{-1}, one workgroup per unit, in fp64 in LDS.
// ||L^{-1} v||^2 = v^T A^{-1} v is what the leverage score of Eq. 10 needs.
#include "jacap_internal.hpp"

namespace jacap {

__host__ __device__ constexpr int pair_index_f(int i, int j, int NB) {
  return i * NB - (i * (i - 1)) / 2 + (j - i);
}

// PF = 0: partials are fp64 D x D (one per chunk, precise path).
// PF = 1: partials are fp32 upper 16x16 blocks in MFMA lane order, kMfmaGramParts per chunk.
template <int D, int PF>
__global__ __launch_bounds__(kThreads) void factor_kernel(Geo g, const void* __restrict__ partials,
                                                          int gchunks, int gchunk, double ridge,
                                                          double piv_rel,
                                                          double* __restrict__ linv64,
                                                          float* __restrict__ linv32,
                                                          uint32_t* status, uint32_t* uflags) {
  constexpr int LD = D + 1;
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  const int u = blockIdx.x, tid = threadIdx.x;
  const Unit un = decode_unit(g, u);
  if (un.n == 0) return;
  const int nch = (un.n + gchunk - 1) / gchunk;

  __shared__ double A[D * LD];
  __shared__ double dg[D];
  __shared__ double tmp[D];
  __shared__ int bad;

  // 1. A (lower triangle incl. diagonal) = ridge I + sum of partials, fixed order.
  if constexpr (PF == 0) {
    const double* P = reinterpret_cast<const double*>(partials) + (int64_t)u * gchunks * D * D;
    for (int e = tid; e < D * D; e += kThreads) {
      const int a = e / D, b = e % D;
      if (b > a) continue;
      // upper-triangle entry (b, a) is used for both halves
      double s = 0.0;
      for (int c = 0; c < nch; ++c) s += P[(int64_t)c * D * D + b * D + a];
      A[a * LD + b] = s;
    }
  } else {
    const float* P = reinterpret_cast<const float*>(partials) +
                     (int64_t)u * gchunks * kMfmaGramParts * (NPAIR * 256);
    for (int e = tid; e < NPAIR * 256; e += kThreads) {
      // decode pair p, lane, r -> (row, col) of the upper block (i <= j)
      const int p = e / 256, rem = e % 256, lane = rem / 4, r = rem % 4;
      int i = 0, j = 0;
      {
        int q = p;
        for (int ii = 0; ii < NB; ++ii) {
          const int cnt = NB - ii;
          if (q < cnt) { i = ii; j = ii + q; break; }
          q -= cnt;
        }
      }
      const int row = i * 16 + (lane >> 4) * 4 + r;  // index into the first operand (channel a)
      const int col = j * 16 + (lane & 15);          // channel b
      if (i == j && row > col) continue;             // diagonal block: keep the upper half
      double s = 0.0;
      for (int c = 0; c < nch * kMfmaGramParts; ++c) s += (double)P[(int64_t)c * (NPAIR * 256) + e];
      A[col * LD + row] = s;  // lower-triangle slot (col >= row)
    }
  }
  __syncthreads();
  if (tid == 0) bad = 0;
  for (int a = tid; a < D; a += kThreads) {
    A[a * LD + a] += ridge;
    dg[a] = A[a * LD + a];
    if (!isfinite(dg[a])) atomicOr(&bad, 2);
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) raise_flags(status, uflags, u, kUnitNonfinite);
    return;
  }

  // 2. Right-looking Cholesky, A <- L (lower).
  const int ty = tid / 16, tx = tid % 16;
  for (int j = 0; j < D; ++j) {
    const double piv = A[j * LD + j];
    // A pivot that has lost all but piv_rel of its diagonal entry is within the
    // rounding noise of the accumulated Gram: A is numerically singular at the
    // path's working precision (rank-deficient M with ridge 0).
    if (!(piv > piv_rel * dg[j]) || !(piv > 0.0)) {
      if (tid == 0) raise_flags(status, uflags, u, isfinite(piv) ? kUnitSingular : kUnitNonfinite);
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
  for (int j = D - 1; j >= 0; --j) {
    const double ajj = 1.0 / A[j * LD + j];
    for (int i = j + 1 + tid; i < D; i += kThreads) tmp[i] = A[i * LD + j];
    __syncthreads();
    for (int i = j + 1 + tid; i < D; i += kThreads) {
      double s = 0.0;
      for (int kk = j + 1; kk <= i; ++kk) s += A[i * LD + kk] * tmp[kk];
      A[i * LD + j] = -ajj * s;
    }
    __syncthreads();
    if (tid == 0) A[j * LD + j] = ajj;
    __syncthreads();
  }

  // 4. Store L^{-1} (zeros above the diagonal) in fp64 and fp32.
  double* o64 = linv64 + (int64_t)u * D * D;
  float* o32 = linv32 + (int64_t)u * D * D;
  for (int e = tid; e < D * D; e += kThreads) {
    const int a = e / D, b = e % D;
    const double x = (b <= a) ? A[a * LD + b] : 0.0;
    o64[e] = x;
    o32[e] = (float)x;
  }
}

hipError_t launch_factor(const Launch& L) {
  const Geo& g = L.geo;
  const void* part = L.wsp + L.ws.gram;
  double* l64 = ws_ptr<double>(L.wsp, L.ws.linv64);
  float* l32 = ws_ptr<float>(L.wsp, L.ws.linv32);
  uint32_t* st = ws_ptr<uint32_t>(L.wsp, L.ws.status);
  uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  const double ridge = (double)L.cfg->ridge;
  // fp32-accumulated Gram (bf16 path) carries ~1e-5 relative noise; the fp64
  // path ~1e-15.
  const double piv_rel = L.ws.mfma ? 1e-4 : 1e-12;
  if (L.ws.mfma) {
    if (g.D == 128)
      factor_kernel<128, 1><<<g.U, kThreads, 0, L.stream>>>(g, part, L.ws.gchunks, L.ws.gchunk, ridge, piv_rel, l64, l32, st, uf);
    else
      factor_kernel<64, 1><<<g.U, kThreads, 0, L.stream>>>(g, part, L.ws.gchunks, L.ws.gchunk, ridge, piv_rel, l64, l32, st, uf);
  } else {
    if (g.D == 128)
      factor_kernel<128, 0><<<g.U, kThreads, 0, L.stream>>>(g, part, L.ws.gchunks, L.ws.gchunk, ridge, piv_rel, l64, l32, st, uf);
    else
      factor_kernel<64, 0><<<g.U, kThreads, 0, L.stream>>>(g, part, L.ws.gchunks, L.ws.gchunk, ridge, piv_rel, l64, l32, st, uf);
  }
  return hipGetLastError();
}

}  // namespace jacap
