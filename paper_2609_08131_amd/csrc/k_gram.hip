// Weighted Gram M = sum_i w_i v_i v_i^T over a unit's tokens (the data term of
// the capacity matrix, Eq. 9), as per-chunk partial sums that the factor
// kernel adds in a fixed order.
//
// bf16 inputs: MFMA 16x16x32 bf16 with fp32 accumulation. The reduction runs
// over tokens, so both operands need 8 consecutive tokens of one channel per
// lane: each wave stages 32 tokens of V transposed ([channel][token]) in LDS.
// V is exact in bf16; the weighted operand x = w v (fp32) is split into three
// bf16 terms x1 + x2 + x3 (24 significant bits, like fp32), so
// M = V^T X1 + V^T X2 + V^T X3 matches an fp32 Gram: the capacity matrix of a
// short or ridge-0 unit can have cond(A) ~ 1e5-1e6, and a two-term split
// (2^-17) then costs more than the 1e-3 score tolerance. Only the
// upper-triangular 16x16 blocks are formed.
//
// fp32 inputs: fp64 VALU accumulation (8x8 or 4x4 register tiles per thread).
#include "jacap_internal.hpp"

namespace jacap {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Per-wave barrier for LDS traffic that stays inside one wave.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Index of the upper-triangular block pair (i <= j) among NB x NB blocks.
__host__ __device__ constexpr int pair_index(int i, int j, int NB) {
  return i * NB - (i * (i - 1)) / 2 + (j - i);
}

template <int D>
__global__ __launch_bounds__(kThreads) void gram_mfma_kernel(
    Geo g, const uint16_t* __restrict__ v, const float* __restrict__ zbuf,
    const float* __restrict__ kbuf, const float* __restrict__ m_u, const double* __restrict__ z_u,
    float* __restrict__ partials, int gchunks, double inv_d) {
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  constexpr int TSTEP = 32;                 // tokens per wave step (MFMA K)
  constexpr int PITCH = TSTEP + 8;          // padded LDS row (u16 elements)
  constexpr int LOADS = TSTEP * D / 8 / 64; // 16-byte loads per lane per step
  const int u = blockIdx.y, chunk = blockIdx.x;
  const Unit un = decode_unit(g, u);
  const int base = chunk * kGChunkMfma;
  if (base >= un.n) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ch = lane & 15, kg = lane >> 4;

  __shared__ __attribute__((aligned(16))) uint16_t vt[kThreads / 64][D][PITCH];
  __shared__ float wsh[kThreads / 64][TSTEP];

  const float m = m_u[u];
  const double Z = z_u[u];
  const uint16_t* vb = v + un.l * g.vsl + un.h * g.vsh;
  const int64_t trow = token_row(g, un);
  const int end = min(un.n, base + kGChunkMfma);

  floatx4 acc[NPAIR];
#pragma unroll
  for (int p = 0; p < NPAIR; ++p) acc[p] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int t0 = base + wave * TSTEP; t0 < end; t0 += TSTEP * (kThreads / 64)) {
    // Stage 32 tokens x D channels, transposed, into this wave's LDS tile.
#pragma unroll
    for (int r = 0; r < LOADS; ++r) {
      const int flat = r * 64 + lane;
      const int tok = flat / (D / 8), oct = flat % (D / 8);
      uint4 raw = make_uint4(0u, 0u, 0u, 0u);
      if (t0 + tok < end) raw = *reinterpret_cast<const uint4*>(vb + (un.t0 + t0 + tok) * g.vst + oct * 8);
      const uint16_t* e = reinterpret_cast<const uint16_t*>(&raw);
#pragma unroll
      for (int q = 0; q < 8; ++q) vt[wave][oct * 8 + q][tok] = e[q];
    }
    if (lane < TSTEP) {
      const int t = t0 + lane;
      float wv = 0.0f;
      if (t < end) wv = (float)importance_weight(zbuf[trow + t], kbuf[trow + t], m, Z, inv_d);
      wsh[wave][lane] = wv;
    }
    wave_lds_sync();

    float wl[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) wl[q] = wsh[wave][kg * 8 + q];
    bf16x8 a[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) a[i] = *reinterpret_cast<const bf16x8*>(&vt[wave][i * 16 + ch][kg * 8]);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      bf16x8 x1, x2, x3;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float x = (float)a[j][q] * wl[q];
        const __bf16 h1 = (__bf16)x;
        const float r1 = x - (float)h1;
        const __bf16 h2 = (__bf16)r1;
        x1[q] = h1;
        x2[q] = h2;
        x3[q] = (__bf16)(r1 - (float)h2);
      }
#pragma unroll
      for (int i = 0; i <= j; ++i) {
        const int p = pair_index(i, j, NB);
        acc[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], x3, acc[p], 0, 0, 0);
        acc[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], x2, acc[p], 0, 0, 0);
        acc[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], x1, acc[p], 0, 0, 0);
      }
    }
    wave_lds_sync();
  }
  // Partial of this wave: block p, lane, element r -> M[16 i + 4 kg + r][16 j + ch].
  float* out = partials + (((int64_t)u * gchunks + chunk) * kMfmaGramParts + wave) * (NPAIR * 256);
#pragma unroll
  for (int p = 0; p < NPAIR; ++p) *reinterpret_cast<floatx4*>(out + p * 256 + lane * 4) = acc[p];
}

// fp64 Gram for fp32 inputs: thread (ty, tx) of a 16 x 16 grid owns a
// (D/16) x (D/16) register tile of M; V is staged 32 tokens at a time.
template <int D>
__global__ __launch_bounds__(kThreads) void gram_precise_kernel(
    Geo g, const float* __restrict__ v, const float* __restrict__ zbuf,
    const float* __restrict__ kbuf, const float* __restrict__ m_u, const double* __restrict__ z_u,
    double* __restrict__ partials, int gchunks, double inv_d) {
  constexpr int R = D / 16;
  const int u = blockIdx.y, chunk = blockIdx.x;
  const Unit un = decode_unit(g, u);
  const int base = chunk * kGChunkPrecise;
  if (base >= un.n) return;
  const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
  __shared__ float vs[32][D];
  __shared__ double ws[32];
  const float m = m_u[u];
  const double Z = z_u[u];
  const float* vb = v + un.l * g.vsl + un.h * g.vsh;
  const int64_t trow = token_row(g, un);
  const int end = min(un.n, base + kGChunkPrecise);
  double acc[R][R];
#pragma unroll
  for (int a = 0; a < R; ++a)
#pragma unroll
    for (int b = 0; b < R; ++b) acc[a][b] = 0.0;
  for (int t0 = base; t0 < end; t0 += 32) {
    __syncthreads();
    for (int e = tid; e < 32 * D; e += kThreads) {
      const int tok = e / D, c = e % D;
      vs[tok][c] = (t0 + tok < end) ? vb[(un.t0 + t0 + tok) * g.vst + c] : 0.0f;
    }
    if (tid < 32) {
      const int t = t0 + tid;
      ws[tid] = (t < end) ? importance_weight(zbuf[trow + t], kbuf[trow + t], m, Z, inv_d) : 0.0;
    }
    __syncthreads();
    for (int tok = 0; tok < 32; ++tok) {
      const double w = ws[tok];
      double xa[R], vb2[R];
#pragma unroll
      for (int a = 0; a < R; ++a) xa[a] = w * (double)vs[tok][ty * R + a];
#pragma unroll
      for (int b = 0; b < R; ++b) vb2[b] = (double)vs[tok][tx * R + b];
#pragma unroll
      for (int a = 0; a < R; ++a)
#pragma unroll
        for (int b = 0; b < R; ++b) acc[a][b] += xa[a] * vb2[b];
    }
  }
  double* out = partials + ((int64_t)u * gchunks + chunk) * D * D;
#pragma unroll
  for (int a = 0; a < R; ++a)
#pragma unroll
    for (int b = 0; b < R; ++b) out[(ty * R + a) * D + tx * R + b] = acc[a][b];
}

hipError_t launch_gram(const Launch& L, const void* v) {
  const Geo& g = L.geo;
  const dim3 grid(L.ws.gchunks, g.U);
  const double inv_d = 1.0 / (double)g.D;
  const float* zb = ws_ptr<float>(L.wsp, L.ws.z);
  const float* kb = ws_ptr<float>(L.wsp, L.ws.kappa);
  const float* mu = ws_ptr<float>(L.wsp, L.ws.smax_m);
  const double* zu = ws_ptr<double>(L.wsp, L.ws.smax_z);
  if (L.ws.mfma) {
    float* part = ws_ptr<float>(L.wsp, L.ws.gram);
    if (g.D == 128)
      gram_mfma_kernel<128><<<grid, kThreads, 0, L.stream>>>(g, (const uint16_t*)v, zb, kb, mu, zu, part, L.ws.gchunks, inv_d);
    else
      gram_mfma_kernel<64><<<grid, kThreads, 0, L.stream>>>(g, (const uint16_t*)v, zb, kb, mu, zu, part, L.ws.gchunks, inv_d);
  } else {
    double* part = ws_ptr<double>(L.wsp, L.ws.gram);
    if (g.D == 128)
      gram_precise_kernel<128><<<grid, kThreads, 0, L.stream>>>(g, (const float*)v, zb, kb, mu, zu, part, L.ws.gchunks, inv_d);
    else
      gram_precise_kernel<64><<<grid, kThreads, 0, L.stream>>>(g, (const float*)v, zb, kb, mu, zu, part, L.ws.gchunks, inv_d);
  }
  return hipGetLastError();
}

}  // namespace jacap
