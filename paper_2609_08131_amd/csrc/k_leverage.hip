// Leverage score of Eq. 10: score_i = w_i v_i^T A^{-1} v_i = w_i ||L^{-1} v_i||^2.
//
// bf16 inputs: Y = V L^{-T} on MFMA 16x16x32 bf16. The token dimension is the
// MFMA row dimension. V rows are read whole (each wave load covers complete
// 128-byte lines, streamed non-temporally, or cached for per-head GQA) and pass through a small
// wave-private LDS tile into the operand layout. L^{-1} is split into bf16
// hi + lo and kept in registers; only the K-blocks with b <= a of the lower
// triangle are multiplied. The squared row norm is reduced across the 16
// lanes that share a token.
//
// fp64 pass (every unit of fp32 inputs; the units of bf16 inputs that the
// factorisation sent to the fp64 path): fp64 VALU, L^{-1} in LDS, 8 threads
// per token.
#include <algorithm>

#include "jacap_internal.hpp"

namespace jacap {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// POL: cache policy of the V loads (streamed, or kept in L2 for the other
// query-head units of the same KV head).
template <int D, int POL>
__global__ __launch_bounds__(kThreads, 2) void leverage_mfma_kernel(
    Geo g, const uint16_t* __restrict__ v, const float* __restrict__ wbuf,
    const uint16_t* __restrict__ lfrag, const uint32_t* __restrict__ uflags,
    float* __restrict__ scores, int lchunks, int lchunk) {
  constexpr int NB = D / 16;                    // output blocks of 16 channels (a)
  constexpr int NK = D / 32;                    // K blocks of 32 channels (b)
  constexpr int NLP = (NB / 2) * (NB / 2 + 1);  // lower (j, kb) block pairs
  int u, chunk;
  if (!grid_unit_chunk<true>(g, lchunks, u, chunk)) return;
  const Unit un = decode_unit(g, u);
  const int base = chunk * lchunk;
  if (base >= un.n) return;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ch = lane & 15, kg = lane >> 4;
  const int rl = 2 * (ch >> 3) + ((ch >> 2) & 1);  // token (of 4) whose score this lane ends with
  const int64_t trow = token_row(g, un);
  const int end = min(un.n, base + lchunk);

  const uint32_t uf = uflags[u];
  if (uf & kUnitRefine) return;  // scored by the fp64 pass
  if (uf & kUnitFailed) {  // unit failed (non-finite input): NaN scores
    for (int t = base + threadIdx.x; t < end; t += kThreads) scores[trow + t] = __builtin_nanf("");
    return;
  }

  // B fragments, pre-split by the factor kernel in lane order.
  bf16x8 bh[NLP], bl[NLP];
  const uint16_t* lf = lfrag + (int64_t)u * NLP * 2 * 64 * 8;
#pragma unroll
  for (int q = 0; q < NLP; ++q) {
    bh[q] = *reinterpret_cast<const bf16x8*>(lf + ((int64_t)(q * 2 + 0) * 64 + lane) * 8);
    bl[q] = *reinterpret_cast<const bf16x8*>(lf + ((int64_t)(q * 2 + 1) * 64 + lane) * 8);
  }
  drain_vmem();

  const uint16_t* vb = v + un.l * g.vsl + un.h * g.vsh + un.t0 * g.vst;

  // A step is 16 tokens (one MFMA row tile). V rows are prefetched two
  // steps ahead into three rotating register buffers (the loop is unrolled
  // by three so the buffers stay in fixed registers). A step's 16 rows are
  // read whole: each wave load brings RPL consecutive rows (d / 8 lanes per
  // row, 1 KB of contiguous lines, cache policy), through a buffer range
  // that ends at the chunk's last row (rows past it load as zeros and are not
  // stored), so every load is unconditional with a fixed per-lane offset and
  // the compiler's wait counts stay static. The rows then pass through a
  // wave-private LDS tile into the MFMA operand layout (lane (ch, kg) of
  // K-block kb: row ch, channels 32 kb + 8 kg .. + 7). MFMAs are issued
  // kb-outer so that consecutive MFMAs update different output blocks.
  // One prefetched step: the lane's V row pieces and the weight of the token
  // whose score this lane writes.
  struct Buf { uint4 a[NK]; float w; };
  // bytes per tile row: a 32-byte pad leaves the operand reads free of bank
  // conflicts, measured (16 bytes: 25 %)
  constexpr int PITCH = D * 2 + 32;
  __shared__ __attribute__((aligned(16))) char tiles[kThreads / 64][16 * PITCH];
  char* tile = tiles[wave];
  const int32_t vstb = (int32_t)g.vst * 2;
  constexpr int LPR = D / 8;                    // lanes per whole row (16 bytes each)
  constexpr int RPL = 64 / LPR;                 // rows per wave load
  static_assert(RPL * NK == 16, "a step's 16 rows in NK whole-row loads");
  const int rrow = lane / LPR, rpc = lane % LPR;  // row (of RPL) and 16-byte piece of a load
  int32_t voff[NK];
#pragma unroll
  for (int i = 0; i < NK; ++i) voff[i] = (RPL * i + rrow) * vstb + rpc * 16;
  const int32_t woff = (4 * kg + rl) * 4;
  const float* wb = wbuf + trow;
  auto load = [&](int t0, Buf& b) {
    const int32_t rows = min(end - t0, 16);
    const auto vr = buffer_range(vb + (int64_t)t0 * g.vst, rows_bytes(rows, vstb, D * 2));
#pragma unroll
    for (int i = 0; i < NK; ++i) b.a[i] = buffer_load16<POL>(vr, voff[i]);
    b.w = buffer_load_f32(buffer_range(wb + t0, max(rows, 0) * 4), woff);
    __builtin_amdgcn_sched_barrier(0);  // issue here, ahead of the MFMAs that follow
  };
  auto step = [&](int t0, const Buf& b) {
    const int tw = t0 + 4 * kg + rl;
    const float wt = b.w;
#pragma unroll
    for (int i = 0; i < NK; ++i)
      *reinterpret_cast<uint4*>(tile + (RPL * i + rrow) * PITCH + rpc * 16) = b.a[i];
    bf16x8 cur[NK];
#pragma unroll
    for (int kb = 0; kb < NK; ++kb)
      cur[kb] = *reinterpret_cast<const bf16x8*>(tile + ch * PITCH + kb * 64 + kg * 16);
    // Output blocks j = 2 jp and 2 jp + 1 share the K-block range kb <= jp:
    // their two accumulation chains are interleaved.
    float ss[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jp = 0; jp < NB / 2; ++jp) {
      floatx4 y0 = {0.f, 0.f, 0.f, 0.f}, y1 = {0.f, 0.f, 0.f, 0.f};
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
    // ss[r] is this lane's channel's part of token 4 kg + r; sum over the 16
    // lanes (channels) of the row by a transposing reduction: the row mirror
    // (ch <-> 15 - ch) leaves tokens 0, 1 to the lower half and 2, 3 to the
    // upper, the half-row mirror (ch <-> 7 - ch) one token per lane, and two
    // quad swaps finish; lane ch then holds token rl.
    const bool hi8 = ch >= 8, hi4 = (ch & 4) != 0;
    const float m0 = (hi8 ? ss[2] : ss[0]) + dpp_f32<kDppMirror>(hi8 ? ss[0] : ss[2]);
    const float m1 = (hi8 ? ss[3] : ss[1]) + dpp_f32<kDppMirror>(hi8 ? ss[1] : ss[3]);
    float sv = (hi4 ? m1 : m0) + dpp_f32<kDppHalfMirror>(hi4 ? m0 : m1);
    sv += dpp_f32<kDppQuadXor1>(sv);
    sv += dpp_f32<kDppQuadXor2>(sv);
    if ((ch & 3) == 0 && tw < end) scores[trow + tw] = wt * sv;
  };
  constexpr int WSTRIDE = 16 * (kThreads / 64);
  const int t_first = base + wave * 16;
  if (t_first >= end) return;
  Buf b0, b1, b2;
  load(t_first, b0);
  load(t_first + WSTRIDE, b1);
  for (int t0 = t_first; t0 < end; t0 += 3 * WSTRIDE) {
    load(t0 + 2 * WSTRIDE, b2);
    step(t0, b0);
    if (t0 + WSTRIDE >= end) break;
    load(t0 + 3 * WSTRIDE, b0);
    step(t0 + WSTRIDE, b1);
    if (t0 + 2 * WSTRIDE >= end) break;
    load(t0 + 4 * WSTRIDE, b1);
    step(t0 + 2 * WSTRIDE, b2);
  }
}

// fp64 leverage: every unit (fp32 inputs), or only the units marked
// kUnitRefine (REFINE_ONLY, bf16 inputs). L^{-1} comes from the reduced-Gram
// buffer in the lower-block layout written by the fp64 factorisation.
template <typename T, int D, bool REFINE_ONLY>
__global__ __launch_bounds__(kThreads) void leverage_precise_kernel(
    Geo g, const T* __restrict__ v, const float* __restrict__ wbuf,
    const double* __restrict__ xred, const uint32_t* __restrict__ uflags,
    float* __restrict__ scores, int lchunks, int lchunk, int items) {
  constexpr int LD = D + 1;
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  constexpr int TPT = 8;                 // threads per token
  constexpr int TOK = kThreads / TPT;    // tokens per tile
  __shared__ double X[D * LD];
  __shared__ float vs[TOK][D + 1];  // padded: the wave's 8 token rows in distinct banks
  if constexpr (REFINE_ONLY) {
    // The flags of all the walk's items at once (a load per thread, not one
    // per item in turn): a workgroup with no marked unit ends here.
    bool any = false;
    for (int item = blockIdx.x + threadIdx.x * gridDim.x; item < items;
         item += gridDim.x * kThreads) {
      int u, chunk;
      any |= grid_unit_chunk_at<true>(g, lchunks, item, u, chunk) && (uflags[u] & kUnitRefine);
    }
    if (!__syncthreads_or(any)) return;
  }
  // one (unit, chunk) item per workgroup, or (REFINE_ONLY) a grid-stride walk
  for (int item = blockIdx.x; item < items; item += gridDim.x) {
  int u, chunk;
  if (!grid_unit_chunk_at<true>(g, lchunks, item, u, chunk)) continue;
  const uint32_t uf = uflags[u];
  if (REFINE_ONLY && !(uf & kUnitRefine)) continue;
  const Unit un = decode_unit(g, u);
  const int base = chunk * lchunk;
  if (base >= un.n) continue;
  const int tid = threadIdx.x;
  const int64_t trow = token_row(g, un);
  const int end = min(un.n, base + lchunk);
  if (uf & kUnitFailed) {  // non-finite input or singular A: NaN scores
    for (int t = base + tid; t < end; t += kThreads) scores[trow + t] = __builtin_nanf("");
    continue;
  }
  __syncthreads();  // the previous item's X and staged tokens are no longer read
  // lower blocks of L^{-1}: pair p = (bi <= bj) holds X[16 bj + r][16 bi + c]
  const double* Xb = xred + (int64_t)u * (NPAIR * 256);
  for (int e = tid; e < NPAIR * 256; e += kThreads) {
    int p = e >> 8, bi = 0;
#pragma unroll
    for (int q = 0; q < NB; ++q)
      if (p >= NB - bi) { p -= NB - bi; ++bi; }
    const int bj = bi + p;
    X[(16 * bj + ((e >> 4) & 15)) * LD + 16 * bi + (e & 15)] = Xb[e];
  }
  const T* vb = v + un.l * g.vsl + un.h * g.vsh;
  const int my_tok = tid / TPT, sub = tid % TPT;
  for (int t0 = base; t0 < end; t0 += TOK) {
    __syncthreads();
    for (int e = tid; e < TOK * D; e += kThreads) {
      const int tk = e / D, c = e % D;
      vs[tk][c] = (t0 + tk < end) ? to_f32(vb[(un.t0 + t0 + tk) * g.vst + c]) : 0.0f;
    }
    __syncthreads();
    double ss = 0.0;
    for (int a = sub; a < D; a += TPT) {
      // four independent chains over b (latency, not order, bounds this loop)
      double y4[4] = {0.0, 0.0, 0.0, 0.0};
      int b = 0;
      for (; b + 3 <= a; b += 4) {
#pragma unroll
        for (int q = 0; q < 4; ++q) y4[q] = fma(X[a * LD + b + q], (double)vs[my_tok][b + q], y4[q]);
      }
      for (; b <= a; ++b) y4[0] = fma(X[a * LD + b], (double)vs[my_tok][b], y4[0]);
      const double y = (y4[0] + y4[1]) + (y4[2] + y4[3]);
      ss += y * y;
    }
#pragma unroll
    for (int o = 1; o < TPT; o <<= 1) ss += __shfl_xor(ss, o);
    const int t = t0 + my_tok;
    if (sub == 0 && t < end) {
      scores[trow + t] = (float)((double)wbuf[trow + t] * ss);
    }
  }
  }
}

hipError_t launch_leverage(const Launch& L, const void* v, float* scores) {
  const Geo& g = L.geo;
  const dim3 grid((unsigned)chunked_grid(g, L.ws.lchunks));
  const float* wb = ws_ptr<float>(L.wsp, L.ws.wgt);
  const uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  if (L.ws.mfma) {
    const uint16_t* lf = ws_ptr<uint16_t>(L.wsp, L.ws.lfrag);
    auto go = [&](auto kern) {
      kern<<<grid, kThreads, 0, L.stream>>>(g, (const uint16_t*)v, wb, lf, uf, scores, L.ws.lchunks,
                                            L.ws.lchunk);
    };
    if (g.D == 128) {
      if (g.V > 1) go(leverage_mfma_kernel<128, kPolicyShared>);
      else go(leverage_mfma_kernel<128, kPolicyStream>);
    } else {
      if (g.V > 1) go(leverage_mfma_kernel<64, kPolicyShared>);
      else go(leverage_mfma_kernel<64, kPolicyStream>);
    }
  } else {
    return launch_leverage_precise(L, v, scores);
  }
  return hipGetLastError();
}

// fp64 leverage: every unit of fp32 inputs, or the marked units of bf16 inputs.
hipError_t launch_leverage_precise(const Launch& L, const void* v, float* scores) {
  const Geo& g = L.geo;
  const int64_t items = chunked_grid(g, L.ws.plchunks);
  const dim3 grid((unsigned)(L.ws.mfma ? std::min<int64_t>(items, kRefineBlocks) : items));
  const float* wb = ws_ptr<float>(L.wsp, L.ws.wgt);
  const uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  const double* xr = ws_ptr<double>(L.wsp, L.ws.gram_red);
  auto go = [&](auto kern, auto vv) {
    kern<<<grid, kThreads, 0, L.stream>>>(g, vv, wb, xr, uf, scores, L.ws.plchunks, L.ws.plchunk,
                                          (int)items);
  };
  if (L.ws.mfma) {
    if (g.D == 128) go(leverage_precise_kernel<uint16_t, 128, true>, (const uint16_t*)v);
    else go(leverage_precise_kernel<uint16_t, 64, true>, (const uint16_t*)v);
  } else {
    if (g.D == 128) go(leverage_precise_kernel<float, 128, false>, (const float*)v);
    else go(leverage_precise_kernel<float, 64, false>, (const float*)v);
  }
  return hipGetLastError();
}

}  // namespace jacap
