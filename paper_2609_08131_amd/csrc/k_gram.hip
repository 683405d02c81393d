// Weighted Gram M = sum_i w_i v_i v_i^T over a unit's tokens (the data term of
// the capacity matrix, Eq. 9), as one partial per workgroup (a chunk of
// tokens), added in a fixed order by the factorisation itself or, for units
// of many chunks, by the reduce kernel below.
//
// Partial layout ("block-lane"): the upper-triangular 16x16 blocks (i <= j) of
// M, block pair p = pair_index(i, j), 256 entries per block in MFMA 16x16
// output order: entry p*256 + lane*4 + r holds M[16i + 4(lane/16) + r][16j + lane%16].
//
// bf16 inputs: MFMA 16x16x32 bf16 with fp32 accumulation; the contraction runs
// over tokens. V is exact in bf16; the weighted operand x = w v (fp32) is split
// into two bf16 terms rounded to nearest (x = x1 + x2 to 2^-17 relative), so
// M = V^T X1 + V^T X2. The factor kernel then marks the units whose capacity
// matrix is ill-conditioned enough for the fp32 rounding to show in the
// scores, and a second pass recomputes only those in fp64.
//
// fp64 pass (every unit of fp32 inputs; the marked units of bf16 inputs): fp64
// VALU accumulation of exact products (register tiles), same partial layout.
#include <type_traits>

#include <algorithm>

#include "jacap_internal.hpp"

namespace jacap {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));

// Transposing 64-bit LDS read (gfx950): inside each group of 16 lanes, lane i
// receives element i % 4 of the 4 x 16-bit values addressed by lanes
// i / 4, 4 + i / 4, 8 + i / 4 and 12 + i / 4 of its group, in that order.
__device__ __forceinline__ s16x4 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(p));
}

// The workgroup walks its chunk in steps of 32 tokens. Each step is read with
// 16-byte buffer loads (non-temporal, or cached when the query-head units of
// a KV head share them; each wave load covers whole 128-byte
// lines), prefetched two steps ahead, and staged in LDS token-major
// (double-buffered, one barrier per step); the four waves share it. The upper 16x16 block pairs (i <= j) are split between the waves by
// column pairs {w, NB-1-w}, which gives every wave the same number of pairs
// (9 at d = 128), so no cross-wave reduction is needed.
//
// Token <-> MFMA K-slot mapping: lane (ch, kg) slot q holds token 8 kg + q of
// the step, for both operands. The operand fragment of a 16-channel block is
// read with two transposing LDS reads: lane (i, kg) addresses token
// 8 kg + i / 4 (+ 4), channels 4 (i % 4) .. + 3 of the block, and receives
// channel i of tokens 8 kg .. 8 kg + 3 (8 kg + 4 .. 8 kg + 7). With a 288-byte
// row pitch the 16 lanes of a group touch 32 distinct banks; the chunk
// swizzle of odd 8-token groups separates the groups served together.
//
// Accumulation: fp32 MFMA chains of kGramFlush steps, each added into a
// second fp32 accumulator (short rounding chains; an ill-conditioned ridge-0
// unit needs them).
constexpr int kGramStep = 32;
constexpr int kGramPitch = 144;  // u16 elements per staged token row (288 bytes)
constexpr int kGramFlush = 4;
static_assert(kGramStep * kGramFlush == kGramSpan, "flush span");

struct GramArgs {
  const uint16_t* vb;   // V of the unit, at its first token
  int64_t vst;
  const float* wrow;    // importance weights of the unit, at its first token
  int base, end, nsteps;  // nsteps: a multiple of kGramFlush
  float* out;           // this chunk's partial (block-lane layout)
};

// Whole chunk for wave W: it owns columns JA = W and JB = NB-1-W (if distinct).
template <int D, int W, int NT, int POL>
__device__ __forceinline__ void gram_wave(const GramArgs& ga, uint16_t* tiles, float* wts) {
  constexpr int NB = D / 16;
  constexpr int OCT = D / 8;                            // 16-byte pieces per token row
  constexpr int LOADS = kGramStep * OCT / kThreads;     // 16-byte loads per thread per step
  constexpr int TILE = kGramStep * kGramPitch;          // u16 per staged step
  constexpr int JA = W, JB = NB - 1 - W;
  constexpr bool HAS_A = JA < NB && JA <= JB;
  constexpr bool HAS_B = JB > JA;
  constexpr int PA = HAS_A ? JA + 1 : 0;                // pairs of column JA
  constexpr int PB = HAS_B ? JB + 1 : 0;                // pairs of column JB
  constexpr int NP = PA + PB > 0 ? PA + PB : 1;
  constexpr int NA = HAS_B ? JB + 1 : (HAS_A ? JA + 1 : 0);  // fragments needed
  constexpr int WPW = kGramStep / (kThreads / 64);      // weights loaded per wave per step
  static_assert(LOADS >= 1, "step too small");
  static_assert((WPW & (WPW - 1)) == 0, "weights per wave must be a power of two");
  const int tid = threadIdx.x, lane = tid & 63;
  const int kg = lane >> 4, il = lane & 15;
  // This lane's address inside a staged step for the transposing reads. Rows
  // of odd 8-token groups hold their 32-byte channel chunks XOR-swizzled by 4
  // (chunk c at position c ^ 4), so the two 16-lane groups that the LDS
  // serves together read disjoint banks. Chunk i < 4 sits at i + sw, chunk
  // i >= 4 at i - sw.
  const int sw = 4 * (kg & 1);
  const int tr_off = (8 * kg + (il >> 2)) * kGramPitch + 4 * (il & 3);
  const int tr_lo = tr_off + 16 * sw, tr_hi = tr_off - 16 * sw;

  floatx4 acc32[NP], acc2[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) acc2[p] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Each step reads its 32 rows through a buffer range that ends at the
  // chunk's last row: rows past it (and their weights) load as zeros, so
  // they add exactly nothing. Per-lane offsets are fixed; only the range's
  // base moves with the step (scalar arithmetic).
  struct Pre { uint4 v[LOADS]; float w; };
  int32_t voff[LOADS];
#pragma unroll
  for (int r = 0; r < LOADS; ++r) {
    const int flat = r * kThreads + tid, tok = flat / OCT, oc = flat % OCT;
    voff[r] = tok * (int32_t)ga.vst * 2 + oc * 16;
  }
  const int32_t woff = (W * WPW + (lane & (WPW - 1))) * 4;
  // Steps are loaded strictly in order (0, 1, 2, ...), so the range advances
  // by one step per call; past the chunk end it is empty.
  const uint16_t* vnext = ga.vb + (int64_t)ga.base * ga.vst;
  const float* wnext = ga.wrow + ga.base;
  int32_t left = ga.end - ga.base;  // rows of the chunk from vnext on
  const int32_t vstb = (int32_t)ga.vst * 2;
  auto gload = [&]() {
    Pre buf;
    const int32_t rows = min(left, kGramStep);
    const auto vr = buffer_range(vnext, rows_bytes(rows, vstb, D * 2));
#pragma unroll
    for (int r = 0; r < LOADS; ++r) buf.v[r] = buffer_load16<POL>(vr, voff[r]);  // whole lines
    buf.w = buffer_load_f32(buffer_range(wnext, max(rows, 0) * 4), woff);
    vnext += kGramStep * ga.vst;
    wnext += kGramStep;
    left -= kGramStep;
    return buf;
  };
  auto stage = [&](const Pre& buf, uint16_t* tile, float* wt) {
#pragma unroll
    for (int r = 0; r < LOADS; ++r) {
      const int flat = r * kThreads + tid, tok = flat / OCT, oc = flat % OCT;
      const int pc = oc ^ (8 * ((tok >> 3) & 1));  // 16-byte piece, chunk swizzle
      *reinterpret_cast<uint4*>(tile + tok * kGramPitch + pc * 8) = buf.v[r];
    }
    if (lane < WPW) wt[W * WPW + lane] = buf.w;
  };
  // Column J of the step: B operand x = w v of block J, split into NT terms,
  // against the A fragments of blocks 0..J. FIRST: the chain restarts.
  auto column = [&](auto jc, auto pbc, auto firstc, const u16x8 (&a)[NA > 0 ? NA : 1],
                    const float (&wl)[8]) {
    constexpr int J = decltype(jc)::value, PBASE = decltype(pbc)::value;
    constexpr bool FIRST = decltype(firstc)::value;
    u16x8 xt[NT];
    static_assert(NT == 2, "two bf16 terms");
    {
      // Pairwise: hi = RNE(x) for two elements with one packed convert, the
      // residual x - hi from an fma on the exact product.
#pragma unroll
      for (int q = 0; q < 8; q += 2) {
        const float v0 = bf16_to_f32(a[J][q]), v1 = bf16_to_f32(a[J][q + 1]);
        const float2v x = {v0 * wl[q], v1 * wl[q + 1]};
        const bf16x2 hi = __builtin_convertvector(x, bf16x2);
        const uint32_t hb = __builtin_bit_cast(uint32_t, hi);
        const float h0 = __uint_as_float(hb << 16), h1 = __uint_as_float(hb & 0xFFFF0000u);
        const float2v r = {fmaf(v0, wl[q], -h0), fmaf(v1, wl[q + 1], -h1)};
        const uint32_t lb = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
        xt[0][q] = (uint16_t)lb; xt[0][q + 1] = (uint16_t)(lb >> 16);
        xt[1][q] = (uint16_t)hb; xt[1][q + 1] = (uint16_t)(hb >> 16);
      }
    }
    // term-outer order, so that consecutive MFMAs write different
    // accumulators. The two-term split issues the high term first: its
    // MFMAs need only the rounded products, and the residual term's VALU
    // work runs under them.
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      const int t = NT == 2 ? 1 - tt : tt;
      const bf16x8 c = __builtin_bit_cast(bf16x8, xt[t]);
#pragma unroll
      for (int i = 0; i <= J; ++i) {
        const bf16x8 ai = __builtin_bit_cast(bf16x8, a[i]);
        if (FIRST && tt == 0)
          acc32[PBASE + i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ai, c, floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
        else
          acc32[PBASE + i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ai, c, acc32[PBASE + i], 0, 0, 0);
      }
    }
  };
  auto compute = [&](const uint16_t* tile, const float* wt, auto firstc) {
    if constexpr (NA > 0) {
      float wl[8];
      const floatx4 w0 = *reinterpret_cast<const floatx4*>(wt + 8 * kg);
      const floatx4 w1 = *reinterpret_cast<const floatx4*>(wt + 8 * kg + 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) { wl[q] = w0[q]; wl[q + 4] = w1[q]; }
      u16x8 a[NA];
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const uint16_t* tb = tile + (i < 4 ? tr_lo : tr_hi) + 16 * i;
        const s16x4 lo = lds_read_tr16(tb);
        const s16x4 hi = lds_read_tr16(tb + 4 * kGramPitch);
#pragma unroll
        for (int q = 0; q < 4; ++q) { a[i][q] = (uint16_t)lo[q]; a[i][q + 4] = (uint16_t)hi[q]; }
      }
      // Column JB (the longer MFMA run) first; the scheduling groups below
      // then issue column JA's operand split between column JB's MFMAs, so
      // the VALU work runs while the matrix core is busy.
      if constexpr (HAS_B) column(std::integral_constant<int, JB>{}, std::integral_constant<int, PA>{}, firstc, a, wl);
      if constexpr (HAS_A) column(std::integral_constant<int, JA>{}, std::integral_constant<int, 0>{}, firstc, a, wl);
      if constexpr (HAS_A && HAS_B && NT == 2) {
        // Column JB's high term (products and their packed rounding), then
        // its high-term MFMAs with the residual term's VALU work between
        // them, then its residual-term MFMAs with column JA's split between
        // them, then column JA's MFMAs.
        constexpr int NBK = JB + 1, MA = NT * (JA + 1);
        constexpr int HALF = 8 * 5 / 2;                  // VALU ops of one term of a column
        constexpr int PER1 = (HALF + NBK - 1) / NBK;
        constexpr int PER2 = (2 * HALF + NBK - 1) / NBK;
        __builtin_amdgcn_sched_group_barrier(0x002, HALF, 0);    // JB: high term
#pragma unroll
        for (int m = 0; m < NBK; ++m) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // JB high-term MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, PER1, 0);  // part of JB's residual
        }
#pragma unroll
        for (int m = 0; m < NBK; ++m) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // JB residual-term MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, PER2, 0);  // part of column JA's split
        }
        __builtin_amdgcn_sched_group_barrier(0x008, MA, 0);      // column JA's MFMAs
      } else if constexpr (HAS_A && HAS_B) {
        constexpr int MB = NT * (JB + 1), MA = NT * (JA + 1);
        constexpr int SPLIT = 8 * 5;                     // VALU ops of one column's split
        constexpr int PER = (SPLIT + MB - 1) / MB;
        __builtin_amdgcn_sched_group_barrier(0x002, SPLIT, 0);   // split of column JB
#pragma unroll
        for (int m = 0; m < MB; ++m) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // one MFMA of column JB
          __builtin_amdgcn_sched_group_barrier(0x002, PER, 0);   // part of column JA's split
        }
        __builtin_amdgcn_sched_group_barrier(0x008, MA, 0);      // column JA's MFMAs
      }
    }
  };
  // One step: stage the prefetched data, barrier, prefetch the step two
  // ahead, compute. The two buffers alternate with the step parity.
  auto step = [&](Pre& buf, int half, auto firstc) {
    stage(buf, tiles + half * TILE, wts + half * kGramStep);
    __syncthreads();
    buf = gload();  // two steps ahead (empty past the chunk end): static wait counts
    __builtin_amdgcn_sched_barrier(0);        // keep the loads ahead of this step's MFMAs
    compute(tiles + half * TILE, wts + half * kGramStep, firstc);
  };

  static_assert(kGramFlush == 4, "the step loop below is unrolled by four");
  Pre b0 = gload();
  Pre b1 = gload();
  drain_vmem();  // prologue loads done: the loop's wait counts then stay static
  for (int st = 0; st < ga.nsteps; st += kGramFlush) {
    step(b0, 0, std::true_type{});
    step(b1, 1, std::false_type{});
    step(b0, 0, std::false_type{});
    step(b1, 1, std::false_type{});
#pragma unroll
    for (int p = 0; p < NP; ++p) acc2[p] = acc2[p] + acc32[p];
  }
  // Emit: column j, row block i -> global pair index of (i, j).
  auto emit = [&](auto jc, auto pbc) {
    constexpr int J = decltype(jc)::value, PBASE = decltype(pbc)::value;
#pragma unroll
    for (int i = 0; i <= J; ++i) {
      const int p = i * NB - (i * (i - 1)) / 2 + (J - i);
      *reinterpret_cast<floatx4*>(ga.out + p * 256 + lane * 4) = acc2[PBASE + i];
    }
  };
  if constexpr (HAS_A) emit(std::integral_constant<int, JA>{}, std::integral_constant<int, 0>{});
  if constexpr (HAS_B) emit(std::integral_constant<int, JB>{}, std::integral_constant<int, PA>{});
}

// NT = 2 bf16 terms of the weighted operand, every unit.
// POL: cache policy of the V loads (streamed, or kept in L2 for the other
// query-head units of the same KV head).
template <int D, int NT, int POL>
__global__ __launch_bounds__(kThreads, 2) void gram_mfma_kernel(
    Geo g, const uint16_t* __restrict__ v, const float* __restrict__ wbuf,
    const uint32_t* __restrict__ uflags, float* __restrict__ partials, int gchunks, int gchunk) {
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  constexpr int TILE = kGramStep * kGramPitch;
  int u, chunk;
  if (!grid_unit_chunk<true>(g, gchunks, u, chunk)) return;
  const Unit un = decode_unit(g, u);
  const int base = chunk * gchunk;
  if (base >= un.n) return;
  __shared__ __attribute__((aligned(16))) uint16_t tiles[2 * TILE];
  __shared__ __attribute__((aligned(16))) float wts[2 * kGramStep];
  GramArgs ga;
  ga.vb = v + un.l * g.vsl + un.h * g.vsh + un.t0 * g.vst;
  ga.vst = g.vst;
  ga.wrow = wbuf + token_row(g, un);
  ga.base = base;
  ga.end = min(un.n, base + gchunk);
  constexpr int SPAN = kGramStep * kGramFlush;
  ga.nsteps = (ga.end - base + SPAN - 1) / SPAN * kGramFlush;
  ga.out = partials + ((int64_t)u * gchunks + chunk) * (NPAIR * 256);
  switch (threadIdx.x >> 6) {
    case 0: gram_wave<D, 0, NT, POL>(ga, tiles, wts); break;
    case 1: gram_wave<D, 1, NT, POL>(ga, tiles, wts); break;
    case 2: gram_wave<D, 2, NT, POL>(ga, tiles, wts); break;
    default: gram_wave<D, 3, NT, POL>(ga, tiles, wts); break;
  }
}

// fp64 Gram: every unit of fp32 inputs, and (REFINE_ONLY) the units of bf16
// inputs that the factorisation marked kUnitRefine. Products w_i v_ij v_ik are
// exact in fp64 (a bf16 or fp32 value times an fp32 weight, times a bf16 or
// fp32 value), the sums fp64. Thread (ty, tx) of a 16 x 16 grid owns a
// (D/16) x (D/16) register tile of M; V is staged 32 tokens at a time. One
// partial per chunk of `pchunk` tokens, in the block-lane layout.
template <typename T, int D, bool REFINE_ONLY>
__global__ __launch_bounds__(kThreads) void gram_precise_kernel(
    Geo g, const T* __restrict__ v, const float* __restrict__ wbuf,
    const uint32_t* __restrict__ uflags, double* __restrict__ partials, int pchunks, int pchunk,
    int items) {
  constexpr int R = D / 16;
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  __shared__ float vs[32][D];
  __shared__ double ws[32];
  if constexpr (REFINE_ONLY) {
    // The flags of all the walk's items at once (a load per thread, not one
    // per item in turn): a workgroup with no marked unit ends here.
    bool any = false;
    for (int item = blockIdx.x + threadIdx.x * gridDim.x; item < items;
         item += gridDim.x * kThreads) {
      int u, chunk;
      any |= grid_unit_chunk_at<true>(g, pchunks, item, u, chunk) && (uflags[u] & kUnitRefine);
    }
    if (!__syncthreads_or(any)) return;
  }
  // one (unit, chunk) item per workgroup, or (REFINE_ONLY) a grid-stride walk
  for (int item = blockIdx.x; item < items; item += gridDim.x) {
  int u, chunk;
  if (!grid_unit_chunk_at<true>(g, pchunks, item, u, chunk)) continue;
  if (REFINE_ONLY && !(uflags[u] & kUnitRefine)) continue;
  const Unit un = decode_unit(g, u);
  const int base = chunk * pchunk;
  if (base >= un.n) continue;
  const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
  const T* vb = v + un.l * g.vsl + un.h * g.vsh;
  const int64_t trow = token_row(g, un);
  const int end = min(un.n, base + pchunk);
  double acc[R][R];
#pragma unroll
  for (int a = 0; a < R; ++a)
#pragma unroll
    for (int b = 0; b < R; ++b) acc[a][b] = 0.0;
  for (int t0 = base; t0 < end; t0 += 32) {
    __syncthreads();
    for (int e = tid; e < 32 * D; e += kThreads) {
      const int tok = e / D, c = e % D;
      vs[tok][c] = (t0 + tok < end) ? to_f32(vb[(un.t0 + t0 + tok) * g.vst + c]) : 0.0f;
    }
    if (tid < 32) {
      const int t = t0 + tid;
      ws[tid] = (t < end) ? (double)wbuf[trow + t] : 0.0;
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
  double* out = partials + ((int64_t)u * pchunks + chunk) * (NPAIR * 256);
#pragma unroll
  for (int a = 0; a < R; ++a)
#pragma unroll
    for (int b = 0; b < R; ++b) {
      const int row = ty * R + a, col = tx * R + b;
      const int i = row / 16, j = col / 16;
      if (i > j) continue;
      const int p = i * NB - (i * (i - 1)) / 2 + (j - i);
      const int ln = ((row % 16) / 4) * 16 + (col % 16);
      out[p * 256 + ln * 4 + (row % 4)] = acc[a][b];
    }
  __syncthreads();  // the staged tokens of this item are read before the next item's
  }
}

hipError_t launch_gram(const Launch& L, const void* v, bool refine) {
  const Geo& g = L.geo;
  const float* wb = ws_ptr<float>(L.wsp, L.ws.wgt);
  const uint32_t* uf = ws_ptr<uint32_t>(L.wsp, L.ws.uflags);
  if (L.ws.mfma && !refine) {
    const dim3 grid((unsigned)chunked_grid(g, L.ws.gchunks));
    float* part = ws_ptr<float>(L.wsp, L.ws.gram);
    const uint16_t* vv = (const uint16_t*)v;
    auto go = [&](auto kern) {
      kern<<<grid, kThreads, 0, L.stream>>>(g, vv, wb, uf, part, L.ws.gchunks, L.ws.gchunk);
    };
    if (g.D == 128) {
      if (g.V > 1) go(gram_mfma_kernel<128, 2, kPolicyShared>);
      else go(gram_mfma_kernel<128, 2, kPolicyStream>);
    } else {
      if (g.V > 1) go(gram_mfma_kernel<64, 2, kPolicyShared>);
      else go(gram_mfma_kernel<64, 2, kPolicyStream>);
    }
    return hipGetLastError();
  }
  if (!L.ws.mfma && refine) return hipSuccess;
  // fp64: all units of fp32 inputs, or the marked units of bf16 inputs
  const int64_t items = chunked_grid(g, L.ws.pchunks);
  const dim3 grid((unsigned)(L.ws.mfma ? std::min<int64_t>(items, kRefineBlocks) : items));
  double* part = ws_ptr<double>(L.wsp, L.ws.gram);
  auto go = [&](auto kern, auto vv) {
    kern<<<grid, kThreads, 0, L.stream>>>(g, vv, wb, uf, part, L.ws.pchunks, L.ws.pchunk,
                                          (int)items);
  };
  if (L.ws.mfma) {
    if (g.D == 128) go(gram_precise_kernel<uint16_t, 128, true>, (const uint16_t*)v);
    else go(gram_precise_kernel<uint16_t, 64, true>, (const uint16_t*)v);
  } else {
    if (g.D == 128) go(gram_precise_kernel<float, 128, false>, (const float*)v);
    else go(gram_precise_kernel<float, 64, false>, (const float*)v);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Reduce the per-chunk partials of each unit, entry by entry, in chunk order
// (fp64). grid = (U, NPAIR): one 16x16 block pair per workgroup.
// ---------------------------------------------------------------------------
template <typename P, int D>
__global__ __launch_bounds__(kThreads) void gram_reduce_kernel(Geo g, const P* __restrict__ partials,
                                                               int gchunks, int gchunk,
                                                               double* __restrict__ red) {
  constexpr int NB = D / 16;
  constexpr int NPAIR = NB * (NB + 1) / 2;
  const int u = blockIdx.x, p = blockIdx.y;
  const Unit un = decode_unit(g, u);
  const int nch = (un.n + gchunk - 1) / gchunk;
  const P* src = partials + (int64_t)u * gchunks * (NPAIR * 256) + p * 256 + threadIdx.x;
  double s = 0.0;
#pragma unroll 8
  for (int c = 0; c < nch; ++c) s += (double)src[(int64_t)c * (NPAIR * 256)];
  red[(int64_t)u * (NPAIR * 256) + p * 256 + threadIdx.x] = s;
}

// Batches whose units have more than kFactorSumChunks chunks; with fewer the
// first factorisation sums its unit's partials itself (see launch_factor).
hipError_t launch_gram_reduce(const Launch& L) {
  const Geo& g = L.geo;
  if (!gram_reduced(L)) return hipSuccess;
  const int NB = g.D / 16, npair = NB * (NB + 1) / 2;
  const dim3 grid(g.U, npair);
  double* red = ws_ptr<double>(L.wsp, L.ws.gram_red);
  if (L.ws.mfma) {
    const float* part = ws_ptr<float>(L.wsp, L.ws.gram);
    if (g.D == 128) gram_reduce_kernel<float, 128><<<grid, kThreads, 0, L.stream>>>(g, part, L.ws.gchunks, L.ws.gchunk, red);
    else gram_reduce_kernel<float, 64><<<grid, kThreads, 0, L.stream>>>(g, part, L.ws.gchunks, L.ws.gchunk, red);
  } else {  // fp64 partials
    const double* part = ws_ptr<double>(L.wsp, L.ws.gram);
    if (g.D == 128) gram_reduce_kernel<double, 128><<<grid, kThreads, 0, L.stream>>>(g, part, L.ws.pchunks, L.ws.pchunk, red);
    else gram_reduce_kernel<double, 64><<<grid, kThreads, 0, L.stream>>>(g, part, L.ws.pchunks, L.ws.pchunk, red);
  }
  return hipGetLastError();
}

}  // namespace jacap
