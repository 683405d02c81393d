// Internal definitions shared by the HIP kernels and the C-ABI host code of
// libjacap.so (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jacap.h"

namespace jacap {

// ---------------------------------------------------------------------------
// Tiling constants
// ---------------------------------------------------------------------------
constexpr int kThreads = 256;        // 4 wave64 per workgroup
constexpr int kKChunk = 1024;        // tokens per workgroup in the K pass
constexpr int kFullMaxQ = 256;       // window queries the FULL-covariance MFMA K pass stages
// FULL covariance: units of at least this many tokens take kappa from the
// triangular factor of Lambda_Q (a fixed per-unit cost that long units repay).
constexpr int kTriMinTokens = 8192;
constexpr int kTriChunks = 4;         // K-pass chunks per workgroup on that path: at most
constexpr int kGChunkMfma = 512;     // tokens per workgroup in the MFMA Gram pass: at least
constexpr int kGChunkMfmaMax = 16384; // ... and at most (larger chunks: fewer partial Grams)
constexpr int kGramMinBlocks = 2048;  // chunks are as large as this many blocks in the grid allow
constexpr int kGramSpan = 128;       // tokens between two flushes of the Gram's short fp32 chains
constexpr int kGChunkPrecise = 128;  // tokens per workgroup in the fp64 Gram pass: at least
constexpr int kPrecisePartials = 256;  // fp64 Gram partials per batch the chunking aims at
constexpr int kLChunkMfma = 4096;    // tokens per workgroup in the MFMA leverage pass: at most
constexpr int kLChunkMfmaMin = 256;  // ... and at least (batches too small to fill the chip)
constexpr int kLevMinBlocks = 2048;  // leverage chunks shrink until the grid has this many blocks
constexpr int kLChunkPrecise = 1024; // tokens per workgroup in the fp64 leverage pass (fp32 keys):
constexpr int kLChunkPreciseMin = 64; // ... at most, and at least (small batches)
constexpr int kLChunkRefine = 4096;  // ... and over the bf16 units that take the fp64 path
constexpr int kWChunk = 4096;        // tokens per workgroup in the weight pass
// The K pass sums a chunk's exp(z - max) terms (all but the max's own) as
// exp(z - max + kRestShift) in fp32, so that they stay normal down to
// z - max ~ -150 (a sharply peaked softmax at small temperature).
constexpr float kRestShift = 64.0f;
constexpr int kGreedyMaxLen = 524288; // longest sequence the greedy selection takes
constexpr int kGreedyMaxD = 128;
constexpr int64_t kMaxTokenStride = int64_t(1) << 24;  // elements between consecutive K / V rows

// Unit flags (per (seq, layer, kv head)); the public flags are the OR of all.
constexpr uint32_t kUnitNonfinite = JACAP_FLAG_NONFINITE;
constexpr uint32_t kUnitSingular = JACAP_FLAG_SINGULAR;
// Internal (bf16 path only): the unit's capacity matrix is ill-conditioned
// enough (or one of its pivots small enough) that the fp32-accumulated Gram
// and the bf16 leverage products could miss the score tolerance; its Gram,
// factor and leverage scores are recomputed in fp64.
constexpr uint32_t kUnitRefine = 1u << 8;
// Internal (FULL covariance on the triangular path): the unit's K pass takes
// the window tile instead -- too few tokens to repay factoring Lambda_Q, a
// numerically rank-deficient Lambda_Q, or non-finite queries.
constexpr uint32_t kUnitKTile = 1u << 9;
constexpr uint32_t kUnitFailed = kUnitNonfinite | kUnitSingular;

// ---------------------------------------------------------------------------
// Geometry passed by value to every kernel
// ---------------------------------------------------------------------------
struct Geo {
  int L, H, Hq, G, D, w, B, U;  // U = B * L * H * V units
  int V;                        // query heads scored apart per KV head (1: the group pooled)
  int maxn;                     // host-declared max sequence length
  int64_t T;                    // packed tokens per (layer, head)
  const int32_t* seq_off;       // device [B+1]
  const double* ridge_mat;      // device [L][H][D][D] replacing ridge * I, or null
  int64_t ksl, ksh, kst;
  int64_t vsl, vsh, vst;
  int64_t qss, qsl, qsh, qsp;
  int64_t oss, osl, osh, osr;
};

struct Unit {
  int b, l, h;  // sequence, layer, KV head
  int s;        // query head within the group, when the V heads are scored apart
  int64_t t0;  // first packed token of the sequence
  int n;       // tokens of the sequence
};

// A sequence whose offsets are inconsistent with the host-declared geometry is
// treated as empty (and reported by the query-statistics kernel), so no kernel
// ever indexes outside [0, T) or past the chunk grid sized from maxn.
__device__ __forceinline__ bool offsets_ok(const Geo& g, int32_t a, int32_t e) {
  return a >= 0 && e >= a && (int64_t)e <= g.T && e - a <= g.maxn;
}

__device__ __forceinline__ Unit decode_unit(const Geo& g, int u) {
  Unit r;
  r.s = u % g.V;
  const int uk = u / g.V;
  r.h = uk % g.H;
  r.l = (uk / g.H) % g.L;
  r.b = uk / (g.H * g.L);
  const int32_t a = g.seq_off[r.b];
  const int32_t e = g.seq_off[r.b + 1];
  r.t0 = a;
  r.n = offsets_ok(g, a, e) ? e - a : 0;
  return r;
}

// Offset of per-token arrays laid out like the scores: [L][H][V][T].
__device__ __forceinline__ int64_t token_row(const Geo& g, const Unit& un) {
  return (((int64_t)un.l * g.H + un.h) * g.V + un.s) * g.T + un.t0;
}

// Workgroup -> (unit, chunk) of the passes that cut units into chunks, over
// a one-dimensional grid of chunked_grid() workgroups. The base order of the
// (KV unit, chunk) pairs is chunk-major (every unit's first chunk, then the
// second ...) or unit-major. With the query heads of a group scored apart
// (V > 1) the V units of one KV head read the same K or V rows: the V
// workgroups of a pair are placed 8 apart in dispatch order, so that they
// land on the same XCD (workgroups go to the 8 XCDs in turn) at about the same
// time, and every read after the first hits that XCD's L2. False for the
// padding past the last pair.
template <bool CHUNK_MAJOR>
__device__ __forceinline__ bool grid_unit_chunk_at(const Geo& g, int nchunks, int p, int& u,
                                                   int& chunk) {
  int s = 0;
  if (g.V > 1) {
    const int r = p % (8 * g.V);
    s = r >> 3;
    p = p / (8 * g.V) * 8 + (r & 7);
  }
  const int nk = g.U / g.V;
  int uk;
  if (CHUNK_MAJOR) {
    uk = p % nk;
    chunk = p / nk;
  } else {
    uk = p / nchunks;
    chunk = p % nchunks;
  }
  u = uk * g.V + s;
  return uk < nk && chunk < nchunks;
}

template <bool CHUNK_MAJOR>
__device__ __forceinline__ bool grid_unit_chunk(const Geo& g, int nchunks, int& u, int& chunk) {
  return grid_unit_chunk_at<CHUNK_MAJOR>(g, nchunks, blockIdx.x, u, chunk);
}

// Workgroups of the kernels that serve only the units marked for the fp64 path
// (usually none or few): they walk the (unit, chunk) items in a grid-stride
// loop and skip unmarked units, so a launch costs a few microseconds however
// many units and chunks the batch has.
constexpr int kRefineBlocks = 512;
constexpr int kComputeUnits = 256;  // MI355X

inline int64_t chunked_grid(const Geo& g, int nchunks) {
  const int64_t pairs = (int64_t)nchunks * (g.U / g.V);
  return g.V == 1 ? pairs : (pairs + 7) / 8 * 8 * g.V;
}

// ---------------------------------------------------------------------------
// Workspace layout (byte offsets from the workspace base; 256-byte aligned)
// ---------------------------------------------------------------------------
struct Workspace {
  size_t status;   // uint32: OR of the public flags
  size_t uflags;   // uint32 [U]
  size_t mu;       // double [U][D]
  size_t lam;      // double [U][D]          (diagonal covariance)
  size_t lamfull;  // float  [U][D][D]       (full covariance, FULL mode only)
  size_t smax_m;   // float  [U]             global logit max
  size_t smax_z;   // double [U]             global sum of exp(z - m)
  size_t wscale;   // double [U]             power of two by which the stored weights are scaled
  size_t z;        // float  [L][H][T]       centre logits
  size_t kappa;    // float  [L][H][T]       query response
  size_t cstat;    // float2 [U][kchunks]    per-chunk (max, sum exp)
  size_t wgt;      // float  [L][H][T]       importance weights (Eq. 8)
  size_t hscore;   // float  [L][H][G][T]    per-query-head scores (per-head GQA mode)
  size_t kept;     // int32  [B][L][H][budget] kept positions, staged by jacap_select_evicted
  size_t gram;     // per-chunk partial Grams: [U][gchunks][NPAIR*256] fp32 (bf16 MFMA pass)
                   // or [U][pchunks][NPAIR*256] fp64 (fp64 pass); one buffer for both
  size_t gram_red; // double [U][NPAIR*256]  the reduced Gram (gram_reduced), block-lane
                   // layout; after an fp64 factorisation, L^{-1} in the lower-block
                   // layout (see k_factor.hip)
  size_t lfrag;    // bf16 [U][NLP][2][64][8] L^{-1} hi/lo MFMA B fragments, bf16 path
  size_t gc;       // double [L][H][T]       greedy: c_i when last computed
  size_t gst;      // int32  [L][H][T]       greedy: picks made at that time (-1 = taken)
  size_t gent;     // GreedyEntry [U][ceil(maxn / 256)]  greedy: best of each 256-position block
  size_t total;
  int kchunks, wchunks, gchunks, gchunk, gparts, lchunks, lchunk;
  int pchunks, pchunk;  // chunks of the fp64 Gram pass
  int plchunks, plchunk;  // chunks of the fp64 leverage pass
  bool mfma;       // bf16 path (MFMA Gram and leverage)
};

// Best token of one 256-position block in the greedy log-det search.
struct GreedyEntry {
  double key;     // w_i c_i (-inf: no candidate left in the block)
  double c;       // c_i = u_i^T A^{-1} u_i as last computed
  int32_t pos;    // position in the sequence (INT32_MAX: none)
  int32_t stamp;  // number of picks when c_i was computed
};

// ---------------------------------------------------------------------------
// Small device helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// float -> bfloat16, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ float to_f32(T x);
template <>
__device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf16_to_f32(x); }

// DPP lane exchanges inside each 16-lane row (one VALU instruction each):
// quad swaps (lane ^ 1, lane ^ 2), the half-row mirror (i <-> 7 - i within 8)
// and the row mirror (i <-> 15 - i).
constexpr int kDppQuadXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, 0xF, 0xF, true);
  const uint32_t hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, 0xF, 0xF, true);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Wave64 butterfly reductions: every lane ends with the same, order-fixed value
// (IEEE addition is commutative, so partner lanes compute identical sums).
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ double wave_max_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Block (kThreads = 4 waves) reductions with a fixed combination order.
template <typename T, typename Op>
__device__ __forceinline__ T block_combine(T wave_val, T* red, Op op) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = wave_val;
  __syncthreads();
  T r = red[0];
#pragma unroll
  for (int i = 1; i < kThreads / 64; ++i) r = op(r, red[i]);
  return r;
}

__device__ __forceinline__ void raise_flags(uint32_t* status, uint32_t* uflags, int u,
                                            uint32_t f) {
  atomicOr(status, f);
  atomicOr(uflags + u, f);
}

// Raw buffer resource over [base, base + bytes): loads at byte offsets at or
// past `bytes` return zeros instead of touching memory (the descriptor's
// range check; stride 0, 32-bit data format). Used to read the rows of one
// step of a streaming loop without clamping row indices: the range ends at
// the last row the step may use, and the per-lane offsets stay constant.
constexpr int kBufferFormat = 0x00020000;
// Cache policy of a streamed load: non-temporal (no reuse expected). Only for
// loads whose wave reads whole 128-byte lines: a line read in halves by two
// loads would be fetched twice.
constexpr int kPolicyStream = 2;
// Cache policy of loads whose lines other workgroups of the XCD read next (the
// query-head units of one KV head): the default, so that they stay in L2.
constexpr int kPolicyShared = 0;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_range(const void* base, int32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kBufferFormat);
}
// Bytes of the rows [0, rows) of a row range whose row stride is `stride`
// bytes and whose rows are `row_bytes` long (0 for rows <= 0). The caller keeps
// rows * stride below 2^31.
__device__ __forceinline__ int32_t rows_bytes(int32_t rows, int32_t stride, int32_t row_bytes) {
  return rows > 0 ? (rows - 1) * stride + row_bytes : 0;
}
template <int POLICY = 0>
__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, int32_t off) {
  const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, POLICY);
  return uint4{x[0], x[1], x[2], x[3]};
}
__device__ __forceinline__ float buffer_load_f32(__amdgpu_buffer_rsrc_t r, int32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// Waits for every outstanding vector-memory load of this wave. Placed after a
// kernel's prologue loads (values used throughout a pipelined loop), so that
// the compiler's wait analysis does not carry them into the loop, where it
// would otherwise wait for all loads -- the prefetched ones included -- in
// every trip.
__device__ __forceinline__ void drain_vmem() {
  // s_waitcnt encoding (gfx9): vmcnt = 0, expcnt = 7, lgkmcnt = 15 (no wait).
  __builtin_amdgcn_s_waitcnt(0x0F70);
}

// ---------------------------------------------------------------------------
// Optional per-phase event timing (jacap_timing_start / _stop): records a HIP
// event pair around the scope on `stream` when the phase is enabled.
// ---------------------------------------------------------------------------
class TimedPhase {
 public:
  // enabled = false: never records (no event is created), whatever the mask.
  TimedPhase(hipStream_t stream, int phase, bool enabled = true);
  ~TimedPhase();
  TimedPhase(const TimedPhase&) = delete;
  TimedPhase& operator=(const TimedPhase&) = delete;

 private:
  hipStream_t stream_;
  int phase_;
  hipEvent_t begin_ = nullptr, end_ = nullptr;
};

// ---------------------------------------------------------------------------
// Launchers (defined in the kernel translation units)
// ---------------------------------------------------------------------------
struct Launch {
  const jacap_config* cfg;
  Geo geo;
  Workspace ws;
  bool timed = true;  // phases may be recorded by the timing API
  char* wsp;  // workspace base
  hipStream_t stream;
};

hipError_t launch_init(const Launch& L);
hipError_t launch_qstats(const Launch& L, const void* q);
hipError_t launch_stats_in(const Launch& L, const double* mu, const double* lambda);
hipError_t launch_kpass(const Launch& L, const void* k, const void* q);
// FULL covariance with bf16 keys and the window queries at hand (q != null):
// the K pass takes the MFMA tile of the queries, and the d x d Lambda is not
// formed.
inline bool full_kpass_on_mfma(const Launch& L, const void* q) {
  return L.cfg->cov_mode == JACAP_COV_FULL && L.cfg->dtype == JACAP_DTYPE_BF16 && q != nullptr &&
         L.geo.G * L.geo.w <= kFullMaxQ;
}
// ... and with at least 2 d window queries, where ||X k||^2 (Lambda_Q = X^T X,
// X lower triangular: about 1.1 d^2 bf16 MACs per token in two terms) costs
// less than the window tile's N_s d, when some unit is long enough: Lambda_Q
// is formed and factored per unit first (launch_qfactor), and the units it
// marks kUnitKTile keep the window tile.
inline bool full_kpass_tri(const Launch& L, const void* q) {
  return full_kpass_on_mfma(L, q) && L.geo.G * L.geo.w >= 2 * L.geo.D &&
         L.geo.maxn >= kTriMinTokens;
}
hipError_t launch_qfactor(const Launch& L, const void* q);
hipError_t launch_softmax_weights(const Launch& L);
hipError_t launch_head_mean(const Launch& L, const float* hs, float* scores);
hipError_t launch_gram(const Launch& L, const void* v, bool refine);
// The first factorisation sums each unit's Gram partials itself when units
// have at most kFactorSumChunks chunks (the loads of a few chunks stay in
// flight together); with more, a reduce kernel sums them over many
// workgroups first and the factorisation reads the reduced Gram.
constexpr int kFactorSumChunks = 4;
inline bool gram_reduced(const Launch& L) {
  return (L.ws.mfma ? L.ws.gchunks : L.ws.pchunks) > kFactorSumChunks;
}
hipError_t launch_gram_reduce(const Launch& L);
hipError_t launch_factor(const Launch& L, bool refine);
hipError_t launch_leverage(const Launch& L, const void* v, float* scores);
hipError_t launch_leverage_precise(const Launch& L, const void* v, float* scores);
hipError_t launch_select(const Launch& L, const float* scores, int32_t* idx);
hipError_t launch_select_evicted(const Launch& L, const float* scores, int32_t* slots, int cap);
hipError_t launch_compact(const Launch& L, const int32_t* idx, const void* k, const void* v,
                          void* ko, void* vo);
hipError_t launch_greedy(const Launch& L, const void* v, int32_t* idx, int32_t* order,
                         double* logdet);

// Host side of the entry points (jacap_host.hip): validation of the
// descriptors and workspace, and the launch sequence of jacap_evict once the
// problem is prepared.
jacap_status prepare_launch(const jacap_config* c, const jacap_batch* b, void* ws, size_t ws_bytes,
                            void* stream, Launch* L);
jacap_status check_evict_ptrs(const jacap_config* c, const jacap_batch* b, const void* q,
                              const void* k, const void* v, const float* scores,
                              const int32_t* idx, const void* k_out, const void* v_out);
jacap_status evict_prepared(const Launch& L, const void* q, const void* k, const void* v,
                            float* scores, int32_t* idx, void* k_out, void* v_out);

template <typename T>
__host__ __device__ __forceinline__ T* ws_ptr(char* base, size_t off) {
  return reinterpret_cast<T*>(base + off);
}

}  // namespace jacap
