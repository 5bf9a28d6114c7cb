// ckv_device.hpp -- device helpers and launch-argument structs shared by the
// libckv kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ckv {

constexpr int kD = 128;            // head_dim supported by the kernels
constexpr int kWave = 64;

// Scoring: a persistent grid; each workgroup scores a balanced contiguous
// range of kStageRows-key groups (4 waves, MFMA blocks of 16 keys).
constexpr int kScoreThreads = 256;
constexpr int kHistScoreWaves = 8;  // waves of the scoring kernel with histograms
constexpr int kStageRows = 32;     // key rows staged per wave per step
constexpr int kStageRowDwords = 68;  // 256-byte row + 16-byte pad (bank spread)
constexpr int kStageDwords = kStageRows * kStageRowDwords;
constexpr int kFlushGroups = 64;   // groups of scores held per wave in LDS
constexpr int kClaimGroups = 64;   // groups per claim of the dynamic scoring pass
constexpr int kMinClaimsPerWg = 4; // claims per workgroup from which a pass takes claims
constexpr int kScoreLdsDwords = 4 * kStageDwords + 4 * kFlushGroups * kStageRows;

// Selection: the first radix digit is the top 11 bits of the order key; a
// 64-bin coarse histogram (top 6 bits) finds its bin quickly.  The remaining
// 21 bits are resolved in two digits of 11 and 10 bits.
constexpr int kHistBits = 11;
constexpr int kHistBins = 1 << kHistBits;
constexpr int kCoarseBins = 64;
constexpr int kCtrlWords = 4;      // per unit: above, cand, digit-1 bin, and (unit 0
constexpr int kCtrlClaim = 3;      //   only) the scoring pass's claim counter
constexpr int kFilterThreads = 256;
constexpr int kFilterTile = 4096;  // positions per filter workgroup
constexpr int kFinishThreads = 1024;
constexpr int kFinishLdsBytes = 128 * 1024;   // candidates or bitmap
constexpr int kCandLds = kFinishLdsBytes / 8;  // (key, pos) pairs held in LDS
constexpr int kBitmapLdsBits = kFinishLdsBytes * 8;
// Contexts up to this many positions are selected by one workgroup per unit
// in a single kernel (scores read once, everything else in LDS).
constexpr int kFusedSelectMaxCtx = 65536;
// Scoring grids are capped at kMaxScoreWgs workgroups.  With per-workgroup
// histograms (ScoreArgs::hist_part) the histogram of unit u is the sum of the
// slots u + wg over the workgroups wg whose range meets the unit's groups
// (all of them, below n_b or not: a range past n_b stores zeros, so the
// slots to read follow from the shape alone); slot u + wg is unique because
// ranges and units are both in group order.  The selection
// reads at most kMaxPartials slots per unit, else the histograms are added
// with atomics.
constexpr int kMaxScoreWgs = 1024;
constexpr int kMaxPartials = 8;

// Attention: one workgroup reduces kAttnRows gathered rows of one unit into a
// partial (running max, sum of weights, weighted V) per query head; each of
// its 4 waves streams kWaveRows of them.
constexpr int kAttnThreads = 256;
constexpr int kWaveRows = 64;
constexpr int kAttnRows = 4 * kWaveRows;
constexpr int kPartStride = 132;   // floats per (chunk, head): m, l, pad, pad, o[128]
constexpr int kMergeChunks = 8;    // partials per unit the fused selection merges

// Selection and attention in one launch (same-step decode): a share of at
// most kSelAttnMaxShare selected rows per workgroup, at most kSelAttnMaxSplit
// shares per unit, group sizes up to 8.
constexpr int kSelAttnMaxShare = 2048;
constexpr int kSelAttnMaxSplit = 8;

// Gather: one thread moves 16 bytes per item; items are (unit, slot, K|V, part).
constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 4;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct ScoreArgs {
  const uint16_t* q;        // [B][Hq][d]
  const uint16_t* keys;     // unit rows at stride key_stride
  const int32_t* ctx_lens;  // [B]
  float* scores;            // [U][max_ctx]
  uint32_t* hist;           // [U][kHistBins] or nullptr
  uint32_t* coarse;         // [U][kCoarseBins]
  uint32_t* hist_part;      // non-null: per-workgroup histograms instead,
                            //   [U + kMaxScoreWgs][kHistBins], stored not added
  uint32_t* claim;          // pipelined launches with added histograms: workgroups
                            //   may take claims of kClaimGroups groups from this
                            //   counter, which is zero before the launch and after it
  int64_t key_stride;
  float scale;
  int Hq, Hkv, max_ctx, units;
  int chunk;                // rows per scored entry: n_b rows give ceil(n_b/chunk) entries
};

struct SelectArgs {
  const float* scores;      // [U][max_ctx]
  const int32_t* ctx_lens;  // [B]
  uint32_t* hist;           // [U][kHistBins]
  uint32_t* coarse;         // [U][kCoarseBins]
  uint32_t* ctrl;           // [U][kCtrlWords]
  const uint32_t* hist_part;  // non-null: the scoring pass wrote per-workgroup
  int score_nwg;            //   histograms with a grid of score_nwg workgroups
  int units;
  int32_t* sel;             // [U][k]   positions above the digit-1 bin, then
                            //          the chosen candidates
  uint2* cand;              // [U][max_ctx] (order key, position)
  uint32_t* bitmap;         // [U][bm_words] when max_ctx > kBitmapLdsBits
  int32_t* idx;             // [U][k]
  int32_t* n_sel;           // [U]
  int64_t bm_words;
  int Hkv, max_ctx, k, tiles;
  int chunk;                // as in ScoreArgs
  // Pipelined calls: the fused selection also merges the attention partials
  // of the launch before it (NULL mpart: a merge kernel runs instead).
  // mchunks <= kMergeChunks and mG * kD <= kFinishThreads.
  const float* mpart;       // [U][mchunks][mG][kPartStride]
  float* mout;              // [B][mHq][d]
  int mchunks, mG, mHq;
  // Non-zero: the slots come from the XCD-affine ranges of the one-launch
  // same-step kernel (xcd_slot0), not from ranges in plain unit order.
  int affine;
};


// The one-launch same-step kernel's hand-over from scoring to selection:
// once a scoring workgroup's scores and histogram slot of a unit are stored
// (device-coherent stores, waited for), it sets that slot's two flags, one for
// each of the unit's two attending workgroups, to the launch's tag; each of
// those waits for its flags of all the unit's slots and then clears them, so
// that they are zero again after the launch.  The tag's halves are each
// other's complement, so no stale word and no zero matches it.  With row
// halves the unit's first workgroup hands its attention partial to the
// second the same way, through the unit's merge flag.
struct FusedSync {
  uint64_t* flags;  // [U + kMaxScoreWgs][2]
  uint64_t* merge;  // [U], row halves only
  uint64_t tag;
};
// Every wait on these flags gives up after this many polls (about a second):
// a broken hand-over leaves outputs undefined but cannot hang a launch.
constexpr uint32_t kFusedSpinLimit = 1u << 20;

struct AttnArgs {
  const uint16_t* q;        // [B][Hq][d]
  const uint16_t* k_rows;   // buffer [U][k][d] or source rows (indexed)
  const uint16_t* v_rows;
  const int32_t* idx;       // indexed mode: [U][k] positions into the source
  const int32_t* n_sel;     // [U]
  float* part;              // [U][chunks][G][kPartStride]
  float* out;               // [B][Hq][d]
  // Two tokens (q2 != NULL): the G head rows of a unit are the current
  // token's G/2 heads (q, out) then the speculative token's (q2, out2); the
  // merge adds the tokens' own rows k_local/v_local [U][2][d] under the
  // causal mask (current: row 0; speculative: rows 0 and 1).
  const uint16_t* q2;
  float* out2;
  const uint16_t* k_local;
  const uint16_t* v_local;
  int64_t row_stride;       // indexed mode: source row stride
  float scale;
  int Hq, Hkv, max_ctx, k, chunks;
};

struct GatherArgs {
  const uint16_t* k_src;
  const uint16_t* v_src;
  const int32_t* idx;
  const int32_t* n_sel;
  const int32_t* slots;     // [U][k] destination slot of entry i; NULL: slot i
  uint16_t* k_dst;
  uint16_t* v_dst;
  int64_t row_stride;
  int64_t items;            // U * k * 32
  int max_ctx, k;
};

// Chunk landmarks: the mean key of every chunk of `chunk` rows.
struct LandmarkArgs {
  const uint16_t* keys;     // unit rows at stride key_stride
  const int32_t* ctx_lens;  // [B]
  uint16_t* landmarks;      // [U][cmax][d]
  int64_t key_stride;
  int64_t items;            // U * cmax * 16 (16 bytes of a landmark each)
  int Hkv, max_ctx, chunk, cmax;
};

// Low-rank key reconstruction: K row = U row . W, rounded once to bf16.
struct ReconArgs {
  const uint16_t* u_fac;    // [U][max_ctx][rank]
  const uint16_t* w_fac;    // [U][rank][d]
  const int32_t* idx;       // [U][k] rows to rebuild
  const int32_t* n_sel;     // [U]
  const int32_t* slots;     // [U][k] destination slot of entry i; NULL: slot i
  uint16_t* k_dst;          // [U][k][d]
  int64_t items;            // U * k * 16
  int max_ctx, k, rank;
};

// Rows of the selected chunks.
struct ExpandArgs {
  const int32_t* chunk_idx; // [U][kc] ascending
  const int32_t* n_chunks;  // [U]
  const int32_t* ctx_lens;  // [B]
  int32_t* rows;            // [U][k] written
  int32_t* n_rows;          // [U] written
  int Hkv, max_ctx, chunk, kc, k;
};

// Miss detection: the selected set against the predicted set in the buffer.
constexpr int kMissThreads = 1024;
constexpr int kMissLds = 8192;  // budgets up to this keep both sets in LDS

struct MissArgs {
  const int32_t* idx_true;  // [U][k] ascending, -1 padded
  const int32_t* n_true;    // [U]
  const int32_t* idx_pred;  // [U][k] ascending, -1 padded
  const int32_t* n_pred;    // [U]
  int32_t* slot_of;         // [U][k] written: buffer slot of idx_true[i]
  int32_t* miss_pos;        // [U][k] written: positions to fetch
  int32_t* miss_slot;       // [U][k] written: their slots
  int32_t* n_miss;          // [U] written
  int32_t* hits;            // [U] written
  int32_t* free_slot;       // [U][k] scratch when k > kMissLds
  int k;
};

// ---- small device helpers ---------------------------------------------------

// Entries of a unit with n_b context rows when one entry covers `chunk` rows:
// ceil(n_b / chunk), clamped to [0, hi].
__device__ __forceinline__ int unit_len(int n_rows, int hi, int chunk) {
  const int n = max(n_rows, 0);
  return min(n / chunk + (n % chunk != 0 ? 1 : 0), hi);
}

__device__ __forceinline__ int clamp_len(int n, int hi) {
  return n < 0 ? 0 : (n > hi ? hi : n);
}

// Workgroup of the balanced split of T groups over nwg workgroups (range
// [wg*T/nwg, (wg+1)*T/nwg)) that holds group g.
__host__ __device__ __forceinline__ int64_t range_owner(int64_t g, int64_t T, int64_t nwg) {
  return ((g + 1) * nwg - 1) / T;
}

// The one-launch same-step kernel's scoring ranges: its scoring workgroups
// are spread over the 8 XCDs round-robin by index, and the workgroups
// x, x + 8, x + 16, ... (XCD x) score the units x, x + 8, x + 16, ... in
// balanced contiguous ranges of those units' groups.  A unit's scores are
// then written on the XCD where its selection and attention run (the same
// index map, split_block), and the units of an XCD are complete as soon as
// that XCD's ranges are.  Needs U and nwg multiples of 8.  The slot of (unit,
// workgroup) is unique within XCD x's block of U/8 + nwg/8 slots, as in plain
// unit order.  xcd_slot0 returns the first slot of `unit` and the number of
// consecutive slots that hold its histogram.
__host__ __device__ __forceinline__ int64_t xcd_slot0(int unit, int units, int nwg,
                                                      int64_t gu, int* nslots) {
  const int x = unit & 7, v = unit >> 3;
  const int ux = units >> 3, nx = nwg >> 3;
  const int64_t T = (int64_t)ux * gu;
  const int64_t lo = range_owner((int64_t)v * gu, T, nx);
  const int64_t hi = range_owner((int64_t)v * gu + gu - 1, T, nx);
  *nslots = (int)(hi - lo + 1);
  return (int64_t)x * (ux + nx) + v + lo;
}

// Monotone map from fp32 to uint32: a < b as floats <=> key(a) < key(b);
// -0 is folded onto +0 so that equal values compare equal.
__device__ __forceinline__ uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// The key test key(x) >= K as one fp32 compare, x >= float(bits), exact for
// every x that is not NaN; K ranges over [0, 2^32] (2^32: no key).  A key at
// or above 0x80000000 maps back to the non-negative float it encodes (+inf
// and beyond: NaN bits, which no x reaches); one at or below that of -inf
// admits every non-NaN x; others map to the negative float with that key
// (0x7fffffff, which no float has, gives -0: x >= -0 <=> key(x) >= +0's).
__host__ __device__ __forceinline__ uint32_t key_floor_bits(uint64_t K) {
  if (K >= (1ull << 32)) return 0x7fc00000u;
  const uint32_t k = (uint32_t)K;
  if (k >= 0x80000000u) return k ^ 0x80000000u;
  if (k <= 0x007fffffu) return 0xff800000u;
  return ~k;
}

__device__ __forceinline__ uint4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Streaming load (nontemporal hint: the line is not kept in the caches).
__device__ __forceinline__ uint4 ld16_nt(const uint16_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Exact widening of the 8 bf16 values packed in v (lowest element first).
// bf16 bit pattern of a finite fp32 value, rounded to nearest, ties to even.
__device__ __forceinline__ uint32_t bf16_rne_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ void unpack8(uint4 v, float* f) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// DPP lane exchange within rows of 16 lanes (no LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Max / sum over the 16 lanes of each row; every lane of the row gets it.
// quad_perm [1,0,3,2] and [2,3,0,1] reduce a quad, row_half_mirror pairs the
// two quads of each half row, row_mirror the two half rows.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_f32<0xB1>(x));
  x = fmaxf(x, dpp_f32<0x4E>(x));
  x = fmaxf(x, dpp_f32<0x141>(x));
  return fmaxf(x, dpp_f32<0x140>(x));
}

__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f32<0xB1>(x);
  x += dpp_f32<0x4E>(x);
  x += dpp_f32<0x141>(x);
  return x + dpp_f32<0x140>(x);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}


// Wave-aggregated append: lanes with `flag` get consecutive slots from the
// counter at *ctr (one atomic per wave); returns this lane's slot.
__device__ __forceinline__ uint32_t wave_append(bool flag, uint32_t* ctr) {
  const unsigned long long mask = __ballot(flag);
  const uint32_t cnt = (uint32_t)__popcll(mask);
  const uint32_t lo = (uint32_t)mask, hi = (uint32_t)(mask >> 32);
  const uint32_t rank = __builtin_amdgcn_mbcnt_hi(hi, __builtin_amdgcn_mbcnt_lo(lo, 0u));
  const int leader = cnt ? __ffsll(mask) - 1 : 0;
  uint32_t base = 0u;
  if (cnt && (int)(threadIdx.x & 63) == leader) base = atomicAdd(ctr, cnt);
  base = __builtin_amdgcn_readlane(base, leader);
  return base + rank;
}

template <int CTRL, int ROW_MASK, bool ZERO_FILL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROW_MASK, 0xF, ZERO_FILL);
}

// Workgroup barrier for LDS traffic only: waits for the wave's own LDS (and
// scalar) operations, not for its outstanding global loads, which
// __syncthreads would drain as well.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Inclusive prefix sum over the 64 lanes of a wave, in DPP moves only: a
// Hillis-Steele scan inside each row of 16 lanes (row_shr 1, 2, 4, 8, lanes
// shifted in from outside the row read 0), then the total of row 0 added to
// row 1 and of row 2 to row 3 (row_bcast:15), then the total of rows 0-1 to
// rows 2-3 (row_bcast:31).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += dpp_u32<0x111, 0xF, true>(x);
  x += dpp_u32<0x112, 0xF, true>(x);
  x += dpp_u32<0x114, 0xF, true>(x);
  x += dpp_u32<0x118, 0xF, true>(x);
  x += dpp_u32<0x142, 0xA, false>(x);
  x += dpp_u32<0x143, 0xC, false>(x);
  return x;
}

// Sum over the 64 lanes of a wave, the same in every lane.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
  return __builtin_amdgcn_readlane(wave_incl_scan(x), 63);
}

// Inclusive prefix sum over a workgroup of NW waves.  `tmp` is LDS scratch of
// at least NW+1 words.  Ends with a barrier; returns the thread's inclusive
// sum and writes the workgroup total to *total.
template <int NW>
__device__ __forceinline__ uint32_t block_incl_scan(uint32_t x, uint32_t* tmp,
                                                    uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t s = wave_incl_scan(x);
  if (lane == 63) tmp[wave] = s;
  __syncthreads();
  if (wave == 0) {
    uint32_t t = lane < NW ? tmp[lane] : 0u;
    uint32_t ts = wave_incl_scan(t);
    if (lane < NW) tmp[lane] = ts - t;  // exclusive wave offsets
    if (lane == NW - 1) tmp[NW] = ts;
  }
  __syncthreads();
  s += tmp[wave];
  *total = tmp[NW];
  __syncthreads();
  return s;
}

}  // namespace ckv
