// ckv_score.hpp -- retrieval scoring of one tile of positions (MFMA path).
//
// The paper scores offloaded entries by the query's inner product with
// GPU-resident key summaries (Sec. 2.2, Sec. 4.1); with a summary per
// position the scan reads every key of the context once.  One KV head serves
// a group of G query heads, so the scores of a 16-key block form the dense
// product Q[16 x d] . K^T[d x 16] (heads padded to 16 rows), which is what a
// v_mfma_f32_16x16x32_bf16 computes in four steps over d = 128 channels.
//
// Operand placement (wave64): lane l holds key (l % 16) of the block as the B
// operand and query head (l % 16) as the A operand; lane group kg = l / 16
// supplies channels [32t + 8kg, 32t + 8kg + 8) of step t, so each load
// instruction reads 64 contiguous bytes of 16 key rows.  The accumulator of
// lane l then holds heads 4kg..4kg+3 of key (l % 16).
#pragma once

#include "ckv_device.hpp"

namespace ckv {

// Adds the workgroup's LDS histogram into the unit's global fine and coarse
// histograms (kScoreThreads threads, kHistBins bins).
__device__ __forceinline__ void flush_hist(const uint32_t* lds_hist,
                                           uint32_t* g_hist,
                                           uint32_t* g_coarse) {
  static_assert(kHistBins == 16 * kScoreThreads, "16 bins per thread");
  static_assert(kHistBins / kCoarseBins == 64, "4 threads per coarse bin");
  const int t = threadIdx.x;
  uint32_t csum = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint32_t v = lds_hist[16 * t + i];
    if (v) {
      atomicAdd(&g_hist[16 * t + i], v);
      csum += v;
    }
  }
  csum += __shfl_xor(csum, 1);
  csum += __shfl_xor(csum, 2);
  if ((t & 3) == 0 && csum) atomicAdd(&g_coarse[t >> 2], csum);
}

// Scores positions [tile*kScoreTile, +kScoreTile) of `unit` into a.scores
// (fp32, -inf at and beyond n_b) and, if HIST, counts their first radix digit.
// Must be called by all kScoreThreads threads of the workgroup.
template <int G, bool HIST>
__device__ __forceinline__ void score_tile(const ScoreArgs& a, int unit,
                                           int tile, uint32_t* lds_hist) {
  const int b = unit / a.Hkv, h = unit - b * a.Hkv;
  const int n = clamp_len(a.ctx_lens[b], a.max_ctx);
  const int j0 = tile * kScoreTile;
  const int jend = min(j0 + kScoreTile, a.max_ctx);
  float* srow = a.scores + (int64_t)unit * a.max_ctx;
  const int tid = threadIdx.x;
  if (j0 >= n) {  // uniform over the workgroup
    for (int j = j0 + tid; j < jend; j += kScoreThreads) srow[j] = -INFINITY;
    return;
  }
  if (HIST) {
    for (int i = tid; i < kHistBins; i += kScoreThreads) lds_hist[i] = 0u;
    __syncthreads();
  }
  const int lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;

  bf16x8 qa[4];
  {
    const uint16_t* qrow =
        a.q + ((int64_t)b * a.Hq + (int64_t)h * G + r16) * kD + 8 * kg;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (r16 < G) v = ld16(qrow + 32 * t);
      qa[t] = as_bf16x8(v);
    }
  }
  const uint16_t* kbase =
      a.keys + (int64_t)unit * a.max_ctx * a.key_stride + 8 * kg;
  const int wj0 = j0 + wave * (kScoreTile / 4);
  constexpr int kBlocks = kScoreTile / 4 / 16;

  for (int blk = 0; blk < kBlocks; blk += kScoreUnroll) {
    uint4 kv[kScoreUnroll][4];
#pragma unroll
    for (int u = 0; u < kScoreUnroll; ++u) {
      const int j = wj0 + (blk + u) * 16 + r16;
      if (j < n) {
        const uint16_t* p = kbase + (int64_t)j * a.key_stride;
#pragma unroll
        for (int t = 0; t < 4; ++t) kv[u][t] = ld16_nt(p + 32 * t);
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) kv[u][t] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int u = 0; u < kScoreUnroll; ++u) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 4; ++t) acc = mfma_16x16x32(qa[t], as_bf16x8(kv[u][t]), acc);
      float s = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (4 * kg + i < G) s = fmaxf(s, acc[i]);
      if (G > 4) s = fmaxf(s, __shfl_xor(s, 16));
      if (G > 8) s = fmaxf(s, __shfl_xor(s, 32));
      s *= a.scale;
      const int j = wj0 + (blk + u) * 16 + lane;
      if (lane < 16) {
        if (j < n) {
          srow[j] = s;
          if (HIST) atomicAdd(&lds_hist[order_key(s) >> (32 - kHistBits)], 1u);
        } else if (j < jend) {
          srow[j] = -INFINITY;
        }
      }
    }
  }
  if (HIST) {
    __syncthreads();
    flush_hist(lds_hist, a.hist + (int64_t)unit * kHistBins,
               a.coarse + (int64_t)unit * kCoarseBins);
  }
}

}  // namespace ckv
