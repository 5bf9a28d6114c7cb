// ckv_attn.hpp -- sparse decode attention over one chunk of selected rows.
//
// Sec. 5.3 / Sec. 5.4: the decoding token attends over exactly the assembled
// sparse set.  A workgroup takes kAttnRows selected rows of one (request, KV
// head) unit and produces, for each of the G query heads, the chunk's logit
// maximum m, the sum of exp(l_i - m) and the exp-weighted sum of V rows; the
// combine kernel merges chunks.
//
// Logits: Q[G x d] . K_chunk^T on MFMA (bf16 products are exact, fp32
// accumulation), same operand placement as the scoring pass.  Weights and the
// weighted V sum stay in fp32 on the VALU: rounding the weights to bf16 for an
// MFMA would cost up to 2^-9 relative per weight.
#pragma once

#include "ckv_device.hpp"

namespace ckv {

template <int G>
struct AttnLds {
  // K stage (4 waves x 32 rows, padded) | logits [G][rows] | partial sums
  // [4 waves][G][kD] | per-head max and weight sum
  static constexpr int kStage = 4 * kStageDwords;
  static constexpr int kFloats = kStage + G * kAttnRows + 4 * G * kD + 2 * G;
};

// All kAttnThreads threads of the workgroup must call this.  INDEXED: rows are
// source rows idx[unit][r] read in place; otherwise slot rows of a dense
// [U][k][d] buffer.
//
// Loads: wave w owns rows [32w, 32w+32); every load instruction reads four
// whole 256-byte rows (16 lanes x 16 bytes per row), K and V alike.  K goes
// through a padded LDS stage into the MFMA operand placement; V stays in
// registers in exactly the placement the weighted sum needs.
template <int G, bool INDEXED>
__device__ __forceinline__ void attn_chunk(const AttnArgs& a, int unit,
                                           int chunk, float* lds) {
  uint32_t* stage_all = reinterpret_cast<uint32_t*>(lds);
  float* lg = lds + AttnLds<G>::kStage;   // [G][kAttnRows] logits, then weights
  float* red = lg + G * kAttnRows;        // [4 waves][G][kD] partial sums
  float* stat = red + 4 * G * kD;         // [2][G] chunk max, weight sum
  const int b = unit / a.Hkv, h = unit - b * a.Hkv;
  const int nsel = clamp_len(a.n_sel[unit], a.k);
  const int r0 = chunk * kAttnRows;
  const int rows = min(kAttnRows, nsel - r0);
  float* part = a.part + ((int64_t)unit * a.chunks + chunk) * G * kPartStride;
  const int tid = threadIdx.x;
  if (rows <= 0) {  // uniform: empty chunk (zero weight, zero sums)
    for (int o = tid; o < G * kPartStride; o += kAttnThreads)
      part[o] = (o % kPartStride) == 0 ? -INFINITY : 0.f;
    return;
  }
  const int lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int lrow = lane >> 4, lchunk = lane & 15;
  uint32_t* stage = stage_all + wave * kStageDwords;

  auto row_off = [&](int i) -> int64_t {
    if (INDEXED) {
      int pos = a.idx[(int64_t)unit * a.k + r0 + i];
      pos = pos < 0 ? 0 : (pos >= a.max_ctx ? a.max_ctx - 1 : pos);
      return ((int64_t)unit * a.max_ctx + pos) * a.row_stride;
    }
    return ((int64_t)unit * a.k + r0 + i) * kD;
  };

  // K and V of rows 32w + 4it + lrow, 16-byte chunk lchunk of each.
  uint4 kr[8], vr[8];
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int i = wave * 32 + it * 4 + lrow;
    kr[it] = make_uint4(0u, 0u, 0u, 0u);
    vr[it] = make_uint4(0u, 0u, 0u, 0u);
    if (i < rows) {
      const int64_t off = row_off(i) + 8 * lchunk;
      kr[it] = ld16(a.k_rows + off);
      vr[it] = ld16(a.v_rows + off);
    }
  }
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
#pragma unroll
  for (int it = 0; it < 8; ++it)
    *reinterpret_cast<uint4*>(stage + (4 * it + lrow) * kStageRowDwords + 4 * lchunk) = kr[it];
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int bk = 0; bk < 2; ++bk) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint4 kv = *reinterpret_cast<const uint4*>(
          stage + (16 * bk + r16) * kStageRowDwords + 4 * (4 * t + kg));
      acc = mfma_16x16x32(qa[t], as_bf16x8(kv), acc);
    }
    const int r = wave * 32 + bk * 16 + r16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * kg + i;
      if (g < G) lg[g * kAttnRows + r] = r < rows ? acc[i] * a.scale : -INFINITY;
    }
  }
  __syncthreads();

  // Per-head softmax over the chunk (one wave per head, two rows per lane).
  for (int g = wave; g < G; g += 4) {
    const float x0 = lg[g * kAttnRows + lane];
    const float x1 = lg[g * kAttnRows + 64 + lane];
    const float mx = wave_max(fmaxf(x0, x1));  // finite: rows >= 1
    const float p0 = __expf(x0 - mx), p1 = __expf(x1 - mx);
    const float l = wave_sum(p0 + p1);
    lg[g * kAttnRows + lane] = p0;
    lg[g * kAttnRows + 64 + lane] = p1;
    if (lane == 0) {
      stat[g] = mx;
      stat[G + g] = l;
    }
  }
  __syncthreads();

  // Weighted V sum: lane holds channels [8*lchunk, +8) of 8 rows.
  float acc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[g][e] = 0.f;
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int i = wave * 32 + it * 4 + lrow;
    float vf[8];
    unpack8(vr[it], vf);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float p = lg[g * kAttnRows + i];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = acc[g][e];
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      acc[g][e] = x;
    }
  if (lrow == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[(wave * G + g) * kD + 8 * lchunk + e] = acc[g][e];
  }
  __syncthreads();
  for (int o = tid; o < G * kD; o += kAttnThreads) {
    const int g = o / kD, c = o - g * kD;
    const float sum = red[(0 * G + g) * kD + c] + red[(1 * G + g) * kD + c] +
                      red[(2 * G + g) * kD + c] + red[(3 * G + g) * kD + c];
    part[g * kPartStride + 4 + c] = sum;
  }
  if (tid < G) {
    part[tid * kPartStride] = stat[tid];
    part[tid * kPartStride + 1] = stat[G + tid];
  }
}

}  // namespace ckv
