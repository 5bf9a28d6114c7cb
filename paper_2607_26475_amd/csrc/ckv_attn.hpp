// ckv_attn.hpp -- sparse decode attention over one chunk of selected rows.
//
// Sec. 5.3 / Sec. 5.4: the decoding token attends over exactly the assembled
// sparse set.  A workgroup takes kAttnRows selected rows of one (request, KV
// head) unit and produces, for each of the G query heads, the chunk's logit
// maximum m, the sum of exp(l_i - m) and the exp-weighted sum of V rows; the
// combine kernel merges chunks.
//
// Logits: Q[G x d] . K_chunk^T on MFMA (bf16 products are exact, fp32
// accumulation), same operand placement as the scoring pass.  Softmax weights
// are fp32.  The weighted V sum also runs on MFMA: each fp32 weight p is split
// into two bf16 parts, hi = bf16(p) and lo = bf16(p - hi) (p - hi is exact in
// fp32), and one 16x16x32 product takes both parts against the same V entry,
// so hi*v + lo*v is accumulated in fp32 with exact products.  |p - hi - lo| <=
// 2^-18 p, so the sum carries at most 2^-18 of sum_i p_i |v_i| beyond fp32
// accumulation (a bf16 weight alone would cost up to 2^-9).  An empty chunk
// (all rows past n_sel) yields m = -inf and zero sums, which the combine
// ignores.
#pragma once

#include "ckv_device.hpp"

namespace ckv {

template <int G>
struct AttnLds {
  // K stage (4 waves x 16 rows, padded) | per-wave weight table
  // [4][16 rows x G + G rescale] | per-wave partials [4][G][kD + 2] |
  // query rows in the MFMA A placement [16][kD] bf16 (rows past G zero)
  static constexpr int kStage = 4 * 16 * kStageRowDwords;
  static constexpr int kPTab = 16 * G + G + (G < 4 ? 4 - G : 0);
  static constexpr int kP = 4 * kPTab;
  static constexpr int kMerge = 4 * G * (kD + 2);
  static constexpr int kQ = 16 * kStageRowDwords;
  static constexpr int kFloats = kStage + kP + kMerge + kQ;
};

// All kAttnThreads threads of the workgroup must call this.  The workgroup
// covers selected rows [chunk*kAttnRows, +kAttnRows) of `unit`; wave w owns
// the kWaveRows rows starting at w*kWaveRows and streams them in blocks of 16
// with an online softmax (running max m, weight sum l and weighted V sum o
// per query head), keeping the next block's loads in flight.  The four
// waves' states are merged through LDS into the chunk's partial.  INDEXED:
// rows are source rows idx[unit][r] read in place; otherwise slot rows of a
// dense [U][k][d] buffer.
//
// Loads: every instruction reads four whole 256-byte rows (16 lanes x 16
// bytes per row), K and V alike.  K goes through a padded per-wave LDS stage
// into the MFMA operand placement (logits Q[G x d] . K^T on MFMA).  V stays in
// registers: lane (r, c) of the wave (r = lane / 16, c = lane % 16) holds
// channels [8c, 8c + 8) of block rows r, r + 4, r + 8, r + 12, which is the
// B placement of a 16x16x32 product over those four rows (each twice, for
// the hi and lo weight parts) for one channel of each 8-channel group.  Eight
// products per block, one per channel offset e, accumulate
// O[head][8n + e] in lane (head / 4, n), register head % 4.
template <int G, bool INDEXED>
__device__ __forceinline__ void attn_chunk(const AttnArgs& a, int unit,
                                           int chunk, float* lds) {
  static_assert(kWaveRows % 16 == 0 && 4 * kWaveRows == kAttnRows, "4 waves per chunk");
  constexpr int kBlocks = kWaveRows / 16;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int lrow = lane >> 4, lchunk = lane & 15;
  const int b = unit / a.Hkv, h = unit - b * a.Hkv;
  const int nsel = clamp_len(a.n_sel[unit], a.k);
  const int w0 = chunk * kAttnRows + wave * kWaveRows;  // first row of this wave
  const int wrows = max(0, min(kWaveRows, nsel - w0));
  uint32_t* stage = reinterpret_cast<uint32_t*>(lds) + wave * 16 * kStageRowDwords;
  float* ptab = lds + AttnLds<G>::kStage + wave * AttnLds<G>::kPTab;  // [16][G], [G]
  float* merge = lds + AttnLds<G>::kStage + AttnLds<G>::kP;
  float* part = a.part + ((int64_t)unit * a.chunks + chunk) * G * kPartStride;

  // Rows this lane loads (block blk, load it -> row 16*blk + 4*it + lrow of
  // the wave), as row numbers from the unit's base; the addresses are formed
  // at each load, so only 32-bit row numbers stay live.  Rows past wrows load
  // the wave's last row instead: every load is unconditional (lane-conditional
  // loads make the compiler wait for all outstanding loads at each use), and
  // those rows are masked out of the softmax.
  const int nblk = (wrows + 15) / 16;
  const int64_t stride = INDEXED ? a.row_stride : kD;
  const int64_t ubase = (INDEXED ? (int64_t)unit * a.max_ctx : (int64_t)unit * a.k) * stride +
                        8 * lchunk;
  int row[kBlocks][4];
  if (wrows > 0) {
#pragma unroll
    for (int blk = 0; blk < kBlocks; ++blk)
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int i = min(16 * blk + 4 * it + lrow, wrows - 1);
        int ps = INDEXED ? a.idx[(int64_t)unit * a.k + w0 + i] : w0 + i;
        if (INDEXED) ps = ps < 0 ? 0 : (ps >= a.max_ctx ? a.max_ctx - 1 : ps);
        row[blk][it] = ps;
      }
  }
  auto load_rows = [&](const uint16_t* base, int blk, uint4* dst) {
#pragma unroll
    for (int it = 0; it < 4; ++it) dst[it] = ld16(base + ubase + (int64_t)row[blk][it] * stride);
  };
  // K and V of one block each: the next block's K is requested once the
  // current K is staged, its V once the current V is consumed (loads return
  // in order, so each wait covers exactly the block it needs)
  uint4 kr[4], vr[4];
  if (nblk > 0) {
    load_rows(a.k_rows, 0, kr);
    load_rows(a.v_rows, 0, vr);
  }

  // the query rows go to LDS once, in the MFMA A placement, and are read
  // back at every block rather than held in registers
  uint32_t* qlds = reinterpret_cast<uint32_t*>(lds + AttnLds<G>::kStage + AttnLds<G>::kP +
                                               AttnLds<G>::kMerge);
  {
    // two tokens: rows [0, G/2) are the current token's heads, the rest the
    // speculative token's (same KV head)
    const int Gq = a.q2 ? G / 2 : G;
    for (int e = tid; e < 16 * (kD / 8); e += kAttnThreads) {
      const int r = e / (kD / 8), c = e - r * (kD / 8);
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (r < G) {
        const bool second = a.q2 && r >= Gq;
        v = ld16((second ? a.q2 : a.q) +
                 ((int64_t)b * a.Hq + (int64_t)h * Gq + (second ? r - Gq : r)) * kD + 8 * c);
      }
      *reinterpret_cast<uint4*>(qlds + r * kStageRowDwords + 4 * c) = v;
    }
    __syncthreads();
  }
  // online state: register i of lane group kg is head 4*kg + i
  float m_i[4], l_i[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m_i[i] = -INFINITY;
    l_i[i] = 0.f;
  }
  // weighted V sums: oacc[e][j] = O[head 4*kg + j][8*r16 + e]
  static_assert(G <= 16, "the heads fill at most the 16 rows of a product");
  f32x4 oacc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) oacc[e] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int blk = 0; blk < kBlocks; ++blk) {
    if (blk >= nblk) break;  // uniform over the wave
#pragma unroll
    for (int it = 0; it < 4; ++it)
      *reinterpret_cast<uint4*>(stage + (4 * it + lrow) * kStageRowDwords + 4 * lchunk) =
          kr[it];
    __builtin_amdgcn_wave_barrier();
    // the scheduler would otherwise hoist the next block's loads above this
    // block's work and hold both blocks in registers
    __builtin_amdgcn_sched_barrier(0);
    // unconditional (rows of blocks past nblk are the wave's last row): a
    // conditional load would become a branch that the compiler hoists
    if (blk + 1 < kBlocks) load_rows(a.k_rows, blk + 1, kr);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint4 kv = *reinterpret_cast<const uint4*>(
          stage + r16 * kStageRowDwords + 4 * (4 * t + kg));
      const uint4 qv = *reinterpret_cast<const uint4*>(
          qlds + r16 * kStageRowDwords + 4 * (4 * t + kg));
      acc = mfma_16x16x32(as_bf16x8(qv), as_bf16x8(kv), acc);
    }
    __builtin_amdgcn_wave_barrier();
    // logits of key r16 of the block for heads 4kg..4kg+3, block max and sum
    // (reductions over the 16 keys of a lane row stay in the row: DPP)
    const bool valid = 16 * blk + r16 < wrows;
    float p[4], al[4];
    bool moved = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lg = (4 * kg + i < G && valid) ? acc[i] * a.scale : -INFINITY;
      const float mn = fmaxf(m_i[i], row16_max(lg));
      moved |= mn != m_i[i];
      al[i] = m_i[i] == -INFINITY ? 0.f : __expf(m_i[i] - mn);
      p[i] = lg == -INFINITY ? 0.f : __expf(lg - mn);
      l_i[i] = l_i[i] * al[i] + row16_sum(p[i]);
      m_i[i] = mn;
    }
    // weights of the block's rows and the rescale factors -> per-wave table
    if (4 * kg < G) {
      if (G >= 4) {
        *reinterpret_cast<float4*>(ptab + r16 * G + 4 * kg) = make_float4(p[0], p[1], p[2], p[3]);
        if (r16 == 0)
          *reinterpret_cast<float4*>(ptab + 16 * G + 4 * kg) =
              make_float4(al[0], al[1], al[2], al[3]);
      } else {
#pragma unroll
        for (int i = 0; i < G; ++i) {
          ptab[r16 * G + i] = p[i];
          if (r16 == 0) ptab[16 * G + i] = al[i];
        }
      }
    }
    const bool rescale = __any(moved);  // running max moved for some head
    __builtin_amdgcn_wave_barrier();
    // rescale factors are lane-local: register j of lane group kg is head 4kg+j
    if (rescale) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int j = 0; j < 4; ++j) oacc[e][j] *= al[j];
    }
    // A operand: weights of head r16 at rows lrow + 4i (k = 8*lrow + 2i + s,
    // s = 0 hi part, 1 lo part), read back transposed from the table
    uint4 aw;
    {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = r16 < G ? ptab[(4 * i + lrow) * G + r16] : 0.f;
        const uint32_t hi = bf16_rne_bits(pv);
        const uint32_t lo = bf16_rne_bits(pv - __uint_as_float(hi << 16));
        w[i] = hi | (lo << 16);
      }
      aw = make_uint4(w[0], w[1], w[2], w[3]);
    }
    // B operand of product e: V[row lrow + 4i][8*lchunk + e], each entry twice
    const uint32_t* vw = reinterpret_cast<const uint32_t*>(vr);  // [row i][4 dwords]
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t x = vw[4 * i + (e >> 1)];
        b[i] = (e & 1) ? ((x >> 16) | (x & 0xffff0000u)) : ((x & 0xffffu) | (x << 16));
      }
      oacc[e] = mfma_16x16x32(as_bf16x8(aw), as_bf16x8(make_uint4(b[0], b[1], b[2], b[3])),
                              oacc[e]);
      __builtin_amdgcn_sched_barrier(0);  // one product's B operand live at a time
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (blk + 1 < kBlocks) load_rows(a.v_rows, blk + 1, vr);
  }
  // lane (kg, r16) holds O[4kg + j][8*r16 + e] in oacc[e][j]
  float* mw = merge + wave * G * (kD + 2);
  if (4 * kg < G) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int g = 4 * kg + j;
      if (g < G) {
#pragma unroll
        for (int e = 0; e < 8; ++e) mw[g * (kD + 2) + 8 * r16 + e] = oacc[e][j];
      }
    }
  }
  if (lchunk == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * lrow + i;
      if (g < G) {
        mw[g * (kD + 2) + kD] = m_i[i];
        mw[g * (kD + 2) + kD + 1] = l_i[i];
      }
    }
  }
  __syncthreads();
  // merge the four waves into the chunk's partial
  for (int oi = tid; oi < G * kD; oi += kAttnThreads) {
    const int g = oi / kD, c = oi - g * kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, merge[(w * G + g) * (kD + 2) + kD]);
    float O = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float* mg = merge + (w * G + g) * (kD + 2);
      const float wt = mg[kD] == -INFINITY ? 0.f : __expf(mg[kD] - M);
      O = fmaf(wt, mg[c], O);
      L = fmaf(wt, mg[kD + 1], L);
    }
    part[g * kPartStride + 4 + c] = O;
    if (c == 0) {
      part[g * kPartStride] = M;
      part[g * kPartStride + 1] = L;
    }
  }
}

}  // namespace ckv

namespace ckv {

// ---- attention by a whole selection workgroup --------------------------------
// After a kFinishThreads workgroup has selected a unit's set, its 16 waves
// attend over its share of it: `nrows` rows whose source positions are in
// LDS (pos[0..nrows)), read in place from the source at row stride
// a.row_stride.  Wave w takes a contiguous run of 16-row blocks.  Per block
// the wave's K and V rows go through its own LDS stages, so the registers
// they were loaded into are free at once and the next block's loads are
// issued before the current block's arithmetic: every wave keeps a block
// (8 KiB) in flight while holding at most 128 registers (16 waves per CU).
// Logits and the weighted V sum are the products of attn_chunk (query rows
// in the A placement, hi + lo bf16 weight parts); the 16 waves' states are
// merged through LDS into the workgroup's result: the normalised output when
// the unit has one share, else the share's partial (max, weight sum,
// weighted V sum) for k_combine.
template <int G>
struct WgAttnLds {
  static constexpr int kKStage = 16 * kStageRowDwords;  // dwords per wave: 16 padded rows
  static constexpr int kVStage = 16 * (kD / 2);         // dwords per wave: 16 rows of 256 B
  static constexpr int kPTab = 16 * G + G + (G < 4 ? 4 - G : 0);  // weight table floats
  static constexpr int kPerWave = kKStage + kVStage + kPTab;
  static constexpr int kStages = (kFinishThreads / 64) * kPerWave;  // dwords
  static constexpr int kQ = 16 * kStageRowDwords;       // query rows in the A placement
  static constexpr int kMerge = (kFinishThreads / 64) * G * (kD + 2);  // floats, in the stages
  static_assert(kMerge + 2 * G <= kStages, "the 16 waves' states and 2 local logits per head fit in the stages");
  static_assert(kPerWave % 4 == 0, "16-byte aligned stages");
};

// Output slots [lo, hi) of share `split` of `nsplit` over a set of m
// positions: equal runs of whole 16-row blocks.
__host__ __device__ __forceinline__ void share_range(int m, int split, int nsplit, int* lo,
                                                     int* hi) {
  const int per = (((m + nsplit - 1) / nsplit) + 15) & ~15;
  *lo = min(split * per, m);
  *hi = min(*lo + per, m);
}

// Row source of attn_wg: the share's positions in LDS.
struct LdsRows {
  const int32_t* pos;
  __device__ __forceinline__ int operator()(int i) const { return pos[i]; }
};

// All kFinishThreads threads call this.  stages: WgAttnLds<G>::kStages
// dwords, qlds: kQ dwords (both free on entry); pos(i): the source row of
// the share's row i, clamped to [0, a.max_ctx).  The workgroup attends with
// the G query heads qh0 .. qh0 + G - 1 of the unit's request (qh0 = h * G
// for a KV head's whole group).  With nloc > 0 (nsplit 1 only) the heads also
// see the nloc rows k_loc / v_loc ([nloc][d] bf16) beside the share's rows:
// the token's own rows in dual-token decoding (Sec. 5.2), which join the
// final merge as one more partial per head.  MERGE2 (nsplit 2, no local
// rows): the two shares' workgroups merge in the launch instead of k_combine.
// Share 0 stores its partial with device-coherent stores and, once they have
// completed, sets *mflag to tag; share 1 waits for the flag (bounded), clears
// it, and merges both partials into the output in k_combine's order of
// operations, so the outputs equal those of the two-launch form bit for bit.
template <int G, class Rows, bool MERGE2 = false>
__device__ __forceinline__ void attn_wg(const AttnArgs& a, int unit, Rows pos, int nrows,
                                        int split, int nsplit, uint32_t* stages,
                                        uint32_t* qlds, int qh0,
                                        const uint16_t* k_loc = nullptr,
                                        const uint16_t* v_loc = nullptr, int nloc = 0,
                                        uint64_t* mflag = nullptr, uint64_t tag = 0) {
  using Lds = WgAttnLds<G>;
  static_assert(G <= 8, "16 waves' states of at most 8 heads fit in the stages");
  constexpr int kW = kFinishThreads / 64;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int lrow = lane >> 4, lchunk = lane & 15;
  const int b = unit / a.Hkv;
  const int nblk = (nrows + 15) >> 4;
  const int blk0 = (wave * nblk) / kW, blk1 = ((wave + 1) * nblk) / kW;
  uint32_t* kst = stages + wave * Lds::kPerWave;
  uint32_t* vst = kst + Lds::kKStage;
  float* ptab = reinterpret_cast<float*>(vst + Lds::kVStage);
  const int64_t stride = a.row_stride;
  const int64_t ubase = (int64_t)unit * a.max_ctx * stride + 8 * lchunk;

  // the query rows first: their loads queue ahead of the first block's
  uint4 qv_ld = make_uint4(0u, 0u, 0u, 0u);
  const int qr = tid >> 4, qc = tid & 15;  // threads 0..255: row qr, 16-byte chunk qc
  if (tid < 16 * 16 && qr < G)
    qv_ld = ld16(a.q + ((int64_t)b * a.Hq + qh0 + qr) * kD + 8 * qc);
  // rows of block blk, clamped to the share (rows past nrows are masked)
  auto load_block = [&](int blk, uint4* kr, uint4* vr) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int i = min(16 * blk + 4 * it + lrow, nrows - 1);
      int p = pos(i);
      p = p < 0 ? 0 : (p >= a.max_ctx ? a.max_ctx - 1 : p);
      const int64_t off = ubase + (int64_t)p * stride;
      kr[it] = ld16(a.k_rows + off);
      vr[it] = ld16(a.v_rows + off);
    }
  };
  uint4 kr[4], vr[4];
  if (blk0 < blk1) load_block(blk0, kr, vr);
  if (tid < 16 * 16) *reinterpret_cast<uint4*>(qlds + qr * kStageRowDwords + 4 * qc) = qv_ld;
  lds_barrier();  // the query rows are in LDS; the first block may still be in flight

  float m_i[4], l_i[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m_i[i] = -INFINITY;
    l_i[i] = 0.f;
  }
  f32x4 oacc[8];  // oacc[e][j] = O[head 4*kg + j][8*r16 + e]
#pragma unroll
  for (int e = 0; e < 8; ++e) oacc[e] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int blk = blk0; blk < blk1; ++blk) {  // bounds uniform over the wave
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      *reinterpret_cast<uint4*>(kst + (4 * it + lrow) * kStageRowDwords + 4 * lchunk) = kr[it];
      *reinterpret_cast<uint4*>(vst + (4 * it + lrow) * (kD / 2) + 4 * lchunk) = vr[it];
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (blk + 1 < blk1) load_block(blk + 1, kr, vr);
    __builtin_amdgcn_sched_barrier(0);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint4 kv = *reinterpret_cast<const uint4*>(kst + r16 * kStageRowDwords + 4 * (4 * t + kg));
      const uint4 qv = *reinterpret_cast<const uint4*>(qlds + r16 * kStageRowDwords + 4 * (4 * t + kg));
      acc = mfma_16x16x32(as_bf16x8(qv), as_bf16x8(kv), acc);
    }
    const bool valid = 16 * blk + r16 < nrows;
    float p[4], al[4];
    bool moved = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lg = (4 * kg + i < G && valid) ? acc[i] * a.scale : -INFINITY;
      const float mn = fmaxf(m_i[i], row16_max(lg));
      moved |= mn != m_i[i];
      al[i] = m_i[i] == -INFINITY ? 0.f : __expf(m_i[i] - mn);
      p[i] = lg == -INFINITY ? 0.f : __expf(lg - mn);
      l_i[i] = l_i[i] * al[i] + row16_sum(p[i]);
      m_i[i] = mn;
    }
    if (4 * kg < G) {
      if (G >= 4) {
        *reinterpret_cast<float4*>(ptab + r16 * G + 4 * kg) = make_float4(p[0], p[1], p[2], p[3]);
      } else {
#pragma unroll
        for (int i = 0; i < G; ++i) ptab[r16 * G + i] = p[i];
      }
    }
    const bool rescale = __any(moved);
    __builtin_amdgcn_wave_barrier();
    if (rescale) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int j = 0; j < 4; ++j) oacc[e][j] *= al[j];
    }
    uint4 aw;
    {
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = r16 < G ? ptab[(4 * i + lrow) * G + r16] : 0.f;
        const uint32_t hi = bf16_rne_bits(pv);
        const uint32_t lo = bf16_rne_bits(pv - __uint_as_float(hi << 16));
        w[i] = hi | (lo << 16);
      }
      aw = make_uint4(w[0], w[1], w[2], w[3]);
    }
    // this lane's own V rows back from the stage: channels [8*lchunk, +8) of
    // rows lrow + 4i, the B operand of product e up to duplication
    uint4 vv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vv[i] = *reinterpret_cast<const uint4*>(vst + (4 * i + lrow) * (kD / 2) + 4 * lchunk);
    const uint32_t* vw = reinterpret_cast<const uint32_t*>(vv);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t bb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t x = vw[4 * i + (e >> 1)];
        bb[i] = (e & 1) ? ((x >> 16) | (x & 0xffff0000u)) : ((x & 0xffffu) | (x << 16));
      }
      oacc[e] = mfma_16x16x32(as_bf16x8(aw), as_bf16x8(make_uint4(bb[0], bb[1], bb[2], bb[3])),
                              oacc[e]);
    }
    __builtin_amdgcn_wave_barrier();
  }

  // merge the 16 waves (their stages are free once every wave is here)
  __syncthreads();
  float* merge = reinterpret_cast<float*>(stages);
  float* mw = merge + wave * G * (kD + 2);
  if (4 * kg < G) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int g = 4 * kg + j;
      if (g < G) {
#pragma unroll
        for (int e = 0; e < 8; ++e) mw[g * (kD + 2) + 8 * r16 + e] = oacc[e][j];
      }
    }
  }
  if (lchunk == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = 4 * lrow + i;
      if (g < G) {
        mw[g * (kD + 2) + kD] = m_i[i];
        mw[g * (kD + 2) + kD + 1] = l_i[i];
      }
    }
  }
  // logits of the local rows, one wave per (head, row): lane l takes
  // channels 2l and 2l + 1
  float* loc = merge + kW * G * (kD + 2);  // [G][2]
  if (wave < G * nloc) {  // uniform over the wave
    const int g = wave / nloc, j = wave - g * nloc;
    const uint32_t qw = qlds[g * kStageRowDwords + lane];
    const uint32_t kw = reinterpret_cast<const uint32_t*>(k_loc + j * kD)[lane];
    float dot = __uint_as_float(qw << 16) * __uint_as_float(kw << 16);
    dot = fmaf(__uint_as_float(qw & 0xffff0000u), __uint_as_float(kw & 0xffff0000u), dot);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) dot += __shfl_xor(dot, o);
    if (lane == 0) loc[g * 2 + j] = dot * a.scale;
  }
  __syncthreads();
  float mine[3];  // MERGE2, share 1: this thread's (M, L, O)
  for (int oi = tid; oi < G * kD; oi += kFinishThreads) {
    const int g = oi / kD, c = oi - g * kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kW; ++w) M = fmaxf(M, merge[(w * G + g) * (kD + 2) + kD]);
    for (int j = 0; j < nloc; ++j) M = fmaxf(M, loc[g * 2 + j]);
    float O = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
      const float* mg = merge + (w * G + g) * (kD + 2);
      const float wt = mg[kD] == -INFINITY ? 0.f : __expf(mg[kD] - M);
      O = fmaf(wt, mg[c], O);
      L = fmaf(wt, mg[kD + 1], L);
    }
    for (int j = 0; j < nloc; ++j) {
      const float wt = __expf(loc[g * 2 + j] - M);
      O = fmaf(wt, __uint_as_float((uint32_t)v_loc[j * kD + c] << 16), O);
      L += wt;
    }
    if constexpr (MERGE2) {
      float* part = a.part + (((int64_t)unit * 2) * G + g) * kPartStride;  // share 0's
      if (split == 0) {
        __hip_atomic_store(part + 4 + c, O, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (c == 0) {
          __hip_atomic_store(part, M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(part + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      } else {
        mine[0] = M;
        mine[1] = L;
        mine[2] = O;
      }
    } else if (nsplit == 1) {
      a.out[((int64_t)b * a.Hq + qh0 + g) * kD + c] = L > 0.f ? O / L : 0.f;
    } else {
      float* part = a.part + (((int64_t)unit * nsplit + split) * G + g) * kPartStride;
      part[4 + c] = O;
      if (c == 0) {
        part[0] = M;
        part[1] = L;
      }
    }
  }
  if constexpr (MERGE2) {
    static_assert(G * kD <= kFinishThreads, "one output per thread");
    if (split == 0) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (tid == 0) __hip_atomic_store(mflag, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    if (tid == 0) {
      for (uint32_t spin = 0;
           __hip_atomic_load(mflag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != tag &&
           spin < kFusedSpinLimit;
           ++spin)
        __builtin_amdgcn_s_sleep(2);
      __hip_atomic_store(mflag, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (tid < G * kD) {
      const int g = tid / kD, c = tid - g * kD;
      const float* p0 = a.part + (((int64_t)unit * 2) * G + g) * kPartStride;
      const float m0 = __hip_atomic_load(p0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const float l0 = __hip_atomic_load(p0 + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const float o0 = __hip_atomic_load(p0 + 4 + c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      // k_combine with two chunks and no local rows, step by step
      float M = fmaxf(-INFINITY, -INFINITY);
      M = fmaxf(M, m0);
      M = fmaxf(M, mine[0]);
      const float w0 = m0 == -INFINITY ? 0.f : __expf(m0 - M);
      float L = fmaf(w0, l0, 0.f);
      const float w1 = mine[0] == -INFINITY ? 0.f : __expf(mine[0] - M);
      L = fmaf(w1, mine[1], L);
      L += 0.f;
      L += 0.f;
      const float inv = L > 0.f ? 1.f / L : 0.f;
      float O = 0.f;
      O = fmaf(w0, o0, O);
      O = fmaf(w1, mine[2], O);
      a.out[((int64_t)b * a.Hq + qh0 + g) * kD + c] = O * inv;
    }
  }
}

}  // namespace ckv
