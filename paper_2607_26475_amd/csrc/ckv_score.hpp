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
// supplies channels [32t + 8kg, 32t + 8kg + 8) of step t.  The accumulator of
// lane l then holds heads 4kg..4kg+3 of key (l % 16).
#pragma once

#include "ckv_device.hpp"

namespace ckv {

// Adds the workgroup's LDS histogram into the unit's global fine and coarse
// histograms (NT threads, kHistBins bins, kBinsPerThread each).
template <int NT = kScoreThreads>
__device__ __forceinline__ void flush_hist(const uint32_t* lds_hist,
                                           uint32_t* g_hist,
                                           uint32_t* g_coarse) {
  constexpr int kBinsPerThread = kHistBins / NT;
  constexpr int kThreadsPerCoarse = kHistBins / kCoarseBins / kBinsPerThread;
  const int t = threadIdx.x;
  uint32_t csum = 0;
#pragma unroll
  for (int i = 0; i < kBinsPerThread; ++i) {
    const uint32_t v = lds_hist[kBinsPerThread * t + i];
    if (v) {
      atomicAdd(&g_hist[kBinsPerThread * t + i], v);
      csum += v;
    }
  }
#pragma unroll
  for (int o = 1; o < kThreadsPerCoarse; o <<= 1) csum += __shfl_xor(csum, o);
  if ((t % kThreadsPerCoarse) == 0 && csum) atomicAdd(&g_coarse[t / kThreadsPerCoarse], csum);
}

// Stores the workgroup's LDS histogram as its slot (NT threads).
template <int NT = kScoreThreads>
__device__ __forceinline__ void store_hist(const uint32_t* lds_hist, uint32_t* slot) {
  constexpr int kPer = kHistBins / NT;
  static_assert(kPer % 4 == 0, "16-byte stores");
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < kPer; i += 4)
    *reinterpret_cast<uint4*>(slot + kPer * t + i) =
        *reinterpret_cast<const uint4*>(lds_hist + kPer * t + i);
}

// An empty slot, for a workgroup whose groups of the unit all lie past n_b.
template <int NT = kScoreThreads>
__device__ __forceinline__ void store_zero_hist(uint32_t* slot) {
  for (int i = 4 * (int)threadIdx.x; i < kHistBins; i += 4 * NT)
    *reinterpret_cast<uint4*>(slot + i) = make_uint4(0u, 0u, 0u, 0u);
}

// The workgroup's LDS histogram (or zeros, lds_hist null) as its slot,
// device-coherent, 8 bytes per lane with consecutive lanes on consecutive
// words (NT threads).
template <int NT>
__device__ __forceinline__ void store_hist_coherent(const uint32_t* lds_hist, uint32_t* slot) {
  constexpr int kPairs = kHistBins / NT / 2;
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < kPairs; ++q) {
    const int i = 2 * (t + NT * q);
    const uint64_t w = lds_hist ? ((uint64_t)lds_hist[i] | ((uint64_t)lds_hist[i + 1] << 32))
                                : 0ull;
    __hip_atomic_store(reinterpret_cast<uint64_t*>(slot + i), w, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
}

// After a fused scoring workgroup's stores of the consecutive slots [slot0,
// slot0 + count): every thread waits for its own stores, the barrier then
// covers the workgroup's, and each slot's two flags take the launch's tag.
__device__ __forceinline__ void hand_over(const FusedSync& fs, int64_t slot0, int count) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int t = threadIdx.x; t < 2 * count; t += blockDim.x)
    __hip_atomic_store(fs.flags + 2 * slot0 + t, fs.tag, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Scores of one staged group (kStageRows keys of one unit starting at row
// jb) into out[0, kStageRows): the MFMA products with the G query rows, the
// maximum over the heads, the scale; rows at or past n get -inf and are not
// counted.  If HIST, counts the first radix digit of the others in lds_hist.
template <int G, bool HIST>
__device__ __forceinline__ void score_group(const uint32_t* stage, const bf16x8* qa, int jb,
                                            int n, float scale, uint32_t* lds_hist,
                                            float* out) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, kg = lane >> 4;
#pragma unroll
  for (int u = 0; u < kStageRows / 16; ++u) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint4 kv = *reinterpret_cast<const uint4*>(
          stage + (16 * u + r16) * kStageRowDwords + 4 * (4 * t + kg));
      acc = mfma_16x16x32(qa[t], as_bf16x8(kv), acc);
    }
    float sc = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (4 * kg + i < G) sc = fmaxf(sc, acc[i]);
    if (G > 4) sc = fmaxf(sc, __shfl_xor(sc, 16));
    if (G > 8) sc = fmaxf(sc, __shfl_xor(sc, 32));
    sc *= scale;
    const int j = jb + 16 * u + lane;
    if (lane < 16) {
      if (j < n) {
        if (HIST) atomicAdd(&lds_hist[order_key(sc) >> (32 - kHistBits)], 1u);
      } else {
        sc = -INFINITY;
      }
      out[16 * u + lane] = sc;
    }
  }
}

// The G query rows of a unit as MFMA A operands (rows past G are zero).
template <int G>
__device__ __forceinline__ void load_query(const ScoreArgs& a, int unit, bf16x8* qa) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, kg = lane >> 4;
  const int b = unit / a.Hkv, h = unit - b * a.Hkv;
  const uint16_t* qrow = a.q + ((int64_t)b * a.Hq + (int64_t)h * G + r16) * kD + 8 * kg;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (r16 < G) v = ld16(qrow + 32 * t);
    qa[t] = as_bf16x8(v);
  }
}

// Scores a balanced share of the whole batch: the positions of every unit are
// cut into groups of kStageRows keys, the groups of all units are numbered
// unit-major, and workgroup `wg` of `nwg` takes the contiguous range
// [wg*T/nwg, (wg+1)*T/nwg) of the T groups.  A range spans few units; for each
// unit it touches the workgroup loads that unit's G query rows once and, if
// HIST, counts the first radix digit of its scores in LDS and, when it leaves
// the unit, adds the counts to the unit's histogram or stores them as its own
// slot (hist_part; an all-zero slot when its groups of the unit all lie at or
// past n_b).  Groups at or beyond n_b only write -inf.  Must be called by all
// 64 * NW threads of the workgroup; lds_stage holds NW * (kStageDwords +
// kFlushGroups * kStageRows) dwords.
//
// Memory path: the NW waves take the range's groups round-robin (wave w the
// groups w, w + NW, ...), so that the workgroup streams one region at a
// time: with a contiguous quarter per wave the scan ran 5 % slower (four
// times as many regions in flight over the device).  A wave reads each group
// with fully coalesced 16-byte loads (one instruction = 4 whole 256-byte
// rows), writes it to a private, padded LDS stage and reads it back in the
// MFMA operand placement while the loads of its next group are in flight.
// Loading the operand placement straight from HBM (16 rows x 64 bytes per
// instruction) costs about a tenth of the achievable bandwidth.
//
// Scores are collected in a per-wave LDS buffer and written out every
// kFlushGroups groups, one 128-byte line per group (for a Llama-8B-sized
// batch that is once, at the end of the range).  A global store pending in the loop
// would make every wait for the current group also wait for the prefetched
// one (loads and stores share one counter), and score writes interleaved
// with the key stream cost bandwidth even in large batches: about 10 % at
// every 16 groups against 2 % when written once.
//
// HALVES: a wave requests the next group in two halves, the second once the
// first has landed (after scoring the current group), so that it has 4 KiB
// rather than 8 KiB in flight.  That suits the scoring role of the one-launch
// attend-and-score kernels, which share the memory system with the
// attention's random row reads: 186-188 against 189-192 us per Llama-8B
// layer, alternated over two sessions.  The 8-wave histogram pass is slower with it (167-170 against
// 158-165 us), as it is with 16-row groups.
//
// FUSED (the scoring role of the one-launch same-step kernel, HIST with
// per-workgroup slots): the ranges are XCD-affine (xcd_slot0); the workgroup
// may have more than NW waves, the others only join its barriers; scores and
// slots are stored device-coherent, 8 bytes per lane over whole lines, and
// each finished (unit, slot) is handed over through fs (FusedSync).
template <int G, bool HIST, int NW = 4, bool HALVES = false, bool FUSED = false>
__device__ __forceinline__ void score_range(const ScoreArgs& a, int wg, int nwg,
                                            uint32_t* lds_hist,
                                            uint32_t* lds_stage, FusedSync fs = FusedSync{}) {
  static_assert(!FUSED || (HIST && !HALVES), "the fused scoring role counts histograms");
  constexpr int NT = 64 * NW;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lrow = lane >> 4, lchunk = lane & 15;
  const bool active = !FUSED || wave < NW;  // uniform over the wave
  constexpr int kLoads = kStageRows / 4;  // 4 rows per load instruction
  const int64_t gpu_groups = (a.max_ctx + kStageRows - 1) / kStageRows;  // per unit
  // FUSED: XCD x = wg % 8 scores units x, x + 8, ... with its nwg / 8 workgroups
  const int xcd = FUSED ? (wg & 7) : 0;
  const int wr = FUSED ? (wg >> 3) : wg, nwr = FUSED ? (nwg >> 3) : nwg;
  const int64_t units_r = FUSED ? (a.units >> 3) : a.units;
  const int64_t total = units_r * gpu_groups;
  const int64_t g0 = total * wr / nwr, g1 = total * (wr + 1) / nwr;
  uint32_t* stage = lds_stage + (active ? wave : 0) * kStageDwords;
  float* sbuf = reinterpret_cast<float*>(lds_stage + NW * kStageDwords) +
                (active ? wave : 0) * kFlushGroups * kStageRows;

  for (int64_t seg = g0; seg < g1;) {
    const int vunit = (int)(seg / gpu_groups);
    const int unit = FUSED ? 8 * vunit + xcd : vunit;
    const int64_t slot = FUSED ? xcd * (units_r + nwr) + vunit + wr : (int64_t)unit + wg;
    const int64_t ubase = (int64_t)vunit * gpu_groups;
    const int64_t seg_end = min(g1, ubase + gpu_groups);
    const int n = unit_len(a.ctx_lens[unit / a.Hkv], a.max_ctx, a.chunk);
    float* srow = a.scores + (int64_t)unit * a.max_ctx;
    // groups [ubase + first_empty, ...) hold no position below n_b
    const int64_t valid_end = min(seg_end, ubase + (n + kStageRows - 1) / kStageRows);
    for (int64_t gg = max(seg, valid_end); gg < seg_end; ++gg) {
      const int j = (int)(gg - ubase) * kStageRows + (tid & (kStageRows - 1));
      if (tid < kStageRows && j < a.max_ctx) srow[j] = -INFINITY;
    }
    if (seg < valid_end) {  // uniform over the workgroup
      if (HIST) {
        if (!FUSED || tid < NT)
          for (int i = tid; i < kHistBins; i += NT) lds_hist[i] = 0u;
        __syncthreads();
      }
      bf16x8 qa[4];
      load_query<G>(a, unit, qa);
      const uint16_t* kunit = a.keys + (int64_t)unit * a.max_ctx * a.key_stride;
      // Rows at or past n_b load row n_b - 1 instead (their scores are
      // replaced by -inf): lane-conditional loads would make the compiler
      // wait for every outstanding load at each use.
      // loads [i0, i1) of a group's kLoads
      auto load_part = [&](int64_t gg, uint4* v, int i0, int i1) {
        const int jb = (int)(gg - ubase) * kStageRows;
#pragma unroll
        for (int i = i0; i < i1; ++i) {
          const int j = min(jb + 4 * i + lrow, n - 1);
          v[i] = ld16_nt(kunit + (int64_t)j * a.key_stride + 8 * lchunk);
        }
      };
      auto load_group = [&](int64_t gg, uint4* v) { load_part(gg, v, 0, kLoads); };
      // writes the scores of the nb buffered groups [first, first + nb): one
      // contiguous run, 16 bytes per lane when rows are 16-byte aligned
      auto flush = [&](int64_t first, int nb) {
        __builtin_amdgcn_wave_barrier();
        const int jb = (int)(first - ubase) * kStageRows;
        const int count = nb * kStageRows;
        if constexpr (FUSED) {
          // 8 bytes per lane, consecutive lanes on consecutive pairs: each
          // instruction covers whole 128-byte lines of four groups
          for (int c = 2 * lane; c < count; c += 128) {
            const int j = jb + (c / kStageRows) * NW * kStageRows + c % kStageRows;
            const float2 v = *reinterpret_cast<const float2*>(sbuf + c);
            if ((a.max_ctx & 1) == 0 && j + 1 < a.max_ctx) {
              const uint64_t w = (uint64_t)__float_as_uint(v.x) |
                                 ((uint64_t)__float_as_uint(v.y) << 32);
              __hip_atomic_store(reinterpret_cast<uint64_t*>(srow + j), w, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
            } else {
              if (j < a.max_ctx)
                __hip_atomic_store(srow + j, v.x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              if (j + 1 < a.max_ctx)
                __hip_atomic_store(srow + j + 1, v.y, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
          }
        } else if ((a.max_ctx & 3) == 0) {
          for (int c = 4 * lane; c < count; c += 256) {
            const float4 v = *reinterpret_cast<const float4*>(sbuf + c);
            const int j = jb + (c / kStageRows) * NW * kStageRows + c % kStageRows;
            if (j + 3 < a.max_ctx) {
              *reinterpret_cast<float4*>(srow + j) = v;
            } else {
              if (j < a.max_ctx) srow[j] = v.x;
              if (j + 1 < a.max_ctx) srow[j + 1] = v.y;
              if (j + 2 < a.max_ctx) srow[j + 2] = v.z;
            }
          }
        } else {
          for (int c = lane; c < count; c += 64) {
            const int j = jb + (c / kStageRows) * NW * kStageRows + c % kStageRows;
            if (j < a.max_ctx) srow[j] = sbuf[c];
          }
        }
        __builtin_amdgcn_wave_barrier();
      };
      // this wave's groups of the segment below n_b: every NW-th one (none
      // for the waves past NW of the fused role)
      const int64_t w1 = valid_end, w0 = active ? seg + wave : w1;
      uint4 cur[kLoads], nxt[kLoads];
      int64_t gg = w0;
      int64_t first = gg;
      int nb = 0;
      if (gg < w1) load_group(gg, cur);
#pragma unroll 1
      for (; gg < w1; gg += NW) {
#pragma unroll
        for (int i = 0; i < kLoads; ++i)
          *reinterpret_cast<uint4*>(stage + (4 * i + lrow) * kStageRowDwords + 4 * lchunk) =
              cur[i];
        const bool more = gg + NW < w1;
        if (more) load_part(gg + NW, nxt, 0, HALVES ? kLoads / 2 : kLoads);
        __builtin_amdgcn_wave_barrier();
        score_group<G, HIST>(stage, qa, (int)(gg - ubase) * kStageRows, n, a.scale, lds_hist,
                             sbuf + nb * kStageRows);
        if (HALVES && more) {
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          load_part(gg + NW, nxt, kLoads / 2, kLoads);
        }
        if (++nb == kFlushGroups) {
          flush(first, nb);
          first = gg + NW;
          nb = 0;
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int i = 0; i < kLoads; ++i) cur[i] = nxt[i];
      }
      if (nb) flush(first, nb);
      if (HIST) {
        __syncthreads();
        if constexpr (FUSED) {
          if (tid < NT) store_hist_coherent<NT>(lds_hist, a.hist_part + slot * kHistBins);
        } else if (a.hist_part) {
          store_hist<NT>(lds_hist, a.hist_part + slot * kHistBins);
        } else {
          flush_hist<NT>(lds_hist, a.hist + (int64_t)unit * kHistBins,
                         a.coarse + (int64_t)unit * kCoarseBins);
        }
        __syncthreads();
      }
    } else if (HIST && a.hist_part) {  // the unit's histogram sums this slot too
      if constexpr (FUSED) {
        if (tid < NT) store_hist_coherent<NT>(nullptr, a.hist_part + slot * kHistBins);
      } else {
        store_zero_hist<NT>(a.hist_part + slot * kHistBins);
      }
    }
    seg = seg_end;
  }
  if constexpr (FUSED) {
    // every slot of the range handed over at its end, after one wait for all
    // its stores (a wait between units would stall the key stream)
    if (g0 < g1) {
      const int v0 = (int)(g0 / gpu_groups), v1 = (int)((g1 - 1) / gpu_groups);
      hand_over(fs, xcd * (units_r + nwr) + v0 + wr, v1 - v0 + 1);
    }
  }
}

// The same pass with dynamic work distribution, for the added histograms
// of the pipelined attend-and-score launch (a.claim set, a.hist_part null).
// The groups of each unit are cut into claims of kClaimGroups; workgroups
// take claims in increasing order from the counter a.claim, so a workgroup
// on a CU slowed by other work (the zero-copy gather running beside the
// pass) takes fewer of them and the pass is not held up by its slowest CUs.
// Within a claim the four waves take its groups round-robin as above.
//
// Thread 0 takes claims two ahead of the one being scored, at the start of
// each claim, and passes them through a two-entry LDS ring (one barrier per
// claim), so each wave knows the next claim while it scores the current one
// and prefetches that claim's first group across the boundary.  A
// workgroup thus holds up to two claims it has not started, which leaves
// workgroups idle at the end unless there are several claims per workgroup:
// the host uses claims from four per workgroup.  (Taking the next claim
// later, two rounds before the current claim's end, made the
// million-token loop's gather beside the pass slower.)  Each workgroup takes
// exactly one claim at or past the total; those take values total ..
// total + nwg - 1, and the workgroup that gets the last one resets the
// counter, so it is zero again when the launch ends.  A wave's scores stay
// in its LDS buffer for up to kFlushGroups / (kClaimGroups / 4) claims
// before one flush writes them, each claim's groups to its own unit's row.
// The LDS histogram counts one unit at a time and is added to that unit's
// histogram when the workgroup's claims move to another unit (claims
// increase, so once per unit) and at the end.  lds_claim: two words.  Must
// be called by all kScoreThreads threads.
template <int G>
__device__ __forceinline__ void score_claims(const ScoreArgs& a, int nwg, uint32_t* lds_hist,
                                             uint32_t* lds_stage, uint32_t* lds_claim) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lrow = lane >> 4, lchunk = lane & 15;
  constexpr int kLoads = kStageRows / 4;
  constexpr int kPerWave = kClaimGroups / 4;       // a wave's groups of one claim
  constexpr int kRecs = kFlushGroups / kPerWave;   // claims per score flush
  static_assert(kClaimGroups % 4 == 0 && kFlushGroups % kPerWave == 0, "claim layout");
  const int gpu_groups = (a.max_ctx + kStageRows - 1) / kStageRows;  // per unit
  const int cpu = (gpu_groups + kClaimGroups - 1) / kClaimGroups;     // claims per unit
  const uint32_t total = (uint32_t)a.units * (uint32_t)cpu;
  uint32_t* stage = lds_stage + wave * kStageDwords;
  float* sbuf = reinterpret_cast<float*>(lds_stage + 4 * kStageDwords) +
                wave * kFlushGroups * kStageRows;

  // thread 0: a new claim; the one that makes the counter reach total + nwg
  // is the last of the launch and resets it
  auto take = [&]() -> uint32_t {
    const uint32_t c = atomicAdd(a.claim, 1u);
    if (c == total + (uint32_t)nwg - 1u) atomicExch(a.claim, 0u);
    return c;
  };
  // a claim's unit, valid length, and groups [g0, g1) of which [g0, v1) lie below n_b
  struct Geo {
    int unit, n, g0, g1, v1;
  };
  auto geo = [&](uint32_t c) {
    Geo r;
    r.unit = (int)(c / (uint32_t)cpu);
    r.g0 = (int)(c - (uint32_t)r.unit * (uint32_t)cpu) * kClaimGroups;
    r.g1 = min(r.g0 + kClaimGroups, gpu_groups);
    r.n = unit_len(a.ctx_lens[r.unit / a.Hkv], a.max_ctx, a.chunk);
    r.v1 = max(r.g0, min(r.g1, (r.n + kStageRows - 1) / kStageRows));
    return r;
  };
  auto load_group = [&](const Geo& c, int g, uint4* v) {
    const uint16_t* kunit = a.keys + (int64_t)c.unit * a.max_ctx * a.key_stride;
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int j = min(g * kStageRows + 4 * i + lrow, c.n - 1);
      v[i] = ld16_nt(kunit + (int64_t)j * a.key_stride + 8 * lchunk);
    }
  };

  // buffered claims of this wave: unit, first group, groups scored
  int rec_unit[kRecs], rec_g0[kRecs], rec_nr[kRecs];
  int nrec = 0;
  auto flush = [&]() {
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int q = 0; q < kRecs; ++q) {
      if (q < nrec) {
        float* srow = a.scores + (int64_t)rec_unit[q] * a.max_ctx;
        const float* src = sbuf + q * kPerWave * kStageRows;
        const int count = rec_nr[q] * kStageRows;
        if ((a.max_ctx & 3) == 0) {
          for (int c = 4 * lane; c < count; c += 256) {
            const float4 v = *reinterpret_cast<const float4*>(src + c);
            const int j = (rec_g0[q] + wave + 4 * (c / kStageRows)) * kStageRows + c % kStageRows;
            if (j + 3 < a.max_ctx) {
              *reinterpret_cast<float4*>(srow + j) = v;
            } else {
              if (j < a.max_ctx) srow[j] = v.x;
              if (j + 1 < a.max_ctx) srow[j + 1] = v.y;
              if (j + 2 < a.max_ctx) srow[j + 2] = v.z;
            }
          }
        } else {
          for (int c = lane; c < count; c += 64) {
            const int j = (rec_g0[q] + wave + 4 * (c / kStageRows)) * kStageRows + c % kStageRows;
            if (j < a.max_ctx) srow[j] = src[c];
          }
        }
      }
    }
    nrec = 0;
    __builtin_amdgcn_wave_barrier();
  };

  if (tid == 0) {  // claims 0 and 1
    const uint32_t c0 = take();
    lds_claim[0] = c0;
    lds_claim[1] = c0 < total ? take() : c0;
  }
  __syncthreads();
  uint32_t cur = lds_claim[0], nxt = lds_claim[1];
  int cur_unit = -1;
  bf16x8 qa[4];
  uint4 cbuf[kLoads], nbuf[kLoads];
  bool have = false;  // cbuf holds this wave's first group of the current claim
#pragma unroll 1
  for (int i = 0; cur < total; ++i) {  // cur is uniform over the workgroup
    const Geo c = geo(cur);
    uint32_t ahead = 0;  // claim i + 2 (none once a claim has failed)
    if (tid == 0) ahead = nxt < total ? take() : nxt;
    if (c.unit != cur_unit) {
      if (cur_unit >= 0) {
        __syncthreads();
        flush_hist(lds_hist, a.hist + (int64_t)cur_unit * kHistBins,
                   a.coarse + (int64_t)cur_unit * kCoarseBins);
        __syncthreads();
      }
      for (int t = tid; t < kHistBins; t += kScoreThreads) lds_hist[t] = 0u;
      __syncthreads();
      load_query<G>(a, c.unit, qa);
      cur_unit = c.unit;
    }
    // groups of the claim at or past n_b hold -inf only
    for (int g = c.v1; g < c.g1; ++g) {
      const int j = g * kStageRows + (tid & (kStageRows - 1));
      if (tid < kStageRows && j < a.max_ctx)
        a.scores[(int64_t)c.unit * a.max_ctx + j] = -INFINITY;
    }
    const int w0 = c.g0 + wave;
    if (!have && w0 < c.v1) load_group(c, w0, cbuf);
    have = false;
    int r = 0;
#pragma unroll 1
    for (int g = w0; g < c.v1; g += 4, ++r) {
#pragma unroll
      for (int k = 0; k < kLoads; ++k)
        *reinterpret_cast<uint4*>(stage + (4 * k + lrow) * kStageRowDwords + 4 * lchunk) =
            cbuf[k];
      bool pf = false;
      if (g + 4 < c.v1) {
        load_group(c, g + 4, nbuf);
        pf = true;
      } else if (nxt < total) {  // the wave's last group: prefetch across the claim
        const Geo d = geo(nxt);
        if (d.g0 + wave < d.v1) {
          load_group(d, d.g0 + wave, nbuf);
          pf = true;
          have = true;
        }
      }
      __builtin_amdgcn_wave_barrier();
      score_group<G, true>(stage, qa, g * kStageRows, c.n, a.scale, lds_hist,
                           sbuf + (nrec * kPerWave + r) * kStageRows);
      __builtin_amdgcn_wave_barrier();
      if (pf) {
#pragma unroll
        for (int k = 0; k < kLoads; ++k) cbuf[k] = nbuf[k];
      }
    }
    if (r) {
#pragma unroll
      for (int q = 0; q < kRecs; ++q)
        if (q == nrec) {
          rec_unit[q] = c.unit;
          rec_g0[q] = c.g0;
          rec_nr[q] = r;
        }
      if (++nrec == kRecs) flush();
    }
    if (tid == 0) lds_claim[i & 1] = ahead;
    __syncthreads();  // publishes claim i + 2
    cur = nxt;
    nxt = lds_claim[i & 1];
  }
  if (nrec) flush();
  if (cur_unit >= 0) {
    __syncthreads();
    flush_hist(lds_hist, a.hist + (int64_t)cur_unit * kHistBins,
               a.coarse + (int64_t)cur_unit * kCoarseBins);
  }
}

}  // namespace ckv
