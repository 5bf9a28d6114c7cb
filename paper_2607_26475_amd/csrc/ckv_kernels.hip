// ckv_kernels.hip -- gfx950 kernels of libckv and their host-side launchers.
#include "ckv_attn.hpp"
#include "ckv_launch.hpp"
#include "ckv_profile.hpp"
#include "ckv_score.hpp"
#include "ckv_topk.hpp"

#include <algorithm>
#include <mutex>

namespace ckv {

constexpr int kMaxDevices = 256;  // devices the per-device host tables serve

// ---- workspace clearing (a kernel, not hipMemsetAsync: safe to capture) ----
__global__ __launch_bounds__(256) void k_zero(uint4* p, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// Fills p with a 32-bit pattern (the pipeline's poison of released buffers).
__global__ __launch_bounds__(256) void k_fill(uint4* p, int64_t n16, uint32_t pattern) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(pattern, pattern, pattern, pattern);
}

// ---- scoring -------------------------------------------------------------
// The pass with histograms runs as one workgroup of kHistScoreWaves waves per
// CU (its LDS allows one): half as many concurrent streams of keys as two
// four-wave workgroups, with the same loads in flight per CU, and so fewer
// histogram slots per unit.  Measured on the Llama-8B layer in one session:
// 159.7-163.9 us against 166.0-167.4 us; without histograms it gained nothing.
template <int G, bool HIST>
__global__ __launch_bounds__(HIST ? 64 * kHistScoreWaves : kScoreThreads) void k_score(ScoreArgs a) {
  constexpr int kWaves = HIST ? kHistScoreWaves : kScoreThreads / 64;
  __shared__ uint32_t lds_hist[HIST ? kHistBins : 1];
  __shared__ __attribute__((aligned(16)))
  uint32_t lds_stage[kWaves * (kStageDwords + kFlushGroups * kStageRows)];
  score_range<G, HIST, kWaves>(a, blockIdx.x, gridDim.x, lds_hist, lds_stage);
}


// The same pass over chunk landmarks (a kernel of its own only so that
// traces and profiles keep the two workloads apart).
template <int G>
__global__ __launch_bounds__(kScoreThreads) void k_score_chunks(ScoreArgs a) {
  __shared__ uint32_t lds_hist[kHistBins];
  __shared__ __attribute__((aligned(16))) uint32_t lds_stage[kScoreLdsDwords];
  score_range<G, true>(a, blockIdx.x, gridDim.x, lds_hist, lds_stage);
}

// ---- selection -----------------------------------------------------------
// First-digit histogram of given scores (standalone selection entry).
__global__ __launch_bounds__(kScoreThreads) void k_hist(SelectArgs a) {
  __shared__ uint32_t lds_hist[kHistBins];
  const int unit = blockIdx.x / a.tiles;
  const int tile = blockIdx.x - unit * a.tiles;
  const int b = unit / a.Hkv;
  const int n = unit_len(a.ctx_lens[b], a.max_ctx, a.chunk);
  const int j0 = tile * kFilterTile;
  if (j0 >= n) return;
  const int jend = min(j0 + kFilterTile, n);
  for (int i = threadIdx.x; i < kHistBins; i += kScoreThreads) lds_hist[i] = 0u;
  __syncthreads();
  const float* srow = a.scores + (int64_t)unit * a.max_ctx;
  for (int j = j0 + threadIdx.x; j < jend; j += kScoreThreads)
    atomicAdd(&lds_hist[order_key(srow[j]) >> (32 - kHistBits)], 1u);
  __syncthreads();
  flush_hist(lds_hist, a.hist + (int64_t)unit * kHistBins,
             a.coarse + (int64_t)unit * kCoarseBins);
}

// Selects positions above the first-digit bin of the m-th largest key and
// collects the positions inside that bin as candidates.
__global__ __launch_bounds__(kFilterThreads) void k_filter(SelectArgs a) {
  constexpr int kPer = kFilterTile / kFilterThreads;  // 16 positions per thread
  __shared__ uint32_t sh[4];
  __shared__ uint32_t scan_tmp[kFilterThreads / 64 + 1];
  const int unit = blockIdx.x / a.tiles;
  const int tile = blockIdx.x - unit * a.tiles;
  const int b = unit / a.Hkv;
  const int n = unit_len(a.ctx_lens[b], a.max_ctx, a.chunk);
  const int m = min(a.k, n);
  const int j0 = tile * kFilterTile;
  if (m == 0 || m >= n || j0 >= n) return;  // uniform
  // issue the score loads first; the bin lookup below overlaps their latency
  const float* srow = a.scores + (int64_t)unit * a.max_ctx;
  float sv[kPer];
#pragma unroll
  for (int r = 0; r < kPer; ++r)  // unconditional loads (clamped position)
    sv[r] = srow[min(j0 + r * kFilterThreads + (int)threadIdx.x, n - 1)];
  if (threadIdx.x < 64)
    find_first_bin(a.coarse + (int64_t)unit * kCoarseBins,
                   a.hist + (int64_t)unit * kHistBins, (uint32_t)m, sh);
  __syncthreads();
  const uint32_t b1 = sh[0];
  uint32_t keys[kPer];
  uint32_t selmask = 0u, candmask = 0u;
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int j = j0 + r * kFilterThreads + threadIdx.x;
    keys[r] = 0u;
    if (j < n) {
      const uint32_t key = order_key(sv[r]);
      const uint32_t d1 = key >> (32 - kHistBits);
      keys[r] = key;
      if (d1 > b1) selmask |= 1u << r;
      else if (d1 == b1) candmask |= 1u << r;
    }
  }
  const uint32_t cnt = (uint32_t)__popc(selmask) | ((uint32_t)__popc(candmask) << 16);
  uint32_t total;
  const uint32_t excl = block_incl_scan<kFilterThreads / 64>(cnt, scan_tmp, &total) - cnt;
  if (threadIdx.x == 0) {
    uint32_t* ctrl = a.ctrl + (int64_t)unit * kCtrlWords;
    sh[2] = (total & 0xffffu) ? atomicAdd(&ctrl[0], total & 0xffffu) : 0u;
    sh[3] = (total >> 16) ? atomicAdd(&ctrl[1], total >> 16) : 0u;
    if (tile == 0) ctrl[2] = b1;
  }
  __syncthreads();
  uint32_t os = sh[2] + (excl & 0xffffu), oc = sh[3] + (excl >> 16);
  int32_t* sel = a.sel + (int64_t)unit * a.k;
  uint2* cand = a.cand + (int64_t)unit * a.max_ctx;
#pragma unroll
  for (int r = 0; r < kPer; ++r) {
    const int j = j0 + r * kFilterThreads + threadIdx.x;
    if ((selmask >> r) & 1u) sel[os++] = j;
    else if ((candmask >> r) & 1u) cand[oc++] = make_uint2(keys[r], (uint32_t)j);
  }
}

// Zeroes the unit's first-digit histogram, coarse histogram and control
// words, as the clearing kernel would, after the selection has read them for
// the last time (all kFinishThreads threads; thread t takes bins 2t and
// 2t + 1, the bins it loaded itself).  A selection that counted its first
// digit into these cleared areas leaves them clear, so a caller running
// several selections on one workspace in stream order clears it once.
__device__ __forceinline__ void clear_unit_hist(const SelectArgs& a, int unit) {
  static_assert(2 * kFinishThreads == kHistBins, "two bins per thread");
  __builtin_amdgcn_s_waitcnt(0);  // this thread's own loads of these words are back
  __syncthreads();                // and every other thread's
  const int t = threadIdx.x;
  *reinterpret_cast<uint2*>(a.hist + (int64_t)unit * kHistBins + 2 * t) = make_uint2(0u, 0u);
  if (t < kCoarseBins) a.coarse[(int64_t)unit * kCoarseBins + t] = 0u;
  if (t < kCtrlWords) a.ctrl[(int64_t)unit * kCtrlWords + t] = 0u;
}

// Writes set bits of bm[0, words) as ascending positions to out[0, limit)
// (when out is not null), the NT / 64 waves each owning a contiguous word range (reads
// are lane-consecutive), and returns the number of set bits.  Output slots
// [lo, hi) also go to share[slot - lo] when share is not null.  The bitmap
// holds exactly m <= limit bits for scores as specified; the limit only keeps
// other input (NaN scores) inside the row.
template <int NT = kFinishThreads>
__device__ __forceinline__ uint32_t emit_bitmap(const uint32_t* bm, int words, int32_t* out,
                                                uint32_t limit, uint32_t* tmp,
                                                int32_t* share = nullptr, uint32_t lo = 0,
                                                uint32_t hi = 0) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int kW = NT / 64;
  const int per = (((words + kW - 1) / kW) + 63) & ~63;
  const int w0 = wave * per, w1 = min(w0 + per, words);
  uint32_t cnt = 0;
  for (int w = w0 + lane; w < w1; w += 64) cnt += (uint32_t)__popc(bm[w]);
  cnt = wave_sum_u32(cnt);
  if (lane == 0) tmp[wave] = cnt;
  __syncthreads();
  uint32_t base = 0, total = 0;
  for (int i = 0; i < kW; ++i) {
    const uint32_t t = tmp[i];
    base += i < wave ? t : 0u;
    total += t;
  }
  for (int ws = w0; ws < w1; ws += 64) {
    const int w = ws + lane;
    uint32_t bits = w < w1 ? bm[w] : 0u;
    const uint32_t c = (uint32_t)__popc(bits);
    const uint32_t incl = wave_incl_scan(c);
    uint32_t o = base + incl - c;
    while (bits) {
      const int bit = __ffs(bits) - 1;
      if (o < limit) {
        if (out) out[o] = w * 32 + bit;
        if (share && o >= lo && o < hi) share[o - lo] = w * 32 + bit;
      }
      ++o;
      bits &= bits - 1u;
    }
    base += __builtin_amdgcn_readlane(incl, 63);
  }
  __syncthreads();
  return total;
}

// Radix select among candidates (order key, position) that share the first
// digit b1: the need largest by (key descending, position ascending).
// Returns the threshold key T; candidates with key > T are all chosen, and of
// those equal to T the ones with position <= *pmax.  All NT threads call
// this; hist needs 2048 words.
template <class Cands, int NT = kFinishThreads>
__device__ __forceinline__ uint32_t refine_threshold(const Cands& cs, uint32_t nc,
                                                     uint32_t need, uint32_t b1,
                                                     uint32_t* hist, uint32_t* tmp,
                                                     uint32_t* misc, uint32_t* pmax) {
  const int tid = threadIdx.x;
  // Second digit: bits 20..10 of the order key (11 bits).
  static_assert(kHistBits == 11, "digits 11 + 11 + 10");
  for (int i = tid; i < 2048; i += NT) hist[i] = 0u;
  __syncthreads();
  for (uint32_t i = tid; i < nc; i += NT)
    atomicAdd(&hist[(cs[i].x >> 10) & 2047u], 1u);
  __syncthreads();
  uint32_t need2;
  const uint32_t b2 = find_bin_block<true, NT>(hist, 2048, need, tmp, misc, &need2);
  // Third digit: bits 9..0, among candidates whose second digit is b2.
  for (int i = tid; i < 1024; i += NT) hist[i] = 0u;
  __syncthreads();
  for (uint32_t i = tid; i < nc; i += NT) {
    const uint32_t key = cs[i].x;
    if (((key >> 10) & 2047u) == b2) atomicAdd(&hist[key & 1023u], 1u);
  }
  __syncthreads();
  uint32_t need3;
  const uint32_t b3 = find_bin_block<true, NT>(hist, 1024, need2, tmp, misc, &need3);
  const uint32_t T = (b1 << 21) | (b2 << 10) | b3;
  const uint32_t eq = hist[b3];  // candidates with key == T
  __syncthreads();

  // Ties at T: keep the need3 lowest positions (radix select on position,
  // ascending, 8 bits at a time).
  *pmax = 0xffffffffu;
  if (eq > need3) {
    uint32_t prefix = 0u, want = need3;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += NT) hist[i] = 0u;
      __syncthreads();
      const uint32_t hi_mask = shift == 24 ? 0u : (0xffffffffu << (shift + 8));
      for (uint32_t i = tid; i < nc; i += NT) {
        const uint2 c = cs[i];
        if (c.x == T && (c.y & hi_mask) == prefix) atomicAdd(&hist[(c.y >> shift) & 255u], 1u);
      }
      __syncthreads();
      uint32_t rest;
      const uint32_t bb = find_bin_block<false, NT>(hist, 256, want, tmp, misc, &rest);
      prefix |= bb << shift;
      want = rest;
    }
    *pmax = prefix;  // the need3-th smallest tied position
  }
  return T;
}

__global__ __launch_bounds__(kFinishThreads) void k_finish(SelectArgs a) {
  __shared__ uint2 area[kCandLds];  // candidates, later the position bitmap
  __shared__ uint32_t hist[2048];
  __shared__ uint32_t tmp[kFinishThreads / 64 + 1];
  __shared__ uint32_t misc[8];
  const int unit = blockIdx.x;
  const int b = unit / a.Hkv;
  const int n = unit_len(a.ctx_lens[b], a.max_ctx, a.chunk);
  const int m = min(a.k, n);
  const int tid = threadIdx.x;
  int32_t* idx = a.idx + (int64_t)unit * a.k;
  if (m >= n) {  // uniform; every position (possibly none) is selected
    for (int i = tid; i < a.k; i += kFinishThreads) idx[i] = i < n ? i : -1;
    if (tid == 0) a.n_sel[unit] = m;
    clear_unit_hist(a, unit);
    return;
  }
  const uint32_t* ctrl = a.ctrl + (int64_t)unit * kCtrlWords;
  const uint32_t above = ctrl[0], nc = ctrl[1], b1 = ctrl[2];
  const uint32_t need = (uint32_t)m - above;  // >= 1 and <= nc
  const uint2* cg = a.cand + (int64_t)unit * a.max_ctx;
  const bool in_lds = nc <= (uint32_t)kCandLds;
  if (in_lds) {
    for (uint32_t i = tid; i < nc; i += kFinishThreads) area[i] = cg[i];
  }
  const uint2* cs = in_lds ? area : cg;
  uint32_t pmax;
  const uint32_t T = refine_threshold(cs, nc, need, b1, hist, tmp, misc, &pmax);

  // Append the chosen candidates after the positions selected by the filter.
  if (tid == 0) misc[4] = above;
  __syncthreads();
  int32_t* sel = a.sel + (int64_t)unit * a.k;
  for (uint32_t i0 = 0; i0 < nc; i0 += kFinishThreads) {
    const uint32_t i = i0 + tid;
    bool take = false;
    uint2 c = make_uint2(0u, 0u);
    if (i < nc) {
      c = cs[i];
      take = c.x > T || (c.x == T && c.y <= pmax);
    }
    const uint32_t slot = wave_append(take, &misc[4]);
    if (take) sel[slot] = (int32_t)c.y;
  }
  __syncthreads();

  // Mark the m chosen positions in a bitmap and emit them in ascending order.
  const int words = (n + 31) >> 5;
  uint32_t* bm = n <= kBitmapLdsBits ? reinterpret_cast<uint32_t*>(area)
                                     : a.bitmap + (int64_t)unit * a.bm_words;
  for (int w = tid; w < words; w += kFinishThreads) bm[w] = 0u;
  __syncthreads();
  for (int i = tid; i < m; i += kFinishThreads) {
    const int p = sel[i];
    atomicOr(&bm[p >> 5], 1u << (p & 31));
  }
  __syncthreads();
  emit_bitmap(bm, words, idx, (uint32_t)a.k, tmp);
  for (int i = m + tid; i < a.k; i += kFinishThreads) idx[i] = -1;
  if (tid == 0) a.n_sel[unit] = m;
  clear_unit_hist(a, unit);
}

// Whole selection of one unit in one workgroup, for n_b <= kFusedSelectMaxCtx.
// The unit's scores are read once, kSelPer per thread per batch of
// kSelBatch positions, all loads of a batch in flight together.  Positions
// above the first-digit bin go straight into an LDS bitmap (one ballot per
// 64 positions, no atomics); positions inside the bin become candidates
// (fp32 bits, position), whose slots are reserved with one atomic per wave.
// The threshold inside the bin is then resolved exactly, the chosen
// candidates marked, and the bitmap written out in ascending order.
constexpr int kSelPer = 32;
constexpr int kSelBatch = kSelPer * kFinishThreads;
static_assert(kFusedSelectMaxCtx % kSelBatch == 0, "whole batches");

template <int NT = kFinishThreads, bool COH = false>
__device__ __forceinline__ void load_score_batch(const float* srow, int j0, int n,
                                                 float (&sv)[kSelPer]) {
  // unconditional loads (clamped position); 32-bit byte offsets from the
  // row base let every load share one scalar base address
  const char* base = reinterpret_cast<const char*>(srow);
#pragma unroll
  for (int u = 0; u < kSelPer; ++u) {
    const uint32_t off = 4u * (uint32_t)min(j0 + u * NT + (int)threadIdx.x, n - 1);
    if constexpr (COH)  // stored by other workgroups of the same launch
      sv[u] = __hip_atomic_load(reinterpret_cast<const float*>(base + off), __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
    else
      sv[u] = *reinterpret_cast<const float*>(base + off);
  }
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Candidate slots of the fused selection: the first CAP in LDS, any beyond
// (heavy ties) in the unit's global candidate area.
template <int CAP = kCandLds>
struct SplitCands {
  uint2* lds;
  uint2* glob;
  __device__ __forceinline__ uint2 operator[](uint32_t i) const {
    return i < (uint32_t)CAP ? lds[i] : glob[i];
  }
  __device__ __forceinline__ void put(uint32_t i, uint2 v) const {
    if (i < (uint32_t)CAP) lds[i] = v;
    else glob[i] = v;
  }
};

// One batch of kSelBatch positions starting at j0, with two fp32 compares
// per position: x >= g_hi <=> key(x) is above the first-digit bin b1 (set in
// the LDS bitmap, one ballot per 64 positions), g_lo <= x < g_hi <=> key(x)
// lies in it (a candidate (fp32 bits, position) appended at *ctr, one atomic
// per wave).  Positions at or past n_b must hold NaN (then neither holds).
template <int NT = kFinishThreads, int CAP = kCandLds>
__device__ __forceinline__ void classify_batch(const float (&sv)[kSelPer], int j0, float g_lo,
                                               float g_hi, uint32_t* bm, const SplitCands<CAP>& cs,
                                               uint32_t* ctr) {
  static_assert(2 * kSelPer == 64, "one bitmap word per lane and batch");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint32_t word = 0u, wc = 0u;
#pragma unroll
  for (int u = 0; u < kSelPer; ++u) {
    const uint64_t hi = __builtin_amdgcn_ballot_w64(sv[u] >= g_hi);
    const uint64_t ge = __builtin_amdgcn_ballot_w64(sv[u] >= g_lo);
    // lane 2u + h keeps word h of the wave's 64 positions.  The compare that
    // wrote `hi` is a VALU write of SGPRs, which a VALU read right after may
    // miss: the nop keeps the wait states the compiler cannot see inside asm.
    asm("s_nop 4\n\tv_writelane_b32 %0, %1, %2\n\tv_writelane_b32 %0, %3, %4"
        : "+v"(word)
        : "s"((uint32_t)hi), "n"(2 * u), "s"((uint32_t)(hi >> 32)), "n"(2 * u + 1));
    wc += (uint32_t)__popcll(ge & ~hi);
  }
  bm[((j0 + (lane >> 1) * NT + wave * 64) >> 5) + (lane & 1)] = word;
  uint32_t base = 0u;
  if (lane == 0 && wc) base = atomicAdd(ctr, wc);
  base = __builtin_amdgcn_readfirstlane(base);
  if (base + wc <= (uint32_t)CAP) {  // the wave's candidates all fit in LDS
#pragma unroll
    for (int u = 0; u < kSelPer; ++u) {
      // compare again rather than keep 2 x kSelPer lane masks live
      float x = sv[u];
      asm volatile("" : "+v"(x));
      const int j = j0 + u * NT + tid;
      // g_lo <= g_hi, so "in the bin" is the exclusive or of the two tests
      const bool ge = x >= g_lo, hi = x >= g_hi;
      const uint64_t cm = __builtin_amdgcn_ballot_w64(ge) & ~__builtin_amdgcn_ballot_w64(hi);
      if (ge != hi) cs.lds[base + lanes_below(cm)] = make_uint2(__float_as_uint(x), (uint32_t)j);
      base += (uint32_t)__popcll(cm);
    }
  } else {
    for (int u = 0; u < kSelPer; ++u) {
      const int j = j0 + u * NT + tid;
      const bool in = sv[u] >= g_lo && !(sv[u] >= g_hi);
      const uint64_t cm = __builtin_amdgcn_ballot_w64(in);
      if (in) cs.put(base + lanes_below(cm), make_uint2(__float_as_uint(sv[u]), (uint32_t)j));
      base += (uint32_t)__popcll(cm);
    }
  }
}

// The candidates as (order key, position): the fused selection stores the
// scores' fp32 bits and converts on every read.
template <int CAP = kCandLds>
struct KeyedCands {
  SplitCands<CAP> c;
  __device__ __forceinline__ uint2 operator[](uint32_t i) const {
    const uint2 v = c[i];
    return make_uint2(order_key(__uint_as_float(v.x)), v.y);
  }
};

// Pipelined calls: merges the attention partials of the launch before the
// selection for one unit into the output, as the merge kernel does and in
// its order of operations: out[b][h*G + g] = sum over chunks of
// exp(m_c - M) o_c / sum over chunks of exp(m_c - M) l_c.  Thread t < mG * kD
// owns channel t % kD of head t / kD; thread t < mchunks * mG reads the
// (max, weight sum) of chunk t / mG, head t % mG.  lds: 16 * (2 *
// kMergeChunks + 1) floats, free on entry.  All kFinishThreads threads call
// it, from one place of the kernel (an inlined second copy kept more of the
// selection's registers live).
__device__ __forceinline__ void merge_partials(const SelectArgs& a, int unit, uint32_t* lds) {
  const int tid = threadIdx.x;
  const int G = a.mG, nc = a.mchunks;
  const float* pu = a.mpart + (int64_t)unit * nc * G * kPartStride;
  // unconditional (clamped) loads
  float mo[kMergeChunks];
  const int og = min(tid / kD, G - 1), oc = tid % kD;
#pragma unroll
  for (int ch = 0; ch < kMergeChunks; ++ch)
    mo[ch] = pu[(min(ch, nc - 1) * G + og) * kPartStride + 4 + oc];
  const int pc = min(tid, nc * G - 1);
  const float mmax = pu[pc * kPartStride], msum = pu[pc * kPartStride + 1];
  float* s_w = reinterpret_cast<float*>(lds);  // [16][kMergeChunks] weights
  float* s_l = s_w + 16 * kMergeChunks;        // [16][kMergeChunks] weight sums
  float* s_inv = s_l + 16 * kMergeChunks;      // [16]
  __syncthreads();
  if (tid < nc * G) {
    const int ch = tid / G, g = tid - ch * G;
    s_w[g * kMergeChunks + ch] = mmax;
    s_l[g * kMergeChunks + ch] = msum;
  }
  __syncthreads();
  if (tid < G) {
    const int g = tid;
    float M = -INFINITY;
    for (int ch = 0; ch < nc; ++ch) M = fmaxf(M, s_w[g * kMergeChunks + ch]);
    float L = 0.f;
    for (int ch = 0; ch < nc; ++ch) {
      const float mc = s_w[g * kMergeChunks + ch];
      const float w = mc == -INFINITY ? 0.f : __expf(mc - M);
      L = fmaf(w, s_l[g * kMergeChunks + ch], L);
      s_w[g * kMergeChunks + ch] = w;
    }
    s_inv[g] = L > 0.f ? 1.f / L : 0.f;
  }
  __syncthreads();
  if (tid < G * kD) {
    const int g = tid / kD, c = tid - g * kD;
    float O = 0.f;
#pragma unroll
    for (int ch = 0; ch < kMergeChunks; ++ch)
      if (ch < nc) O = fmaf(s_w[g * kMergeChunks + ch], mo[ch], O);
    const int b = unit / a.Hkv, h = unit - b * a.Hkv;
    a.mout[((int64_t)b * a.mHq + (int64_t)h * G + g) * kD + c] = O * s_inv[g];
  }
}

// LDS of a one-workgroup selection (see select_unit).
struct SelLds {
  uint2* cand;      // [CAP of select_unit]
  uint32_t* bm;     // [kFusedSelectMaxCtx / 32]
  uint32_t* lhist;  // [2048]
  uint32_t* tmp;    // [threads / 64 + 1]
  uint32_t* misc;   // [8]
};

// The whole selection of one unit by one workgroup of NT threads, for
// n_b <= kFusedSelectMaxCtx.  The unit's scores are read once, kSelPer per
// thread per batch of kSelPer * NT positions, all loads of a batch in flight
// together.  Positions above the first-digit bin go straight into an LDS
// bitmap (one ballot per 64 positions, no atomics); positions inside the bin
// become candidates (fp32 bits, position), whose slots are reserved with one
// atomic per wave.  The threshold inside the bin is then resolved exactly,
// the chosen candidates marked, and the bitmap written out in ascending
// order: to idx/n_sel when `write`, and output slots [lo, hi) to share[slot -
// lo] when share is not null.  When the first digit was counted into the
// cleared per-unit histogram (no hist_part) and `clear` is set, the unit's
// histogram and control words are left cleared; only the unit's one reader
// may do that (kFinishThreads workgroups only).  Returns the number of
// positions selected.
template <int NT = kFinishThreads, int CAP = kCandLds, bool COH = false>
__device__ __forceinline__ int select_unit(const SelectArgs& a, int unit, const SelLds& L,
                                           bool write, int32_t* share, uint32_t lo,
                                           uint32_t hi, bool clear) {
  static_assert(NT >= 128 && kHistBins % NT == 0 && kFusedSelectMaxCtx % (kSelPer * NT) == 0,
                "workgroup shape");
  constexpr int kBatch = kSelPer * NT;
  const int tid = threadIdx.x;
  uint2* const cand = L.cand;
  uint32_t* const bm = L.bm;
  uint32_t* const lhist = L.lhist;
  uint32_t* const tmp = L.tmp;
  uint32_t* const misc = L.misc;
  // Every read the workgroup needs first is issued before anything waits:
  // the histogram, and the first batch of scores (clamped to the row, not
  // to n_b, which is not known yet; positions at or past n_b are masked).
  // The histogram is the sum of the slots unit + wg of the workgroups that
  // scored the unit's groups (every such workgroup stores one, zeros where
  // its groups lie past n_b), or one slot already summed.
  const uint32_t* slots = a.hist + (int64_t)unit * kHistBins;
  int nslots = 1;
  if (a.hist_part) {
    const int64_t gu = (a.max_ctx + kStageRows - 1) / kStageRows;
    if (a.affine) {
      slots = a.hist_part + xcd_slot0(unit, a.units, a.score_nwg, gu, &nslots) * kHistBins;
      nslots = min(nslots, kMaxPartials);  // the host keeps it below
    } else {
      const int64_t T = gu * a.units, g0 = (int64_t)unit * gu;
      const int64_t lo_wg = range_owner(g0, T, a.score_nwg);
      const int64_t hi_wg = range_owner(g0 + gu - 1, T, a.score_nwg);
      slots = a.hist_part + (unit + lo_wg) * kHistBins;
      nslots = (int)min<int64_t>(hi_wg - lo_wg + 1, kMaxPartials);  // the host keeps it below
    }
  }
  const int len_b = a.ctx_lens[unit / a.Hkv];
  uint2 hv[kMaxPartials][kHistBins / NT / 2];
  load_hist_slots<NT, COH>(slots, nslots, hv);
  // every wave's histogram loads queue ahead of all score loads (a bare
  // barrier: no wait for the loads themselves)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  const float* srow = a.scores + (int64_t)unit * a.max_ctx;
  float sv0[kSelPer];
  load_score_batch<NT, COH>(srow, 0, a.max_ctx, sv0);
  __builtin_amdgcn_sched_barrier(0);  // n_b is waited for only here
  const int n = unit_len(len_b, a.max_ctx, a.chunk);
  const int m = min(a.k, n);
  int32_t* idx = a.idx + (int64_t)unit * a.k;
  if (m >= n) {  // uniform; every position (possibly none) is selected
    for (int i = tid; i < a.k; i += NT) {
      if (write) idx[i] = i < n ? i : -1;
      if (share && i < n && (uint32_t)i >= lo && (uint32_t)i < hi) share[i - lo] = i;
    }
    if (write && tid == 0) a.n_sel[unit] = m;
    if constexpr (NT == kFinishThreads) {
      if (clear && !a.hist_part) clear_unit_hist(a, unit);
    }
    return m;
  }
  store_hist_sum<NT>(hv, nslots, lhist);
  if (tid == 64) misc[7] = 0u;
  // the scores may still be in flight across both barriers
  lds_barrier();
  if (tid < 64) find_first_bin_lds(lhist, (uint32_t)m, misc + 4);
  lds_barrier();
  const SplitCands<CAP> cs{cand, a.cand + (int64_t)unit * a.max_ctx};
  const uint32_t b1 = misc[4], above = misc[5];
  const float g_lo = __uint_as_float(key_floor_bits((uint64_t)b1 << (32 - kHistBits)));
  const float g_hi = __uint_as_float(key_floor_bits((uint64_t)(b1 + 1u) << (32 - kHistBits)));
  // the last, partial batch holds NaN past n_b
  auto pad = [&](float (&sv)[kSelPer], int j0) {
    if (j0 + kBatch > n) {
#pragma unroll
      for (int u = 0; u < kSelPer; ++u)
        if (j0 + u * NT + tid >= n) sv[u] = __builtin_nanf("");
    }
  };
  // the first batch apart, so that its compares start as its loads land
  pad(sv0, 0);
  classify_batch<NT, CAP>(sv0, 0, g_lo, g_hi, bm, cs, &misc[7]);
  for (int j0 = kBatch; j0 < n; j0 += kBatch) {
    float sv[kSelPer];
    load_score_batch<NT, COH>(srow, j0, n, sv);
    pad(sv, j0);
    classify_batch<NT, CAP>(sv, j0, g_lo, g_hi, bm, cs, &misc[7]);
  }
  __syncthreads();
  const uint32_t nc = misc[7];
  const uint32_t need = (uint32_t)m - above;
  const KeyedCands<CAP> kc{cs};
  uint32_t pmax;
  const uint32_t T = refine_threshold<KeyedCands<CAP>, NT>(kc, nc, need, b1, lhist, tmp, misc, &pmax);
  for (uint32_t i = tid; i < nc; i += NT) {
    const uint2 c = kc[i];
    if (c.x > T || (c.x == T && c.y <= pmax)) atomicOr(&bm[c.y >> 5], 1u << (c.y & 31));
  }
  __syncthreads();
  // m positions for scores as specified (fewer only with NaN scores)
  const int got = (int)min(emit_bitmap<NT>(bm, (n + 31) >> 5, write ? idx : nullptr,
                                       (uint32_t)a.k, tmp, share, lo, hi),
                           (uint32_t)m);
  if (write) {
    for (int i = got + tid; i < a.k; i += NT) idx[i] = -1;
    if (tid == 0) a.n_sel[unit] = got;
  }
  if constexpr (NT == kFinishThreads) {
      if (clear && !a.hist_part) clear_unit_hist(a, unit);
    }
  return got;
}

__global__ __launch_bounds__(kFinishThreads) void k_select_fused(SelectArgs a) {
  __shared__ uint2 cand[kCandLds];
  __shared__ uint32_t bm[kFusedSelectMaxCtx / 32];
  __shared__ uint32_t lhist[2048];
  __shared__ uint32_t tmp[kFinishThreads / 64 + 1];
  __shared__ uint32_t misc[8];
  const int unit = blockIdx.x;
  select_unit(a, unit, SelLds{cand, bm, lhist, tmp, misc}, true, nullptr, 0, 0, true);
  // one call site, so that the merge appears once (a second inlined copy
  // kept more of the selection's registers live)
  if (a.mpart) merge_partials(a, unit, lhist);
}

// ---- selection and attention in one launch ------------------------------------
// Same-step decode with a set of at most kSelAttnMaxShare rows per share:
// each workgroup selects its unit's set (select_unit; share 0 writes idx and
// n_sel), keeps the positions of its share in LDS and attends over them with
// all 16 waves (attn_wg).  A unit has nsplit shares, each selected in full by
// its own workgroup, so that the attention has a workgroup on every CU.  The
// LDS is a union: the selection's candidates, bitmap and histogram, then the
// attention's stages and query rows; the share's positions lie past the
// selection's area, since they are written while its bitmap is emitted.
template <int G>
struct SelAttnLds {
  static constexpr int kSel = 2 * kCandLds + kFusedSelectMaxCtx / 32 + 2048;  // dwords
  static constexpr int kQOff = WgAttnLds<G>::kStages;
  static constexpr int kPosOff =
      kSel > kQOff + WgAttnLds<G>::kQ ? kSel : kQOff + WgAttnLds<G>::kQ;
  static constexpr int kDwords = kPosOff + kSelAttnMaxShare;
};

// Workgroup -> (unit, share).  Workgroups are spread over the XCDs round-robin
// by index, so the shares of unit u take indices 8*S*(u/8) + 8*s + u%8: all
// on the XCD of u % 8, where the second read of the unit's scores can hit
// the L2.  Indices past the last unit have no work.
__device__ __forceinline__ void split_block(int blk, int nsplit, int* unit, int* split) {
  if (nsplit == 1) {
    *unit = blk;
    *split = 0;
    return;
  }
  const int grp = blk / (8 * nsplit), r = blk - grp * 8 * nsplit;
  *split = r >> 3;
  *unit = grp * 8 + (r & 7);
}

// HEADS == 1: the unit's set is split into nsplit shares of rows, each
// attended by one workgroup with all G heads, and k_combine merges the
// shares.  HEADS > 1: HEADS workgroups per unit each attend over the whole
// set with G / HEADS of the heads and write their outputs directly (no
// partials, no merge launch); the second workgroup's reads of each row come
// while the first one's are recent, from the XCD's L2.
// One workgroup's part of k_select_attn: the selection of `unit`, then the
// attention over its share of the rows or with its share of the heads.
// COH: the scores and slots were stored by other workgroups of the same launch.
// MERGE2 (HEADS 1, nsplit 2): the two shares merge through fs (attn_wg).
template <int G, int HEADS, bool COH = false, bool MERGE2 = false>
__device__ __forceinline__ void select_attn_part(const SelectArgs& sa, const AttnArgs& at,
                                                 int unit, int split, int nsplit,
                                                 uint32_t* lds, uint32_t* tmp,
                                                 uint32_t* misc,
                                                 const FusedSync* fs = nullptr) {
  static_assert(!MERGE2 || HEADS == 1, "the merge joins row shares");
  static_assert(G % HEADS == 0, "whole heads per workgroup");
  constexpr int GA = G / HEADS;  // heads each workgroup attends with
  using Lds = SelAttnLds<GA>;
  const SelLds L{reinterpret_cast<uint2*>(lds), lds + 2 * kCandLds,
                 lds + 2 * kCandLds + kFusedSelectMaxCtx / 32, tmp, misc};
  int32_t* share = reinterpret_cast<int32_t*>(lds + Lds::kPosOff);
  // the share of a set of m positions is known before the set is: m =
  // min(k, n_b), and the split is by m
  const int n = unit_len(sa.ctx_lens[unit / sa.Hkv], sa.max_ctx, sa.chunk);
  int lo = 0, hi = min(sa.k, n);
  if (HEADS == 1) share_range(hi, split, nsplit, &lo, &hi);
  // the workgroups of a unit all read its histogram: none clears it
  select_unit<kFinishThreads, kCandLds, COH>(sa, unit, L, split == 0, share, (uint32_t)lo,
                                             (uint32_t)hi, false);
  __syncthreads();
  const int qh0 = (unit % sa.Hkv) * G + (HEADS > 1 ? split * GA : 0);
  if constexpr (MERGE2)
    attn_wg<GA, LdsRows, true>(at, unit, LdsRows{share}, hi - lo, split, 2, lds,
                               lds + Lds::kQOff, qh0, nullptr, nullptr, 0, fs->merge + unit,
                               fs->tag);
  else
    attn_wg<GA>(at, unit, LdsRows{share}, hi - lo, HEADS > 1 ? 0 : split,
                HEADS > 1 ? 1 : nsplit, lds, lds + Lds::kQOff, qh0);
}

// MERGE2: two row shares that merge in the launch through fs (attn_wg).
template <int G, int HEADS, bool MERGE2 = false>
__global__ __launch_bounds__(kFinishThreads) void k_select_attn(SelectArgs sa, AttnArgs at,
                                                                  int nsplit, FusedSync fs) {
  __shared__ __attribute__((aligned(16))) uint32_t lds[SelAttnLds<G / HEADS>::kDwords];
  __shared__ uint32_t tmp[kFinishThreads / 64 + 1];
  __shared__ uint32_t misc[8];
  int unit, split;
  split_block(blockIdx.x, HEADS > 1 ? HEADS : nsplit, &unit, &split);
  if (unit >= sa.units) return;  // uniform over the workgroup
  select_attn_part<G, HEADS, false, MERGE2>(sa, at, unit, split, nsplit, lds, tmp, misc, &fs);
}

// ---- the same-step layer in one launch ------------------------------------
// Scoring, selection and attention of a same-step call in one launch, for
// the head-halves form at U and grid multiples of 8.  The first nS
// workgroups (one per CU, dispatched first) score with XCD-affine ranges
// (xcd_slot0): the units of XCD x are complete as soon as its ranges are.
// The XCDs stream at different rates, so the units of the faster ones select
// and attend while the slower ones still score, and no unit waits for a
// launch boundary.  The 2U workgroups after them are k_select_attn's head
// halves, placed by the same index map on the XCD that scored their unit.
// Each waits for the hand-over flags of its unit's slots (FusedSync), then
// reads the scores and slots with device-coherent loads, so nothing rests on
// where the workgroups run.  Only higher-indexed workgroups wait, and only
// for lower-indexed ones that never wait.  The wait is bounded all the same
// (kFusedSpinLimit polls): a broken hand-over leaves the outputs undefined
// but cannot hang the launch.
template <int G, bool ROWS>
__global__ __launch_bounds__(kFinishThreads) void k_critical(ScoreArgs sc, SelectArgs sa,
                                                             AttnArgs at, FusedSync fs, int nS) {
  using Lds = SelAttnLds<ROWS ? G : G / 2>;
  static_assert(kHistBins + kHistScoreWaves * (kStageDwords + kFlushGroups * kStageRows) <=
                    Lds::kDwords,
                "the scoring role's histogram, stages and score buffers fit");
  __shared__ __attribute__((aligned(16))) uint32_t lds[Lds::kDwords];
  __shared__ uint32_t tmp[kFinishThreads / 64 + 1];
  __shared__ uint32_t misc[8];
  if ((int)blockIdx.x < nS) {
    score_range<G, true, kHistScoreWaves, false, true>(sc, blockIdx.x, nS, lds,
                                                       lds + kHistBins, fs);
    return;
  }
  int unit, half;
  split_block(blockIdx.x - nS, 2, &unit, &half);
  if (unit >= sa.units) return;  // uniform over the workgroup
  int nslots;
  const int64_t s0 = xcd_slot0(unit, sa.units, sa.score_nwg,
                               (sa.max_ctx + kStageRows - 1) / kStageRows, &nslots);
  if ((int)threadIdx.x < nslots) {
    uint64_t* f = fs.flags + 2 * (s0 + threadIdx.x) + half;
    for (uint32_t spin = 0;
         __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != fs.tag &&
         spin < kFusedSpinLimit;
         ++spin)
      __builtin_amdgcn_s_sleep(2);
    __hip_atomic_store(f, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if constexpr (ROWS)
    select_attn_part<G, 1, true, true>(sa, at, unit, half, 2, lds, tmp, misc, &fs);
  else
    select_attn_part<G, 2, true>(sa, at, unit, half, 1, lds, tmp, misc);
}

// Same-step over chunks (Sec. 2.2): sa is the chunk problem (one landmark
// score per chunk of sa.chunk rows, budget k / chunk), at the attention over
// rows.  Like k_select_attn with head halves, each of the unit's two
// workgroups selects the unit's chunks, then expands them in LDS to the rows
// below n_b and attends over all of them with half of the group's heads.
// The first workgroup also writes the chunk list (sa.idx, sa.n_sel) and the
// rows as k_expand does: e.rows[i] = row i of the ascending expansion, -1 at
// or past n_b and past the last chunk, and e.n_rows.  Needs k / chunk <=
// kFinishThreads and k <= kSelAttnMaxShare.
template <int G>
__global__ __launch_bounds__(kFinishThreads) void k_select_attn_chunks(SelectArgs sa,
                                                                         AttnArgs at,
                                                                         ExpandArgs e) {
  constexpr int GA = G / 2;
  using Lds = SelAttnLds<GA>;
  __shared__ __attribute__((aligned(16))) uint32_t lds[Lds::kDwords];
  __shared__ uint32_t tmp[kFinishThreads / 64 + 1];
  __shared__ uint32_t misc[8];
  const int tid = threadIdx.x;
  int unit, split;
  split_block(blockIdx.x, 2, &unit, &split);
  if (unit >= sa.units) return;  // uniform over the workgroup
  const SelLds L{reinterpret_cast<uint2*>(lds), lds + 2 * kCandLds,
                 lds + 2 * kCandLds + kFusedSelectMaxCtx / 32, tmp, misc};
  int32_t* list = reinterpret_cast<int32_t*>(lds + Lds::kPosOff);
  const int nc = unit_len(sa.ctx_lens[unit / sa.Hkv], sa.max_ctx, sa.chunk);
  const int m = select_unit(sa, unit, L, split == 0, list, 0u, (uint32_t)min(sa.k, nc), false);
  __syncthreads();
  // chunk tid's number, then its rows in place (chunk c of the list holds
  // list slots [c * chunk, c * chunk + chunk))
  const int C = e.chunk;
  const int n = clamp_len(e.ctx_lens[unit / e.Hkv], e.max_ctx);
  const int c_mine = tid < m ? list[tid] : -1;
  const int c_last = m > 0 ? list[m - 1] : 0;
  __syncthreads();
  if (c_mine >= 0)
    for (int r = 0; r < C; ++r) list[tid * C + r] = c_mine * C + r;
  const int rows = m == 0 ? 0 : (m - 1) * C + max(0, min(C, n - c_last * C));
  __syncthreads();
  if (split == 0) {
    int32_t* out_rows = e.rows + (int64_t)unit * e.k;
    for (int i = tid; i < e.k; i += kFinishThreads) out_rows[i] = i < rows ? list[i] : -1;
    if (tid == 0) e.n_rows[unit] = rows;
  }
  const int qh0 = (unit % sa.Hkv) * G + split * GA;
  attn_wg<GA>(at, unit, LdsRows{list}, rows, 0, 1, lds, lds + Lds::kQOff, qh0);
}

// Co-batched dual-token attention over an assembled buffer (Sec. 5.2) when
// two workgroups per unit fit on the CUs: the unit's first workgroup attends
// with the current token's G heads, the second with the speculative token's,
// each over all of the unit's rows (buffer slots 0 .. n_sel - 1; the second
// read of a row mostly comes from the XCD's L2, both workgroups being on the
// same XCD), and each merges its token's own rows under the causal mask
// (current: row 0; speculative: rows 0 and 1) into its outputs.  No partials
// and no merge launch.
struct SlotRows {
  __device__ __forceinline__ int operator()(int i) const { return i; }
};

template <int G>
__global__ __launch_bounds__(kFinishThreads) void k_dual_token_wg(AttnArgs a, int units) {
  using Lds = WgAttnLds<G>;
  __shared__ __attribute__((aligned(16))) uint32_t lds[Lds::kStages + Lds::kQ];
  int unit, tok;
  split_block(blockIdx.x, 2, &unit, &tok);
  if (unit >= units) return;  // uniform over the workgroup
  AttnArgs t = a;
  t.max_ctx = a.k;  // the unit's buffer rows
  if (tok) {
    t.q = a.q2;
    t.out = a.out2;
  }
  const int n = clamp_len(a.n_sel[unit], a.k);
  const uint16_t* kl = a.k_local + (int64_t)unit * 2 * kD;
  const uint16_t* vl = a.v_local + (int64_t)unit * 2 * kD;
  attn_wg<G>(t, unit, SlotRows{}, n, 0, 1, lds, lds + Lds::kStages, (unit % a.Hkv) * G, kl, vl,
             tok ? 2 : 1);
}

// ---- read-rate probe --------------------------------------------------------
// Reads rows pos(i0) .. pos(i1) of a unit (positions clamped to the unit's
// rows) as the attention does: 4 rows per load instruction, K and V of a
// block of 16 rows, the next block requested once the current one is in
// (one block in flight per wave); a checksum stands for the arithmetic.
template <class Rows>
__device__ __forceinline__ uint32_t probe_rows(const ProbeArgs& a, int unit, Rows pos, int i0,
                                               int i1) {
  const int lane = threadIdx.x & 63;
  const int lrow = lane >> 4, lchunk = lane & 15;
  const int64_t ubase = (int64_t)unit * a.max_ctx * a.row_stride + 8 * lchunk;
  uint4 kr[4], vr[4];
  auto load = [&](int b) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      int p = pos(min(b + 4 * it + lrow, i1));
      p = p < 0 ? 0 : (p >= a.max_ctx ? a.max_ctx - 1 : p);
      const int64_t off = ubase + (int64_t)p * a.row_stride;
      kr[it] = ld16(a.k_rows + off);
      vr[it] = ld16(a.v_rows + off);
    }
  };
  uint32_t acc = 0u;
  load(i0);
  for (int b = i0; b <= i1; b += 16) {  // bounds uniform over the wave
#pragma unroll
    for (int it = 0; it < 4; ++it)
      acc ^= kr[it].x ^ kr[it].y ^ kr[it].z ^ kr[it].w ^ vr[it].x ^ vr[it].y ^ vr[it].z ^ vr[it].w;
    if (b + 16 <= i1) load(b + 16);
  }
  return acc;
}

struct GlobalRows {
  const int32_t* p;
  __device__ __forceinline__ int operator()(int i) const { return p[i]; }
};

// MODE CKV_PROBE_STANDALONE: k_attn's grid (one kAttnThreads workgroup per
// kAttnRows rows, kAttnRows / 4 rows per wave, indices from global memory).
// Otherwise the fused same-step launch's: two kFinishThreads workgroups per
// unit with its LDS (one per CU) and its workgroup -> (unit, part) mapping,
// positions staged in LDS, each wave a contiguous run of 16-row blocks of the
// part's rows (its half of the set, or all of it).
template <int MODE>
__global__ __launch_bounds__(MODE == CKV_PROBE_STANDALONE ? kAttnThreads : kFinishThreads) void
k_probe_rows(ProbeArgs a) {
  const int tid = threadIdx.x, wave = tid >> 6;
  uint32_t acc = 0u;
  if constexpr (MODE == CKV_PROBE_STANDALONE) {
    // LDS that leaves two workgroups per CU, the attention kernel's residency
    // (its registers allow two waves per SIMD)
    __shared__ uint32_t lds[18 * 1024];
    if (tid == 0) lds[blockIdx.x & 1023] = 0u;
    const int chunks = (a.k + kAttnRows - 1) / kAttnRows;
    const int unit = blockIdx.x / chunks, c = blockIdx.x - unit * chunks;
    constexpr int kRowsPerWave = kAttnRows / (kAttnThreads / 64);
    const int i0 = c * kAttnRows + wave * kRowsPerWave;
    const int i1 = min(i0 + kRowsPerWave, a.k) - 1;
    if (i0 <= i1) acc = probe_rows(a, unit, GlobalRows{a.idx + (int64_t)unit * a.k}, i0, i1);
    __syncthreads();
    if (a.k < 0) acc ^= lds[(tid + 1) & 1023];  // never (k >= 1): keeps the LDS allocated
    a.sink[(int64_t)blockIdx.x * kAttnThreads + tid] = acc;
  } else {
    __shared__ __attribute__((aligned(16))) uint32_t lds[SelAttnLds<4>::kDwords];
    int unit, part;
    split_block(blockIdx.x, 2, &unit, &part);
    if (unit < a.units) {  // uniform over the workgroup
      int lo = 0, hi = a.k;
      if (MODE == CKV_PROBE_ROW_HALVES) share_range(a.k, part, 2, &lo, &hi);
      int32_t* pos = reinterpret_cast<int32_t*>(lds);
      for (int i = lo + tid; i < hi; i += kFinishThreads) pos[i - lo] = a.idx[(int64_t)unit * a.k + i];
      __syncthreads();
      constexpr int kW = kFinishThreads / 64;
      const int nblk = (hi - lo + 15) >> 4;
      const int b0 = (wave * nblk) / kW, b1 = ((wave + 1) * nblk) / kW;
      if (b0 < b1) acc = probe_rows(a, unit, LdsRows{pos}, 16 * b0, min(16 * b1, hi - lo) - 1);
    }
    a.sink[(int64_t)blockIdx.x * kFinishThreads + tid] = acc;
  }
}

// ---- debug-mode input check -------------------------------------------------
__global__ __launch_bounds__(256) void k_check(CheckArgs a) {
  const int64_t U = (int64_t)a.B * a.Hkv;
  const int64_t total = a.B + U + (a.idx ? U * a.k : 0);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
    unsigned long long code = ~0ull;
    if (t < a.B) {
      if (a.ctx_lens) {
        const int v = a.ctx_lens[t];
        if (v < 0 || v > a.max_ctx) code = (1ull << 40) | (unsigned long long)t;
      }
    } else if (t < a.B + U) {
      const int64_t u = t - a.B;
      if (a.n_sel) {
        const int v = a.n_sel[u];
        if (v < 0 || v > a.k) code = (2ull << 40) | (unsigned long long)u;
      }
    } else {
      const int64_t e = t - a.B - U, u = e / a.k;
      const int i = (int)(e - u * a.k);
      const int count = a.n_sel ? min(max(a.n_sel[u], 0), a.k) : a.k;
      if (i < count) {
        const int bound = a.ctx_lens ? min(max(a.ctx_lens[u / a.Hkv], 0), a.max_ctx) : a.max_ctx;
        const int v = a.idx[e];
        if (v != -1 && (v < 0 || v >= bound)) code = (3ull << 40) | (unsigned long long)e;
      }
    }
    if (code != ~0ull) atomicMin(a.flag, code);
  }
}

// ---- attention -------------------------------------------------------------
template <int G, bool INDEXED>
__global__ __launch_bounds__(kAttnThreads) void k_attn(AttnArgs a) {
  __shared__ float lds[AttnLds<G>::kFloats];
  const int unit = blockIdx.x / a.chunks;
  const int chunk = blockIdx.x - unit * a.chunks;
  attn_chunk<G, INDEXED>(a, unit, chunk, lds);
}

// The scoring role of a pipelined launch: claims from a.claim (CLAIMS),
// else the static ranges, each wave with half a group in flight.  They are
// separate kernels so that each keeps its own register allocation.
template <int G, bool CLAIMS>
__device__ __forceinline__ void score_role(const ScoreArgs& a, int wg, int nwg, uint32_t* lds_hist,
                                           uint32_t* lds_stage, uint32_t* lds_claim) {
  if constexpr (CLAIMS)
    score_claims<G>(a, nwg, lds_hist, lds_stage, lds_claim);
  else
    score_range<G, true, 4, true>(a, wg, nwg, lds_hist, lds_stage);
}

// One launch, two roles (pipelined decode): the first attn_blocks workgroups
// attend with q_att over the buffer assembled for this step, the rest score
// the context with q_sel for the next step's selection.
template <int G, bool INDEXED, bool CLAIMS>
__global__ __launch_bounds__(kAttnThreads) void k_dual(AttnArgs at, ScoreArgs sc,
                                                      int attn_blocks) {
  static_assert(kAttnThreads == kScoreThreads, "roles share the block size");
  constexpr int kA = AttnLds<G>::kFloats;
  constexpr int kS = kHistBins + kScoreLdsDwords;
  __shared__ __attribute__((aligned(16))) float lds[kA > kS ? kA : kS];
  __shared__ uint32_t lds_claim[2];
  if ((int)blockIdx.x < attn_blocks) {
    const int unit = blockIdx.x / at.chunks;
    attn_chunk<G, INDEXED>(at, unit, blockIdx.x - unit * at.chunks, lds);
  } else {
    uint32_t* l32 = reinterpret_cast<uint32_t*>(lds);
    score_role<G, CLAIMS>(sc, blockIdx.x - attn_blocks, gridDim.x - attn_blocks, l32 + kScoreLdsDwords,
                  l32, lds_claim);
  }
}

// The same with a third role for the decode loop: the first sel_blocks
// workgroups select the previous layer's sets for the next step (sel: that
// layer's selection over the scores and per-workgroup histogram slots its
// own launch left), as the fused selection does but with kAttnThreads
// threads and the first kDualSelCands candidates in LDS.  Those sets are not
// needed before the next step, so the selection's latency-bound work runs
// beside this layer's streams instead of as a launch between layers.  TWO:
// the attention role has the 2G head rows of two tokens, as in k_dual2.
constexpr int kDualSelCands = 7168;
template <int G, bool INDEXED, bool TWO = false>
__global__ __launch_bounds__(kAttnThreads) void k_dual_sel(AttnArgs at, ScoreArgs sc,
                                                          SelectArgs sel, int attn_blocks,
                                                          int sel_blocks) {
  constexpr int GA = TWO ? 2 * G : G;  // attention head rows
  constexpr int kA = AttnLds<GA>::kFloats;
  constexpr int kS = kHistBins + kScoreLdsDwords;
  constexpr int kL = kA > kS ? kA : kS;
  static_assert(2 * kDualSelCands + kFusedSelectMaxCtx / 32 + 2048 <= kL,
                "the selection role's candidates, bitmap and histogram fit");
  __shared__ __attribute__((aligned(16))) float lds[kL];
  __shared__ uint32_t tmp[kAttnThreads / 64 + 1];
  __shared__ uint32_t misc[8];
  uint32_t* l32 = reinterpret_cast<uint32_t*>(lds);
  int blk = blockIdx.x;
  if (blk < sel_blocks) {
    const SelLds L{reinterpret_cast<uint2*>(l32), l32 + 2 * kDualSelCands,
                   l32 + 2 * kDualSelCands + kFusedSelectMaxCtx / 32, tmp, misc};
    select_unit<kAttnThreads, kDualSelCands>(sel, blk, L, true, nullptr, 0, 0, false);
    return;
  }
  blk -= sel_blocks;
  if (blk < attn_blocks) {
    const int unit = blk / at.chunks;
    attn_chunk<GA, INDEXED>(at, unit, blk - unit * at.chunks, lds);
  } else {
    score_range<G, true, 4, true>(sc, blk - attn_blocks, gridDim.x - sel_blocks - attn_blocks,
                                  l32 + kScoreLdsDwords, l32);
  }
}

// The same with two tokens (Sec. 5.2, dual-token decoding): the attention
// role has the 2G head rows of the current and the speculative token (the
// merge kernel adds their own rows under the causal mask), the scoring role
// the speculative token's G heads.
template <int G, bool INDEXED, bool CLAIMS>
__global__ __launch_bounds__(kAttnThreads) void k_dual2(AttnArgs at, ScoreArgs sc,
                                                       int attn_blocks) {
  constexpr int kA = AttnLds<2 * G>::kFloats;
  constexpr int kS = kHistBins + kScoreLdsDwords;
  __shared__ __attribute__((aligned(16))) float lds[kA > kS ? kA : kS];
  __shared__ uint32_t lds_claim[2];
  if ((int)blockIdx.x < attn_blocks) {
    const int unit = blockIdx.x / at.chunks;
    attn_chunk<2 * G, INDEXED>(at, unit, blockIdx.x - unit * at.chunks, lds);
  } else {
    uint32_t* l32 = reinterpret_cast<uint32_t*>(lds);
    score_role<G, CLAIMS>(sc, blockIdx.x - attn_blocks, gridDim.x - attn_blocks, l32 + kScoreLdsDwords,
                  l32, lds_claim);
  }
}

// Merges the chunk partials of every query head into the output.  The
// per-chunk (max, weight sum) pairs go through LDS first so that each thread's
// loads of the weighted sums are independent of one another.  With two tokens
// the tokens' own rows join the merge as one more partial each (Sec. 5.2:
// the current token sees its own row, the speculative token both rows).
template <int G>
__global__ __launch_bounds__(kAttnThreads) void k_combine(AttnArgs a) {
  constexpr int kMaxChunks = 64;
  __shared__ float s_m[G][kMaxChunks], s_w[G][kMaxChunks], s_inv[G], s_loc[G][2];
  const int unit = blockIdx.x;
  const int b = unit / a.Hkv, h = unit - b * a.Hkv;
  const float* pu = a.part + (int64_t)unit * a.chunks * G * kPartStride;
  const int tid = threadIdx.x;
  const bool dual = a.q2 != nullptr;
  const int Gq = dual ? G / 2 : G;
  auto out_row = [&](int g) {
    if (!dual) return a.out + ((int64_t)b * a.Hq + (int64_t)h * G + g) * kD;
    return g < Gq ? a.out + ((int64_t)b * a.Hq + (int64_t)h * Gq + g) * kD
                  : a.out2 + ((int64_t)b * a.Hq + (int64_t)h * Gq + g - Gq) * kD;
  };
  // logits of the local rows each head row sees (-inf where masked)
  if (tid < 2 * G) {
    const int g = tid >> 1, j = tid & 1;
    float lg = -INFINITY;
    if (dual && (j == 0 || g >= Gq)) {
      const uint16_t* q = (g < Gq ? a.q : a.q2) +
                          ((int64_t)b * a.Hq + (int64_t)h * Gq + (g < Gq ? g : g - Gq)) * kD;
      const uint16_t* kr = a.k_local + ((int64_t)unit * 2 + j) * kD;
      float dot = 0.f;
      for (int c = 0; c < kD; c += 8) {
        float qf[8], kf[8];
        unpack8(ld16(q + c), qf);
        unpack8(ld16(kr + c), kf);
#pragma unroll
        for (int e = 0; e < 8; ++e) dot = fmaf(qf[e], kf[e], dot);
      }
      lg = dot * a.scale;
    }
    s_loc[g][j] = lg;
  }
  if (a.chunks <= kMaxChunks) {
    const int nc = a.chunks;
    // With at most kMergeChunks partials, every thread's weighted sums are
    // loaded first, with the (max, weight sum) pairs, so the merge waits for
    // one round trip: unconditional loads of clamped chunks and outputs,
    // used only where valid.
    constexpr int kPer = (G * kD + kAttnThreads - 1) / kAttnThreads;
    const bool pre = nc <= kMergeChunks;
    float opre[kPer][kMergeChunks];
    if (pre) {
#pragma unroll
      for (int r = 0; r < kPer; ++r) {
        const int o = min(tid + r * kAttnThreads, G * kD - 1);
        const int g = o / kD, c = o - g * kD;
#pragma unroll
        for (int ch = 0; ch < kMergeChunks; ++ch)
          opre[r][ch] = pu[(min(ch, nc - 1) * G + g) * kPartStride + 4 + c];
      }
    }
    for (int i = tid; i < nc * G; i += kAttnThreads) {
      const int ch = i / G, g = i - ch * G;
      s_m[g][ch] = pu[(ch * G + g) * kPartStride];
      s_w[g][ch] = pu[(ch * G + g) * kPartStride + 1];
    }
    __syncthreads();
    if (tid < G) {  // per head: global max, chunk and local weights, 1/L
      const int g = tid;
      float M = fmaxf(s_loc[g][0], s_loc[g][1]);
      for (int ch = 0; ch < nc; ++ch) M = fmaxf(M, s_m[g][ch]);
      float L = 0.f;
      for (int ch = 0; ch < nc; ++ch) {
        const float w = s_m[g][ch] == -INFINITY ? 0.f : __expf(s_m[g][ch] - M);
        L = fmaf(w, s_w[g][ch], L);
        s_m[g][ch] = w;
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const float w = s_loc[g][j] == -INFINITY ? 0.f : __expf(s_loc[g][j] - M);
        L += w;
        s_loc[g][j] = w;
      }
      s_inv[g] = L > 0.f ? 1.f / L : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int o = tid + r * kAttnThreads;
      if (o >= G * kD) break;
      const int g = o / kD, c = o - g * kD;
      float O = 0.f;  // empty chunks carry weight 0 and zero sums
      if (pre) {
#pragma unroll
        for (int ch = 0; ch < kMergeChunks; ++ch)
          if (ch < nc) O = fmaf(s_m[g][ch], opre[r][ch], O);
      } else {
        for (int ch = 0; ch < nc; ++ch)
          O = fmaf(s_m[g][ch], pu[(ch * G + g) * kPartStride + 4 + c], O);
      }
      if (dual)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          O = fmaf(s_loc[g][j],
                   __uint_as_float((uint32_t)a.v_local[((int64_t)unit * 2 + j) * kD + c] << 16),
                   O);
      out_row(g)[c] = O * s_inv[g];
    }
    return;
  }
  // More chunks than fit in LDS: straightforward per-output loop.
  __syncthreads();
  for (int o = tid; o < G * kD; o += kAttnThreads) {
    const int g = o / kD, c = o - g * kD;
    float M = fmaxf(s_loc[g][0], s_loc[g][1]);
    for (int ch = 0; ch < a.chunks; ++ch) M = fmaxf(M, pu[(ch * G + g) * kPartStride]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
      for (int ch = 0; ch < a.chunks; ++ch) {
        const float* p = pu + (ch * G + g) * kPartStride;
        if (p[0] == -INFINITY) continue;
        const float w = __expf(p[0] - M);
        L = fmaf(w, p[1], L);
        O = fmaf(w, p[4 + c], O);
      }
      for (int j = 0; j < 2; ++j) {
        if (s_loc[g][j] == -INFINITY) continue;
        const float w = __expf(s_loc[g][j] - M);
        L += w;
        O = fmaf(w,
                 __uint_as_float((uint32_t)a.v_local[((int64_t)unit * 2 + j) * kD + c] << 16),
                 O);
      }
    }
    out_row(g)[c] = L > 0.f ? O / L : 0.f;
  }
}

// ---- chunk landmarks -----------------------------------------------------------
// Nearest bf16 to x, ties to the even significand, from the binary64 fields:
// normal results keep 7 of the 52 stored significand bits; below the
// smallest normal bf16 (2^-126) the quantum is 2^-133.
__device__ __forceinline__ uint16_t f64_to_bf16_rne(double x) {
  uint64_t b = (uint64_t)__double_as_longlong(x);
  const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
  b &= 0x7fffffffffffffffull;
  if (b == 0) return sign;
  if ((int)(b >> 52) < 1023 - 126) {
    const double r = rint(__longlong_as_double((long long)b) * 0x1p133);
    return (uint16_t)(sign | (uint16_t)r);  // r = 128 is the smallest normal
  }
  b += 0x00000fffffffffffull + ((b >> 45) & 1u);  // 2^44 - 1 + kept lsb
  const uint32_t e = (uint32_t)(b >> 52) - 1023u + 127u;
  return (uint16_t)(sign | (e << 7) | (uint32_t)((b >> 45) & 0x7fu));
}

// One item = 8 channels of one landmark: the fp64 sum of the chunk's rows
// below n_b in row order, divided by their count, rounded once to bf16.
__global__ __launch_bounds__(kGatherThreads) void k_landmarks(LandmarkArgs a) {
  const int64_t stride = (int64_t)gridDim.x * kGatherThreads;
  for (int64_t it = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x; it < a.items;
       it += stride) {
    const int part = (int)(it & 15);
    const int64_t uc = it >> 4;
    const int64_t unit = uc / a.cmax;
    const int c = (int)(uc - unit * a.cmax);
    const int n = clamp_len(a.ctx_lens[unit / a.Hkv], a.max_ctx);
    const int j0 = c * a.chunk;
    if (j0 >= n) continue;
    const int j1 = min(j0 + a.chunk, n);
    const uint16_t* src = a.keys + (unit * a.max_ctx + j0) * a.key_stride + 8 * part;
    double sum[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = j0; j < j1; ++j, src += a.key_stride) {
      float f[8];
      unpack8(ld16(src), f);
#pragma unroll
      for (int e = 0; e < 8; ++e) sum[e] += (double)f[e];
    }
    const double cnt = (double)(j1 - j0);
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = (uint32_t)f64_to_bf16_rne(sum[2 * e] / cnt) |
             ((uint32_t)f64_to_bf16_rne(sum[2 * e + 1] / cnt) << 16);
    *reinterpret_cast<uint4*>(a.landmarks + uc * kD + 8 * part) =
        make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// Row i of a unit's expanded set is row t = i % chunk of its (i / chunk)-th
// selected chunk; chunks are ascending, so only the last one can run past n_b
// and the valid rows form a prefix.
__global__ __launch_bounds__(kGatherThreads) void k_expand(ExpandArgs a) {
  const int unit = blockIdx.y;
  const int i = blockIdx.x * kGatherThreads + threadIdx.x;
  const int n = clamp_len(a.ctx_lens[unit / a.Hkv], a.max_ctx);
  const int m = clamp_len(a.n_chunks[unit], a.kc);
  const int32_t* ci = a.chunk_idx + (int64_t)unit * a.kc;
  if (i < a.k) {
    const int c = i / a.chunk;
    int row = -1;
    if (c < m) {
      row = ci[c] * a.chunk + (i - c * a.chunk);
      if (row >= n) row = -1;
    }
    a.rows[(int64_t)unit * a.k + i] = row;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0)
    a.n_rows[unit] =
        m == 0 ? 0 : (m - 1) * a.chunk + max(0, min(a.chunk, n - ci[m - 1] * a.chunk));
}

// ---- low-rank key reconstruction -------------------------------------------------
// One item = 8 channels of one rebuilt key: the fp64 sum over the rank in
// ascending order (bf16 products are exact in fp64), rounded once to bf16.
__device__ __forceinline__ void reconstruct_range(const ReconArgs& a, int blk, int nblk) {
  const int64_t stride = (int64_t)nblk * kGatherThreads;
  for (int64_t it = (int64_t)blk * kGatherThreads + threadIdx.x; it < a.items;
       it += stride) {
    const int part = (int)(it & 15);
    const int64_t slot = it >> 4;
    const int64_t unit = slot / a.k;
    const int i = (int)(slot - unit * a.k);
    if (i >= clamp_len(a.n_sel[unit], a.k)) continue;
    const int row = a.idx[slot];
    const int di = a.slots ? a.slots[slot] : i;
    if (row < 0 || row >= a.max_ctx || di < 0 || di >= a.k) continue;
    const uint16_t* u = a.u_fac + (unit * a.max_ctx + row) * a.rank;
    const uint16_t* w = a.w_fac + unit * a.rank * kD + 8 * part;
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int j = 0; j < a.rank; ++j) {
      const double uj = (double)__uint_as_float((uint32_t)u[j] << 16);
      float wf[8];
      unpack8(ld16(w + (int64_t)j * kD), wf);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += uj * (double)wf[e];
    }
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = (uint32_t)f64_to_bf16_rne(acc[2 * e]) |
             ((uint32_t)f64_to_bf16_rne(acc[2 * e + 1]) << 16);
    *reinterpret_cast<uint4*>(a.k_dst + (unit * a.k + di) * kD + 8 * part) =
        make_uint4(o[0], o[1], o[2], o[3]);
  }
}

__global__ __launch_bounds__(kGatherThreads) void k_reconstruct(ReconArgs a) {
  reconstruct_range(a, blockIdx.x, gridDim.x);
}

// ---- miss detection -----------------------------------------------------------
// First index i in [0, n) with a[i] >= v (a ascending).
template <class P>
__device__ __forceinline__ int lower_bound_i32(P a, int n, int v) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// One unit: which rows of the selected set (T, nt) the buffer already holds
// (the predicted set P, np, in slot order), and where the others go.  Free
// slots are those whose predicted row is not selected, then slots np..nt-1;
// there are at least as many as misses.  Miss r (in set order) takes the r-th
// free slot.  T/P/F are LDS arrays or the global sets, per IN_LDS.
template <bool IN_LDS>
__device__ __forceinline__ void miss_unit(const MissArgs& a, int unit, const int32_t* T,
                                          const int32_t* P, int32_t* F, int nt, int np,
                                          uint32_t* tmp) {
  const int k = a.k, tid = threadIdx.x;
  const int64_t base = (int64_t)unit * k;
  const int ns = max(np, nt);
  uint32_t nfree = 0;
  for (int s0 = 0; s0 < ns; s0 += kMissThreads) {
    const int sl = s0 + tid;
    bool fr = false;
    if (sl < ns) {
      if (sl < np) {
        const int pos = P[sl];
        const int j = lower_bound_i32(T, nt, pos);
        fr = !(j < nt && T[j] == pos);
      } else {
        fr = true;
      }
    }
    uint32_t total;
    const uint32_t incl = block_incl_scan<kMissThreads / 64>(fr ? 1u : 0u, tmp, &total);
    if (fr) F[nfree + incl - 1] = sl;
    nfree += total;
  }
  __syncthreads();  // the free list is complete
  uint32_t nmiss = 0;
  for (int i0 = 0; i0 < nt; i0 += kMissThreads) {
    const int i = i0 + tid;
    bool miss = false;
    int slot = -1, pos = 0;
    if (i < nt) {
      pos = T[i];
      const int j = lower_bound_i32(P, np, pos);
      if (j < np && P[j] == pos) slot = j;
      else miss = true;
    }
    uint32_t total;
    const uint32_t incl = block_incl_scan<kMissThreads / 64>(miss ? 1u : 0u, tmp, &total);
    if (miss) {
      const uint32_t r = nmiss + incl - 1;  // < nfree
      slot = F[r];
      a.miss_pos[base + r] = pos;
      a.miss_slot[base + r] = slot;
    }
    if (i < nt) a.slot_of[base + i] = slot;
    nmiss += total;
  }
  if (tid == 0) {
    a.n_miss[unit] = (int32_t)nmiss;
    a.hits[unit] = nt - (int32_t)nmiss;
  }
}

__global__ __launch_bounds__(kMissThreads) void k_miss(MissArgs a) {
  __shared__ int32_t l_true[kMissLds], l_pred[kMissLds], l_free[kMissLds];
  __shared__ uint32_t tmp[kMissThreads / 64 + 1];
  const int unit = blockIdx.x, k = a.k;
  const int nt = clamp_len(a.n_true[unit], k), np = clamp_len(a.n_pred[unit], k);
  const int32_t* gt = a.idx_true + (int64_t)unit * k;
  const int32_t* gp = a.idx_pred + (int64_t)unit * k;
  if (k <= kMissLds) {  // uniform
    for (int i = threadIdx.x; i < nt; i += kMissThreads) l_true[i] = gt[i];
    for (int i = threadIdx.x; i < np; i += kMissThreads) l_pred[i] = gp[i];
    __syncthreads();
    miss_unit<true>(a, unit, l_true, l_pred, l_free, nt, np, tmp);
  } else {
    miss_unit<false>(a, unit, gt, gp, a.free_slot + (int64_t)unit * k, nt, np, tmp);
  }
}

// ---- gather ----------------------------------------------------------------
// Item it = ((unit*k + slot)*2 + kv)*16 + part moves 16 bytes; the 32 items of
// one slot are its K row then its V row (contiguous for K|V interleaved rows).
// With a slot list, entry slot of the unit lands in slot slots[unit][slot].
// K items are skipped when k_dst is NULL.
__device__ __forceinline__ void gather_range(const GatherArgs& a, int blk, int nblk) {
  const int64_t step = (int64_t)nblk * kGatherThreads * kGatherUnroll;
  for (int64_t it0 = (int64_t)blk * kGatherThreads * kGatherUnroll; it0 < a.items;
       it0 += step) {
    uint4 v[kGatherUnroll];
    uint16_t* dst[kGatherUnroll];
#pragma unroll
    for (int u = 0; u < kGatherUnroll; ++u) {
      const int64_t it = it0 + u * kGatherThreads + threadIdx.x;
      dst[u] = nullptr;
      if (it < a.items) {
        const int part = (int)(it & 15);
        const int kv = (int)((it >> 4) & 1);
        const int64_t slot = it >> 5;
        const int64_t unit = slot / a.k;
        const int i = (int)(slot - unit * a.k);
        if (i < a.n_sel[unit]) {
          const int pos = a.idx[slot];
          const int di = a.slots ? a.slots[slot] : i;
          if (pos >= 0 && pos < a.max_ctx && di >= 0 && di < a.k && (kv || a.k_dst)) {
            const uint16_t* src = (kv ? a.v_src : a.k_src) +
                                  (unit * a.max_ctx + pos) * a.row_stride + part * 8;
            v[u] = ld16(src);
            dst[u] = (kv ? a.v_dst : a.k_dst) + (unit * a.k + di) * kD + part * 8;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kGatherUnroll; ++u)
      if (dst[u]) *reinterpret_cast<uint4*>(dst[u]) = v[u];
  }
}

__global__ __launch_bounds__(kGatherThreads) void k_gather(GatherArgs a) {
  gather_range(a, blockIdx.x, gridDim.x);
}

// Misses of a layer with key reconstruction: the first `nfetch` workgroups
// fetch the missing values while the others rebuild the missing keys, so the
// transfer and the arithmetic overlap in one launch.
__global__ __launch_bounds__(kGatherThreads) void k_miss_fill(GatherArgs g, ReconArgs r,
                                                              int nfetch) {
  if ((int)blockIdx.x < nfetch)
    gather_range(g, blockIdx.x, nfetch);
  else
    reconstruct_range(r, blockIdx.x - nfetch, gridDim.x - nfetch);
}

// ---- fixed scratch for callers that cannot allocate -------------------------
// The workspace of ckv_critical_kv_attn_noalloc: one array per device, held
// for the life of the process.  Its name is a host-side stand-in in host
// code, never an address: the device address of each device's copy is asked
// of the runtime once, with that device current, and only that address is
// passed to kernels.
static __device__ __align__(256) uint8_t scratch[CKV_NOALLOC_SCRATCH_BYTES];

int noalloc_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "current device");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CKV_EUNSUPPORTED, "device %d (the fixed scratch serves devices below %d)", dev,
                kMaxDevices);
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "device address of the fixed scratch");
    if (!p) return fail(CKV_EHIP, "device address of the fixed scratch is NULL");
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return CKV_OK;
}

// ---- launchers ---------------------------------------------------------------
static inline int blocks_for(int64_t n, int per, int cap) {
  int64_t b = (n + per - 1) / per;
  if (b < 1) b = 1;
  return (int)(b > cap ? cap : b);
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 == 0) return hipSuccess;
  launch_kernel(CKV_K_ZERO, k_zero, dim3(blocks_for(n16, 256 * 4, 2048)), dim3(256), s,
                reinterpret_cast<uint4*>(p), n16);
  return launch_status();
}

hipError_t launch_fill(void* p, size_t bytes, uint32_t pattern, hipStream_t s) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 == 0) return hipSuccess;
  launch_kernel(CKV_K_ZERO, k_fill, dim3(blocks_for(n16, 256 * 4, 2048)), dim3(256), s,
                reinterpret_cast<uint4*>(p), n16, pattern);
  return launch_status();
}

// Workgroups of a kernel of `threads` threads that fit on the device at once,
// per (kernel, device): queried once and kept in a fixed table (no allocation
// on the call path), so a call makes no occupancy query.  The persistent
// scoring grid is this many workgroups (or fewer if there is less work).
static int resident_blocks(const void* fn, int threads = kScoreThreads) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 1024;
  struct Entry {
    const void* fn;
    int dev, blocks;
  };
  constexpr int kEntries = 512;
  static Entry table[kEntries];
  static int used = 0;
  static std::mutex mu;
  {
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < used; ++i)
      if (table[i].fn == fn && table[i].dev == dev) return table[i].blocks;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus < 1)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) !=
          hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  std::lock_guard<std::mutex> lk(mu);
  if (used < kEntries) table[used++] = Entry{fn, dev, cus * per_cu};
  return cus * per_cu;
}

int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  static std::mutex mu;
  static int cus[kMaxDevices] = {};
  std::lock_guard<std::mutex> lk(mu);
  if (!cus[dev]) {
    int c = 0;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c < 1)
      c = 256;
    cus[dev] = c;
  }
  return cus[dev];
}

// The kernel whose residency sets a scoring grid (the claim variants of the
// pipelined kernels have the same block size and LDS, so the same residency).
template <int G>
static const void* score_kernel(ScoreKind kind, int chunk) {
  switch (kind) {
    case ScoreKind::kPlain: return (const void*)k_score<G, false>;
    case ScoreKind::kHist:
      return chunk > 1 ? (const void*)k_score_chunks<G> : (const void*)k_score<G, true>;
    case ScoreKind::kDual: return (const void*)k_dual<G, false, false>;
    case ScoreKind::kDualIndexed: return (const void*)k_dual<G, true, false>;
    case ScoreKind::kDual2:
      if constexpr (G <= 8) return (const void*)k_dual2<G, false, false>;
      return nullptr;
    case ScoreKind::kDual2Indexed:
      if constexpr (G <= 8) return (const void*)k_dual2<G, true, false>;
      return nullptr;
    case ScoreKind::kDualSel: return (const void*)k_dual_sel<G, false>;
    case ScoreKind::kDualSelIndexed: return (const void*)k_dual_sel<G, true>;
    case ScoreKind::kDual2Sel:
      if constexpr (G <= 8) return (const void*)k_dual_sel<G, false, true>;
      return nullptr;
    case ScoreKind::kDual2SelIndexed:
      if constexpr (G <= 8) return (const void*)k_dual_sel<G, true, true>;
      return nullptr;
  }
  return nullptr;
}

// Whether a pipelined launch's scoring grid of nwg workgroups takes claims:
// when it adds its histograms, has a claim counter, and has at least
// kMinClaimsPerWg claims per workgroup (each workgroup holds two claims
// ahead, which idles workgroups at the end of a pass with fewer).
static bool use_claims(const ScoreArgs& a, int nwg) {
  if (!a.claim || a.hist_part) return false;
  const int64_t gu = (a.max_ctx + kStageRows - 1) / kStageRows;
  const int64_t claims = (int64_t)a.units * ((gu + kClaimGroups - 1) / kClaimGroups);
  return claims >= (int64_t)kMinClaimsPerWg * nwg;
}

int score_blocks(const ScoreArgs& a, int G, ScoreKind kind) {
  const void* fn = nullptr;
  switch (G) {
    case 1: fn = score_kernel<1>(kind, a.chunk); break;
    case 2: fn = score_kernel<2>(kind, a.chunk); break;
    case 4: fn = score_kernel<4>(kind, a.chunk); break;
    case 8: fn = score_kernel<8>(kind, a.chunk); break;
    case 16: fn = score_kernel<16>(kind, a.chunk); break;
    default: return 0;
  }
  if (!fn) return 0;
  const int64_t groups = (int64_t)a.units * ((a.max_ctx + kStageRows - 1) / kStageRows);
  const bool wide = kind == ScoreKind::kHist && a.chunk <= 1;  // k_score<G, true>
  int64_t slots = resident_blocks(fn, wide ? 64 * kHistScoreWaves : kScoreThreads);
  if (slots > kMaxScoreWgs) slots = kMaxScoreWgs;
  return (int)(groups < slots ? groups : slots);
}

template <int G>
static void launch_score_g(const ScoreArgs& a, bool hist, int nwg, hipStream_t s) {
  const dim3 grid(nwg), block(kScoreThreads);
  if (a.chunk > 1) launch_kernel(CKV_K_SCORE, k_score_chunks<G>, grid, block, s, a);
  else if (hist) launch_kernel(CKV_K_SCORE, k_score<G, true>, grid, dim3(64 * kHistScoreWaves), s, a);
  else launch_kernel(CKV_K_SCORE, k_score<G, false>, grid, block, s, a);
}

hipError_t launch_score(const ScoreArgs& a, int G, bool hist, int nwg, hipStream_t s) {
  if (nwg < 1 || nwg > kMaxScoreWgs) return hipErrorInvalidValue;
  switch (G) {
    case 1: launch_score_g<1>(a, hist, nwg, s); break;
    case 2: launch_score_g<2>(a, hist, nwg, s); break;
    case 4: launch_score_g<4>(a, hist, nwg, s); break;
    case 8: launch_score_g<8>(a, hist, nwg, s); break;
    case 16: launch_score_g<16>(a, hist, nwg, s); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

hipError_t launch_hist(const SelectArgs& a, int units, hipStream_t s) {
  launch_kernel(CKV_K_HIST, k_hist, dim3(units * a.tiles), dim3(kScoreThreads), s, a);
  return launch_status();
}

hipError_t launch_filter(const SelectArgs& a, int units, hipStream_t s) {
  launch_kernel(CKV_K_FILTER, k_filter, dim3(units * a.tiles), dim3(kFilterThreads), s, a);
  return launch_status();
}

hipError_t launch_finish(const SelectArgs& a, int units, hipStream_t s) {
  launch_kernel(CKV_K_FINISH, k_finish, dim3(units), dim3(kFinishThreads), s, a);
  return launch_status();
}

hipError_t launch_select_fused(const SelectArgs& a, int units, hipStream_t s) {
  launch_kernel(CKV_K_FINISH, k_select_fused, dim3(units), dim3(kFinishThreads), s, a);
  return launch_status();
}

template <int G>
static void launch_attn_g(const AttnArgs& a, bool indexed, int units, hipStream_t s) {
  const dim3 grid(units * a.chunks), block(kAttnThreads);
  if (indexed) launch_kernel(CKV_K_ATTN, k_attn<G, true>, grid, block, s, a);
  else launch_kernel(CKV_K_ATTN, k_attn<G, false>, grid, block, s, a);
}

hipError_t launch_attn(const AttnArgs& a, int G, bool indexed, int units, hipStream_t s) {
  switch (G) {
    case 1: launch_attn_g<1>(a, indexed, units, s); break;
    case 2: launch_attn_g<2>(a, indexed, units, s); break;
    case 4: launch_attn_g<4>(a, indexed, units, s); break;
    case 8: launch_attn_g<8>(a, indexed, units, s); break;
    case 16: launch_attn_g<16>(a, indexed, units, s); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

hipError_t launch_combine(const AttnArgs& a, int G, int units, hipStream_t s) {
  const dim3 grid(units), block(kAttnThreads);
  switch (G) {
    case 1: launch_kernel(CKV_K_COMBINE, k_combine<1>, grid, block, s, a); break;
    case 2: launch_kernel(CKV_K_COMBINE, k_combine<2>, grid, block, s, a); break;
    case 4: launch_kernel(CKV_K_COMBINE, k_combine<4>, grid, block, s, a); break;
    case 8: launch_kernel(CKV_K_COMBINE, k_combine<8>, grid, block, s, a); break;
    case 16: launch_kernel(CKV_K_COMBINE, k_combine<16>, grid, block, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

template <int G, bool INDEXED>
static void launch_dual_g(const AttnArgs& at, const ScoreArgs& sc, int attn_blocks, int nwg,
                          hipStream_t s) {
  if (use_claims(sc, nwg))
    launch_kernel(CKV_K_DUAL, k_dual<G, INDEXED, true>, dim3(attn_blocks + nwg),
                  dim3(kAttnThreads), s, at, sc, attn_blocks);
  else
    launch_kernel(CKV_K_DUAL, k_dual<G, INDEXED, false>, dim3(attn_blocks + nwg),
                  dim3(kAttnThreads), s, at, sc, attn_blocks);
}

template <bool INDEXED>
static hipError_t launch_dual_i(const AttnArgs& at, const ScoreArgs& sc, int G,
                                int attn_blocks, int nwg, hipStream_t s) {
  switch (G) {
    case 1: launch_dual_g<1, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 2: launch_dual_g<2, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 4: launch_dual_g<4, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 8: launch_dual_g<8, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 16: launch_dual_g<16, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

template <int G, bool INDEXED>
static void launch_dual2_g(const AttnArgs& at, const ScoreArgs& sc, int attn_blocks, int nwg,
                           hipStream_t s) {
  if (use_claims(sc, nwg))
    launch_kernel(CKV_K_DUAL, k_dual2<G, INDEXED, true>, dim3(attn_blocks + nwg),
                  dim3(kAttnThreads), s, at, sc, attn_blocks);
  else
    launch_kernel(CKV_K_DUAL, k_dual2<G, INDEXED, false>, dim3(attn_blocks + nwg),
                  dim3(kAttnThreads), s, at, sc, attn_blocks);
}

template <bool INDEXED>
static hipError_t launch_dual2_i(const AttnArgs& at, const ScoreArgs& sc, int G,
                                 int attn_blocks, int nwg, hipStream_t s) {
  switch (G) {
    case 1: launch_dual2_g<1, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 2: launch_dual2_g<2, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 4: launch_dual2_g<4, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    case 8: launch_dual2_g<8, INDEXED>(at, sc, attn_blocks, nwg, s); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

hipError_t launch_dual(const AttnArgs& at, const ScoreArgs& sc, int G, bool indexed,
                       int units, int nwg, hipStream_t s) {
  if (nwg < 1 || nwg > kMaxScoreWgs) return hipErrorInvalidValue;
  const int attn_blocks = units * at.chunks;
  if (at.q2)  // two tokens: 2G head rows attend, G score
    return indexed ? launch_dual2_i<true>(at, sc, G, attn_blocks, nwg, s)
                   : launch_dual2_i<false>(at, sc, G, attn_blocks, nwg, s);
  return indexed ? launch_dual_i<true>(at, sc, G, attn_blocks, nwg, s)
                 : launch_dual_i<false>(at, sc, G, attn_blocks, nwg, s);
}

template <bool INDEXED, bool TWO>
static hipError_t launch_dual_sel_i(const AttnArgs& at, const ScoreArgs& sc,
                                    const SelectArgs& sel, int G, int attn_blocks,
                                    int sel_blocks, int nwg, hipStream_t s) {
  const dim3 grid(sel_blocks + attn_blocks + nwg), block(kAttnThreads);
#define CKV_DS(g) launch_kernel(CKV_K_DUAL, k_dual_sel<g, INDEXED, TWO>, grid, block, s, at, sc, sel, attn_blocks, sel_blocks)
  switch (G) {
    case 1: CKV_DS(1); break;
    case 2: CKV_DS(2); break;
    case 4: CKV_DS(4); break;
    case 8: CKV_DS(8); break;
    case 16:
      if constexpr (!TWO) {
        CKV_DS(16);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
#undef CKV_DS
  return launch_status();
}

hipError_t launch_dual_sel(const AttnArgs& at, const ScoreArgs& sc, const SelectArgs& sel,
                           int G, bool indexed, int units, int nwg, hipStream_t s) {
  if (nwg < 1 || nwg > kMaxScoreWgs || !sc.hist_part || !sel.hist_part ||
      sel.max_ctx > kFusedSelectMaxCtx)
    return hipErrorInvalidValue;
  const int ab = units * at.chunks, sb = sel.units;
  if (at.q2)  // two tokens: 2G head rows attend, G score
    return indexed ? launch_dual_sel_i<true, true>(at, sc, sel, G, ab, sb, nwg, s)
                   : launch_dual_sel_i<false, true>(at, sc, sel, G, ab, sb, nwg, s);
  return indexed ? launch_dual_sel_i<true, false>(at, sc, sel, G, ab, sb, nwg, s)
                 : launch_dual_sel_i<false, false>(at, sc, sel, G, ab, sb, nwg, s);
}

hipError_t launch_select_attn(const SelectArgs& sa, const AttnArgs& at, int G, int nsplit,
                              int heads, const FusedSync* merge, hipStream_t s) {
  if (nsplit < 1 || nsplit > kSelAttnMaxSplit) return hipErrorInvalidValue;
  if (heads != 1 && (heads != 2 || nsplit != 1 || G % 2)) return hipErrorInvalidValue;
  if (merge && (heads != 1 || nsplit != 2 || !merge->merge || !at.part))
    return hipErrorInvalidValue;
  const int per = heads > 1 ? heads : nsplit;  // workgroups per unit
  const int blocks = per == 1 ? sa.units : (sa.units + 7) / 8 * 8 * per;
  const dim3 grid(blocks), block(kFinishThreads);
  const FusedSync fs = merge ? *merge : FusedSync{nullptr, nullptr, 0};
#define CKV_SA(g, hh) launch_kernel(CKV_K_SELECT_ATTN, k_select_attn<g, hh>, grid, block, s, sa, at, nsplit, fs)
#define CKV_SAM(g) launch_kernel(CKV_K_SELECT_ATTN, k_select_attn<g, 1, true>, grid, block, s, sa, at, nsplit, fs)
  if (merge) {
    switch (G) {
      case 1: CKV_SAM(1); break;
      case 2: CKV_SAM(2); break;
      case 4: CKV_SAM(4); break;
      case 8: CKV_SAM(8); break;
      default: return hipErrorInvalidValue;
    }
  } else if (heads == 1) {
    switch (G) {
      case 1: CKV_SA(1, 1); break;
      case 2: CKV_SA(2, 1); break;
      case 4: CKV_SA(4, 1); break;
      case 8: CKV_SA(8, 1); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (G) {
      case 2: CKV_SA(2, 2); break;
      case 4: CKV_SA(4, 2); break;
      case 8: CKV_SA(8, 2); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef CKV_SA
#undef CKV_SAM
  return launch_status();
}

template <int G>
static const void* critical_kernel(bool rows) {
  return rows ? (const void*)k_critical<G, true> : (const void*)k_critical<G, false>;
}

int critical_blocks(int G, int units, int nwg, bool rows) {
  if (units < 8 || units % 8 || nwg < 8 || nwg % 8) return 0;
  const void* fn = G == 2 ? critical_kernel<2>(rows) : G == 4 ? critical_kernel<4>(rows)
                 : G == 8 ? critical_kernel<8>(rows) : nullptr;
  // every scoring workgroup resident at once, so that none waits for a
  // workgroup that waits for it
  if (!fn || nwg > resident_blocks(fn, kFinishThreads)) return 0;
  return nwg + 2 * units;
}

hipError_t launch_critical(const ScoreArgs& sc, const SelectArgs& sa, const AttnArgs& at,
                           const FusedSync& fs, int G, int nwg, bool rows, hipStream_t s) {
  const int blocks = critical_blocks(G, sa.units, nwg, rows);
  if (!blocks || !sa.affine || sa.score_nwg != nwg || !sc.hist_part || (rows && !fs.merge) ||
      (rows && !at.part))
    return hipErrorInvalidValue;
  const dim3 grid(blocks), block(kFinishThreads);
#define CKV_CRITICAL(GG)                                                                        \
  rows ? launch_kernel(CKV_K_CRITICAL, k_critical<GG, true>, grid, block, s, sc, sa, at, fs, nwg) \
       : launch_kernel(CKV_K_CRITICAL, k_critical<GG, false>, grid, block, s, sc, sa, at, fs, nwg)
  switch (G) {
    case 2: CKV_CRITICAL(2); break;
    case 4: CKV_CRITICAL(4); break;
    case 8: CKV_CRITICAL(8); break;
    default: return hipErrorInvalidValue;
  }
#undef CKV_CRITICAL
  return launch_status();
}

hipError_t launch_select_attn_chunks(const SelectArgs& sa, const AttnArgs& at,
                                    const ExpandArgs& e, int G, hipStream_t s) {
  if (G % 2 || sa.k > kFinishThreads || e.k > kSelAttnMaxShare || e.chunk < 2)
    return hipErrorInvalidValue;
  const dim3 grid((sa.units + 7) / 8 * 8 * 2), block(kFinishThreads);
  switch (G) {
    case 2: launch_kernel(CKV_K_SELECT_ATTN, k_select_attn_chunks<2>, grid, block, s, sa, at, e); break;
    case 4: launch_kernel(CKV_K_SELECT_ATTN, k_select_attn_chunks<4>, grid, block, s, sa, at, e); break;
    case 8: launch_kernel(CKV_K_SELECT_ATTN, k_select_attn_chunks<8>, grid, block, s, sa, at, e); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

hipError_t launch_dual_token_wg(const AttnArgs& a, int G, int units, hipStream_t s) {
  const dim3 grid((units + 7) / 8 * 8 * 2), block(kFinishThreads);
  switch (G) {
    case 1: launch_kernel(CKV_K_ATTN, k_dual_token_wg<1>, grid, block, s, a, units); break;
    case 2: launch_kernel(CKV_K_ATTN, k_dual_token_wg<2>, grid, block, s, a, units); break;
    case 4: launch_kernel(CKV_K_ATTN, k_dual_token_wg<4>, grid, block, s, a, units); break;
    case 8: launch_kernel(CKV_K_ATTN, k_dual_token_wg<8>, grid, block, s, a, units); break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

size_t probe_sink_words(int64_t units, int k, int mode) {
  if (mode == CKV_PROBE_STANDALONE)
    return (size_t)units * ((k + kAttnRows - 1) / kAttnRows) * kAttnThreads;
  return (size_t)((units + 7) / 8 * 8 * 2) * kFinishThreads;
}

hipError_t launch_probe(const ProbeArgs& a, int mode, hipStream_t s) {
  switch (mode) {
    case CKV_PROBE_STANDALONE:
      launch_kernel(CKV_K_PROBE, k_probe_rows<CKV_PROBE_STANDALONE>,
                    dim3((unsigned)(a.units * ((a.k + kAttnRows - 1) / kAttnRows))),
                    dim3(kAttnThreads), s, a);
      break;
    case CKV_PROBE_ROW_HALVES:
      launch_kernel(CKV_K_PROBE, k_probe_rows<CKV_PROBE_ROW_HALVES>,
                    dim3((unsigned)((a.units + 7) / 8 * 8 * 2)), dim3(kFinishThreads), s, a);
      break;
    case CKV_PROBE_HEAD_HALVES:
      launch_kernel(CKV_K_PROBE, k_probe_rows<CKV_PROBE_HEAD_HALVES>,
                    dim3((unsigned)((a.units + 7) / 8 * 8 * 2)), dim3(kFinishThreads), s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return launch_status();
}

hipError_t launch_check(const CheckArgs& a, hipStream_t s) {
  const int64_t U = (int64_t)a.B * a.Hkv;
  const int64_t total = a.B + U + (a.idx ? U * a.k : 0);
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(k_check, dim3(blocks > 0 ? blocks : 1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_landmarks(const LandmarkArgs& a, hipStream_t s) {
  const int blocks = blocks_for(a.items, kGatherThreads, 8192);
  launch_kernel(CKV_K_LANDMARKS, k_landmarks, dim3(blocks), dim3(kGatherThreads), s, a);
  return launch_status();
}

hipError_t launch_reconstruct(const ReconArgs& a, hipStream_t s) {
  const int blocks = blocks_for(a.items, kGatherThreads, 8192);
  launch_kernel(CKV_K_RECONSTRUCT, k_reconstruct, dim3(blocks), dim3(kGatherThreads), s, a);
  return launch_status();
}

hipError_t launch_miss_fill(const GatherArgs& g, int fetch_blocks, const ReconArgs& r,
                            hipStream_t s) {
  const int nf = blocks_for(g.items, kGatherThreads * kGatherUnroll, fetch_blocks);
  const int nr = blocks_for(r.items, kGatherThreads, 8192);
  launch_kernel(CKV_K_RECONSTRUCT, k_miss_fill, dim3(nf + nr), dim3(kGatherThreads), s, g, r,
                nf);
  return launch_status();
}

hipError_t launch_expand(const ExpandArgs& a, int units, hipStream_t s) {
  const dim3 grid((a.k + kGatherThreads - 1) / kGatherThreads, units);
  launch_kernel(CKV_K_EXPAND, k_expand, grid, dim3(kGatherThreads), s, a);
  return launch_status();
}

hipError_t launch_miss(const MissArgs& a, int units, hipStream_t s) {
  launch_kernel(CKV_K_MISS, k_miss, dim3(units), dim3(kMissThreads), s, a);
  return launch_status();
}

hipError_t launch_gather(const GatherArgs& a, int max_blocks, hipStream_t s) {
  const int blocks = blocks_for(a.items, kGatherThreads * kGatherUnroll, max_blocks);
  launch_kernel(CKV_K_GATHER, k_gather, dim3(blocks), dim3(kGatherThreads), s, a);
  return launch_status();
}

}  // namespace ckv
