// ckv_topk.hpp -- GQA-aware top-k selection by radix select on fp32 order
// keys (Sec. 2.2: only the critical entries within the sparse budget are
// retrieved; one index set per KV head).
//
// Three passes, all exact:
//   1. histogram of the first digit (top 11 bits of the order key), fused
//      into the scoring pass or run over given scores;
//   2. filter (many workgroups per unit): positions whose first digit is
//      above the bin holding the m-th largest key are selected outright;
//      positions in that bin become candidates (order key, position);
//   3. finish (one workgroup per unit): radix select over the candidates on
//      the remaining 21 bits finds the exact threshold key T; ties at T are
//      resolved by lower position; the chosen positions are marked in a
//      bitmap and written out in ascending order.
#pragma once

#include "ckv_device.hpp"

namespace ckv {

// Wave 0 only: bin of the first digit that holds the m-th largest key, and
// the number of keys in higher bins.  out[0] = bin, out[1] = count above.
__device__ __forceinline__ void find_first_bin(const uint32_t* coarse,
                                               const uint32_t* hist,
                                               uint32_t m, uint32_t* out) {
  constexpr int kFine = kHistBins / kCoarseBins;  // fine bins per coarse bin
  static_assert(kCoarseBins == 64 && kFine <= 64, "one lane per bin");
  const int lane = threadIdx.x & 63;
  const uint32_t c = coarse[kCoarseBins - 1 - lane];  // descending bins
  const uint32_t s = wave_incl_scan(c);
  int L = __ffsll((unsigned long long)__ballot(s >= m)) - 1;
  if (L < 0) L = kCoarseBins - 1;  // only if the histogram were inconsistent
  const uint32_t above_c = __builtin_amdgcn_readlane(s - c, L);
  const int sb = kCoarseBins - 1 - L;
  const uint32_t f = lane < kFine ? hist[sb * kFine + kFine - 1 - lane] : 0u;
  const uint32_t s2 = wave_incl_scan(f) + above_c;
  int L2 = __ffsll((unsigned long long)__ballot(lane < kFine && s2 >= m)) - 1;
  if (L2 < 0) L2 = kFine - 1;
  const uint32_t above = __builtin_amdgcn_readlane(s2 - f, L2);
  if (lane == 0) {
    out[0] = (uint32_t)(sb * kFine + kFine - 1 - L2);
    out[1] = above;
  }
}

// Wave 0: lane l holds the count c of coarse range cb = 63 - l, whose 32 fine
// bins are at stage[cb*32 ..]; finds the bin holding the m-th largest key by
// two wave scans (ranges, then the chosen range's bins, both descending).
// out[0] = bin, out[1] = keys in higher bins, out[2] = keys in the bin.
__device__ __forceinline__ void walk_first_bin(const uint32_t* stage, uint32_t c, uint32_t m,
                                               uint32_t* out) {
  constexpr int kFine = kHistBins / 64;
  static_assert(kFine <= 64, "one lane per fine bin");
  const int lane = threadIdx.x & 63;
  const uint32_t s = wave_incl_scan(c);
  int L = __ffsll((unsigned long long)__ballot(s >= m)) - 1;
  if (L < 0) L = 63;  // only if the histogram were inconsistent
  const uint32_t above_c = __builtin_amdgcn_readlane(s - c, L);
  const int cb = 63 - L;
  const uint32_t f = lane < kFine ? stage[cb * kFine + kFine - 1 - lane] : 0u;
  const uint32_t s2 = wave_incl_scan(f) + above_c;
  int L2 = __ffsll((unsigned long long)__ballot(lane < kFine && s2 >= m)) - 1;
  if (L2 < 0) L2 = kFine - 1;  // the range's lowest bin
  const uint32_t above = __builtin_amdgcn_readlane(s2 - f, L2);
  const uint32_t in_bin = __builtin_amdgcn_readlane(f, L2);
  if (lane == 0) {
    out[0] = (uint32_t)(cb * kFine + kFine - 1 - L2);
    out[1] = above;
    out[2] = in_bin;
  }
}

// All NT threads: the first-digit histogram is the sum of nslots (1 ..
// kMaxPartials) consecutive slots of kHistBins counts.  Every thread loads
// its kHistBins / NT consecutive bins of every slot at once (one round trip;
// slots past nslots repeat slot 0 and are not added) ...
template <int NT = kFinishThreads, bool COH = false>
__device__ __forceinline__ void load_hist_slots(const uint32_t* hist, int nslots,
                                                uint2 (&v)[kMaxPartials][kHistBins / NT / 2]) {
  constexpr int kPairs = kHistBins / NT / 2;
  static_assert(kPairs >= 1, "two bins per thread at least");
  const int t = threadIdx.x;
#pragma unroll
  for (int p = 0; p < kMaxPartials; ++p)
#pragma unroll
    for (int q = 0; q < kPairs; ++q) {
      const uint32_t* src =
          hist + (int64_t)(p < nslots ? p : 0) * kHistBins + 2 * (kPairs * t + q);
      if constexpr (COH) {  // stored by other workgroups of the same launch
        const uint64_t w = __hip_atomic_load(reinterpret_cast<const uint64_t*>(src),
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        v[p][q] = make_uint2((uint32_t)w, (uint32_t)(w >> 32));
      } else {
        v[p][q] = *reinterpret_cast<const uint2*>(src);
      }
    }
}

// ... and stores the sums to lhist (LDS); the caller synchronises before
// reading it.
template <int NT = kFinishThreads>
__device__ __forceinline__ void store_hist_sum(const uint2 (&v)[kMaxPartials][kHistBins / NT / 2],
                                               int nslots, uint32_t* lhist) {
  constexpr int kPairs = kHistBins / NT / 2;
#pragma unroll
  for (int q = 0; q < kPairs; ++q) {
    uint2 acc = make_uint2(0u, 0u);
#pragma unroll
    for (int p = 0; p < kMaxPartials; ++p)
      if (p < nslots) {
        acc.x += v[p][q].x;
        acc.y += v[p][q].y;
      }
    *reinterpret_cast<uint2*>(lhist + 2 * (kPairs * threadIdx.x + q)) = acc;
  }
}

// Wave 0 only: the bin holding the m-th largest key, from the histogram in
// LDS (lhist).  out[0] = bin, out[1] = keys in higher bins, out[2] = keys in
// the bin.
__device__ __forceinline__ void find_first_bin_lds(const uint32_t* lhist, uint32_t m,
                                                   uint32_t* out) {
  constexpr int kFine = kHistBins / 64;
  const int cb = 63 - (threadIdx.x & 63);
  uint32_t c = 0u;
#pragma unroll
  for (int i = 0; i < kFine / 4; ++i) {
    const uint4 v = reinterpret_cast<const uint4*>(lhist + cb * kFine)[i];
    c += v.x + v.y + v.z + v.w;
  }
  walk_first_bin(lhist, c, m, out);
}

// All threads of an NT-thread workgroup: given a histogram of nb bins in
// LDS (nb a multiple of NT or at most NT), find the
// bin where the running count (from the top bin down when DESC, else from
// bin 0 up) first reaches `need`.  Returns the bin and sets *rest to the
// number still needed inside that bin.
template <bool DESC, int NT = kFinishThreads>
__device__ __forceinline__ uint32_t find_bin_block(const uint32_t* hist, int nb,
                                                   uint32_t need, uint32_t* tmp,
                                                   uint32_t* misc,
                                                   uint32_t* rest) {
  const int t = threadIdx.x;
  if (t == 0) {
    misc[0] = 0u;
    misc[1] = 0u;
  }
  const int per = nb > NT ? nb / NT : 1;
  // thread t owns scan positions [t*per, t*per + per)
  auto bin_at = [&](int pos) { return DESC ? nb - 1 - pos : pos; };
  uint32_t v = 0u;
  if (t * per < nb)
    for (int i = 0; i < per; ++i) v += hist[bin_at(t * per + i)];
  uint32_t total;
  const uint32_t incl = block_incl_scan<NT / 64>(v, tmp, &total);
  if (t * per < nb && incl >= need && incl - v < need) {
    uint32_t run = incl - v;
    for (int i = 0; i < per; ++i) {
      const int bin = bin_at(t * per + i);
      const uint32_t c = hist[bin];
      if (run + c >= need) {
        misc[0] = (uint32_t)bin;
        misc[1] = need - run;
        break;
      }
      run += c;
    }
  }
  __syncthreads();
  const uint32_t b = misc[0];
  *rest = misc[1];
  __syncthreads();
  return b;
}

}  // namespace ckv
