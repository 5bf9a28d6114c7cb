// ckv_api.cpp -- the C ABI of libckv: argument checks, workspace layout and
// the launch sequences of each entry point.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "ckv.h"
#include "ckv_launch.hpp"
#include "ckv_profile.hpp"

namespace ckv {

namespace {
thread_local std::string g_detail;
}  // namespace

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_detail = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(CKV_EHIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

const char* last_detail() { return g_detail.c_str(); }

int debug_check(hipStream_t s, const int32_t* ctx_lens, const int32_t* idx,
                const int32_t* n_sel, int B, int Hkv, int max_ctx, int k) {
  if (!debug_on() || B == 0 || (!ctx_lens && !idx && !n_sel)) return CKV_OK;
  // one 16-byte flag per device, kept until the process ends (debug mode only)
  static std::mutex mu;
  static unsigned long long* flags[256] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "debug check");
  if (dev < 0 || dev >= 256) return fail(CKV_EUNSUPPORTED, "device %d", dev);
  {
    std::lock_guard<std::mutex> lk(mu);
    if (!flags[dev] && (e = hipMalloc(&flags[dev], 16)) != hipSuccess)
      return hip_fail(e, "debug check flag");
  }
  CheckArgs a;
  a.ctx_lens = ctx_lens;
  a.idx = idx;
  a.n_sel = n_sel;
  a.flag = flags[dev];
  a.B = B;
  a.Hkv = Hkv;
  a.max_ctx = max_ctx;
  a.k = k;
  unsigned long long got = 0;
  if ((e = launch_fill(a.flag, 16, 0xffffffffu, s)) != hipSuccess ||
      (e = launch_check(a, s)) != hipSuccess ||
      (e = hipMemcpyAsync(&got, a.flag, 8, hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (e = hipStreamSynchronize(s)) != hipSuccess)
    return hip_fail(e, "debug check");
  if (got == ~0ull) return CKV_OK;
  const unsigned kind = (unsigned)(got >> 40);
  const long long item = (long long)(got & ((1ull << 40) - 1));
  if (kind == 1) return fail(CKV_EINVAL, "debug check: ctx_lens[%lld] outside [0, %d]", item, max_ctx);
  if (kind == 2)
    return fail(CKV_EINVAL, "debug check: n_sel of unit %lld outside [0, %d]", item, k);
  return fail(CKV_EINVAL,
              "debug check: index entry %lld of unit %lld is neither -1 nor a position below "
              "the unit's context length",
              item % k, item / k);
}

}  // namespace ckv

namespace {

using namespace ckv;

#define CKV_TRY_HIP(expr, what)                 \
  do {                                          \
    hipError_t e_ = (expr);                     \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

struct Dims {
  int B, Hq, Hkv, G, U, max_ctx;
  int64_t key_stride, kv_stride;
};

// ckv_set_one_launch_same_step
std::atomic<int> g_one_launch{CKV_ONE_LAUNCH_ROW_HALVES};

// A tag for one launch of the one-launch same-step kernel: a 32-bit value
// that is never zero in the high half and its complement in the low half.
uint64_t next_fused_tag() {
  static std::atomic<uint32_t> counter{0};
  uint32_t t = counter.fetch_add(1u, std::memory_order_relaxed) + 1u;
  t *= 2654435761u;  // spread consecutive calls over the 32 bits
  t |= 1u;
  return ((uint64_t)t << 32) | (uint32_t)~t;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_shape(const ckv_shape* s, Dims* d) {
  if (!s) return fail(CKV_EINVAL, "shape is NULL");
  if (s->reserved != 0) return fail(CKV_EINVAL, "shape.reserved must be 0");
  if (s->batch < 0 || s->num_q_heads < 1 || s->num_kv_heads < 1)
    return fail(CKV_ESHAPE, "batch=%d num_q_heads=%d num_kv_heads=%d", s->batch,
                s->num_q_heads, s->num_kv_heads);
  if (s->num_q_heads % s->num_kv_heads)
    return fail(CKV_ESHAPE, "num_q_heads %d not a multiple of num_kv_heads %d",
                s->num_q_heads, s->num_kv_heads);
  if (s->head_dim != kD)
    return fail(CKV_EUNSUPPORTED, "head_dim %d (only %d is supported)", s->head_dim, kD);
  const int G = s->num_q_heads / s->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16)
    return fail(CKV_EUNSUPPORTED, "group size %d not in {1,2,4,8,16}", G);
  if (s->max_ctx < 1 || s->max_ctx > (1 << 30))
    return fail(CKV_ESHAPE, "max_ctx %d outside [1, 2^30]", s->max_ctx);
  if (s->key_row_stride < kD || (s->key_row_stride & 7))
    return fail(CKV_ESHAPE, "key_row_stride %lld (>= 128, multiple of 8)",
                (long long)s->key_row_stride);
  if (s->kv_row_stride < kD || (s->kv_row_stride & 7))
    return fail(CKV_ESHAPE, "kv_row_stride %lld (>= 128, multiple of 8)",
                (long long)s->kv_row_stride);
  const int64_t units = (int64_t)s->batch * s->num_kv_heads;
  if (units > (1 << 24)) return fail(CKV_EUNSUPPORTED, "batch*num_kv_heads too large");
  d->B = s->batch;
  d->Hq = s->num_q_heads;
  d->Hkv = s->num_kv_heads;
  d->G = G;
  d->U = (int)units;
  d->max_ctx = s->max_ctx;
  d->key_stride = s->key_row_stride;
  d->kv_stride = s->kv_row_stride;
  return CKV_OK;
}

int check_k(int32_t k) {
  if (k < 1 || k > (1 << 20)) return fail(CKV_ESHAPE, "k %d outside [1, 2^20]", k);
  return CKV_OK;
}

int check_rank(int32_t rank) {
  if (rank < 1 || rank > CKV_MAX_RANK)
    return fail(CKV_ESHAPE, "rank %d outside [1, %d]", rank, CKV_MAX_RANK);
  return CKV_OK;
}

int check_scale(float scale) {
  if (!(scale > 0.f) || scale > 3.0e38f)
    return fail(CKV_EINVAL, "scale must be a finite positive number");
  return CKV_OK;
}

#define CKV_PTR(p)                                                          \
  do {                                                                      \
    if (!(p)) return fail(CKV_EINVAL, "%s is NULL", #p);                    \
    if (!aligned16(p)) return fail(CKV_EINVAL, "%s is not 16-byte aligned", #p); \
  } while (0)

// Debug mode: the entry's device-side inputs, checked before its launches
// (d: the entry's Dims).
#define CKV_DEBUG_CHECK(stream, lens, idx, nsel, kk)                                       \
  do {                                                                                    \
    const int rc_ = debug_check((hipStream_t)(stream), (lens), (idx), (nsel), d.B, d.Hkv,  \
                                d.max_ctx, (kk));                                         \
    if (rc_) return rc_;                                                                  \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace regions, each 256-byte aligned.  [0, zero_end) is cleared at the
// start of every selecting call.
struct Layout {
  size_t hist = 0, coarse = 0, ctrl = 0, hist2 = 0, coarse2 = 0, ctrl2 = 0, zero_end = 0;
  size_t sel = 0, cand = 0, bitmap = 0, scores = 0, part = 0, hist_part = 0, hist_part_bytes = 0;
  size_t slot_of = 0, miss_pos = 0, miss_slot = 0, n_miss = 0, free_slot = 0, total = 0;
  size_t chunk_idx = 0, n_chunks = 0;  // decode step: selected chunks of a chunked layer
  size_t scores_b = 0, hist_part_b = 0;  // decode step: the second scores and slots region
  size_t flags = 0;  // the same-step layer in one launch: hand-over flags per slot
  size_t merge = 0;  // and its row halves' merge flags per unit
  int64_t bm_words = 0;
  int chunks = 0, filter_tiles = 0;
};

Layout make_layout(const Dims& d, int32_t k, int entry) {
  Layout L;
  const size_t U = (size_t)d.U;
  size_t off = 0;
  L.filter_tiles = (d.max_ctx + kFilterTile - 1) / kFilterTile;
  L.chunks = (k + kAttnRows - 1) / kAttnRows;
  // the decode step's workspace serves every layer kind: corrected layers,
  // two-token layers (2G head rows of partials) and chunked layers (chunk lists)
  const bool step = entry == CKV_ENTRY_DECODE_STEP;
  const bool corrected = entry == CKV_ENTRY_CORRECTED_ATTN || step;
  const bool select = entry == CKV_ENTRY_SELECT_TOPK || entry == CKV_ENTRY_CRITICAL_KV_ATTN ||
                      corrected;
  const bool two_tokens = entry == CKV_ENTRY_DUAL_TOKEN_ATTN || step;
  const bool attn = entry == CKV_ENTRY_SPARSE_DECODE_ATTN ||
                    entry == CKV_ENTRY_CRITICAL_KV_ATTN || corrected || two_tokens;
  if (select) {
    L.hist = off;
    off += U * kHistBins * 4;
    L.coarse = off;
    off += U * kCoarseBins * 4;
    L.ctrl = off;
    off += U * kCtrlWords * 4;
    if (corrected) {  // the second selection of the call starts from zero too
      L.hist2 = off;
      off += U * kHistBins * 4;
      L.coarse2 = off;
      off += U * kCoarseBins * 4;
      L.ctrl2 = off;
      off += U * kCtrlWords * 4;
    }
    off = align256(off);
    L.zero_end = off;
    L.sel = off;
    off = align256(off + U * (size_t)k * 4);
    L.cand = off;
    off = align256(off + U * (size_t)d.max_ctx * 8);
    if (d.max_ctx > kBitmapLdsBits) {
      L.bm_words = (d.max_ctx + 31) / 32;
      L.bitmap = off;
      off = align256(off + U * (size_t)L.bm_words * 4);
    }
  }
  if (entry == CKV_ENTRY_CRITICAL_KV_ATTN || corrected) {
    L.scores = off;
    off = align256(off + U * (size_t)d.max_ctx * 4);
    // per-workgroup histograms of the scoring pass (slots unit + workgroup)
    const int64_t groups = (int64_t)U * ((d.max_ctx + kStageRows - 1) / kStageRows);
    L.hist_part = off;
    L.hist_part_bytes = (U + (size_t)std::min<int64_t>(groups, kMaxScoreWgs)) * kHistBins * 4;
    off = align256(off + L.hist_part_bytes);
    if (entry == CKV_ENTRY_CRITICAL_KV_ATTN) {  // two 64-bit flags per slot, one per unit
      L.flags = off;
      off = align256(off + (U + (size_t)std::min<int64_t>(groups, kMaxScoreWgs)) * 16);
      L.merge = off;
      off = align256(off + U * 8);
    }
  }
  if (attn) {
    L.part = off;
    off = align256(off + U * (size_t)L.chunks * (two_tokens ? 2 : 1) * d.G * kPartStride * 4);
  }
  if (corrected) {
    const size_t list = align256(U * (size_t)k * 4);
    L.slot_of = off;
    off += list;
    L.miss_pos = off;
    off += list;
    L.miss_slot = off;
    off += list;
    L.n_miss = off;
    off = align256(off + U * 4);
    if (k > kMissLds) {
      L.free_slot = off;
      off += list;
    }
  }
  if (step) {
    L.chunk_idx = off;
    off += align256(U * (size_t)k * 4);
    L.n_chunks = off;
    off += align256(U * 4);
    // consecutive plain layers of the decode loop alternate between the
    // scores and slots above (at the fused entry's offsets) and these
    L.scores_b = off;
    off = align256(off + U * (size_t)d.max_ctx * 4);
    L.hist_part_b = off;
    off = align256(off + L.hist_part_bytes);
  }
  L.total = off;
  return L;
}

int check_grid(const Dims& d, const Layout& L) {
  // work-items per dispatch must stay below 2^32
  const int64_t limit = ((int64_t)1 << 32) / 1024 - 1;
  if ((int64_t)d.U * L.filter_tiles > limit || (int64_t)d.U * L.chunks > limit)
    return fail(CKV_EUNSUPPORTED, "grid too large for this shape");
  return CKV_OK;
}

int check_ws(void* ws, size_t ws_bytes, const Layout& L) {
  if (L.total == 0) return CKV_OK;
  if (!ws) return fail(CKV_EWORKSPACE, "workspace is NULL (%zu bytes needed)", L.total);
  if (reinterpret_cast<uintptr_t>(ws) & 255u)
    return fail(CKV_EWORKSPACE, "workspace is not 256-byte aligned");
  if (ws_bytes < L.total)
    return fail(CKV_EWORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, L.total);
  return CKV_OK;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Device address of a host-pinned buffer (hipHostMalloc / torch pin_memory).
int host_to_device(const uint16_t* p, const uint16_t** out) {
  void* dp = nullptr;
  hipError_t e = hipHostGetDevicePointer(&dp, const_cast<uint16_t*>(p), 0);
  if (e != hipSuccess || !dp)
    return fail(CKV_EINVAL, "source is not host-pinned memory visible to the device (%s)",
                hipGetErrorString(e));
  *out = static_cast<const uint16_t*>(dp);
  return CKV_OK;
}

int resolve_src(int src_kind, const uint16_t** k_src, const uint16_t** v_src) {
  if (src_kind == CKV_SRC_DEVICE) return CKV_OK;
  if (src_kind != CKV_SRC_HOST_PINNED) return fail(CKV_EINVAL, "bad src_kind %d", src_kind);
  int rc = host_to_device(*k_src, k_src);
  if (rc) return rc;
  return host_to_device(*v_src, v_src);
}

ReconArgs recon_args(const Dims& d, int32_t rank, const uint16_t* u_fac, const uint16_t* w_fac,
                     const int32_t* idx, const int32_t* n_sel, const int32_t* slots, int32_t k,
                     uint16_t* k_dst) {
  ReconArgs r;
  r.u_fac = u_fac;
  r.w_fac = w_fac;
  r.idx = idx;
  r.n_sel = n_sel;
  r.slots = slots;
  r.k_dst = k_dst;
  r.items = (int64_t)d.U * k * 16;
  r.max_ctx = d.max_ctx;
  r.k = k;
  r.rank = rank;
  return r;
}

// Workgroups of a gather: a pinned source is read over the host link, which
// 256 workgroups keep at its copy rate; device sources take a full grid.
int gather_blocks(int src_kind) { return src_kind == CKV_SRC_HOST_PINNED ? 256 : 4096; }


SelectArgs select_args(const Dims& d, const Layout& L, void* ws, const float* scores,
                       const int32_t* ctx_lens, int32_t k, int32_t* idx, int32_t* n_sel) {
  SelectArgs a;
  a.scores = scores;
  a.ctx_lens = ctx_lens;
  a.hist = at<uint32_t>(ws, L.hist);
  a.coarse = at<uint32_t>(ws, L.coarse);
  a.ctrl = at<uint32_t>(ws, L.ctrl);
  a.sel = at<int32_t>(ws, L.sel);
  a.cand = at<uint2>(ws, L.cand);
  a.bitmap = L.bm_words ? at<uint32_t>(ws, L.bitmap) : nullptr;
  a.idx = idx;
  a.n_sel = n_sel;
  a.bm_words = L.bm_words;
  a.Hkv = d.Hkv;
  a.max_ctx = d.max_ctx;
  a.k = k;
  a.tiles = L.filter_tiles;
  a.chunk = 1;
  a.hist_part = nullptr;
  a.score_nwg = 0;
  a.units = d.U;
  a.mpart = nullptr;
  a.mout = nullptr;
  a.mchunks = a.mG = a.mHq = 0;
  a.affine = 0;
  return a;
}

// Scoring arguments; with sel set, the pass counts the first digit into that
// selection's histograms, and a pipelined launch with enough work may take
// it as claims from the selection's claim counter (unit 0's control word
// kCtrlClaim, cleared with the histograms; the pass leaves it zero), unless
// a caller switches the pass to per-workgroup histograms.
ScoreArgs score_args(const Dims& d, const Layout& L, const uint16_t* q,
                     const uint16_t* keys, const int32_t* ctx_lens, float scale,
                     float* scores, const SelectArgs* sel) {
  ScoreArgs a;
  a.q = q;
  a.keys = keys;
  a.ctx_lens = ctx_lens;
  a.scores = scores;
  a.hist = sel ? sel->hist : nullptr;
  a.coarse = sel ? sel->coarse : nullptr;
  // claim numbers (and the nwg failing ones past them) must fit in 32 bits
  const int64_t claims =
      (int64_t)d.U * (((d.max_ctx + kStageRows - 1) / kStageRows + kClaimGroups - 1) / kClaimGroups);
  a.claim = sel && claims + kMaxScoreWgs < ((int64_t)1 << 31) ? sel->ctrl + kCtrlClaim : nullptr;
  a.key_stride = d.key_stride;
  a.scale = scale;
  a.Hq = d.Hq;
  a.Hkv = d.Hkv;
  a.max_ctx = d.max_ctx;
  a.units = d.U;
  a.chunk = 1;
  a.hist_part = nullptr;
  return a;
}

AttnArgs attn_args(const Dims& d, const Layout& L, void* ws, const uint16_t* q,
                   const uint16_t* k_rows, const uint16_t* v_rows, const int32_t* idx,
                   const int32_t* n_sel, int64_t row_stride, int32_t k, float scale,
                   float* out) {
  AttnArgs a;
  a.q = q;
  a.k_rows = k_rows;
  a.v_rows = v_rows;
  a.idx = idx;
  a.n_sel = n_sel;
  a.part = at<float>(ws, L.part);
  a.out = out;
  a.q2 = nullptr;
  a.out2 = nullptr;
  a.k_local = nullptr;
  a.v_local = nullptr;
  a.row_stride = row_stride;
  a.scale = scale;
  a.Hq = d.Hq;
  a.Hkv = d.Hkv;
  a.max_ctx = d.max_ctx;
  a.k = k;
  a.chunks = L.chunks;
  return a;
}

// Selection given scores and a filled first-digit histogram: one workgroup
// per unit for contexts that fit its LDS, else the many-workgroup filter
// followed by the per-unit finish.
// The scoring pass leaves per-workgroup histograms (stored, so no clearing
// and no atomics) when the fused selection reads them and no unit needs more
// than kMaxPartials of them; then the call has nothing to clear.  Otherwise
// the histograms are added into cleared per-unit counts.
bool use_partials(const Dims& d, const Layout& L, int nwg) {
  if (!L.hist_part_bytes || d.max_ctx > kFusedSelectMaxCtx || nwg < 1) return false;
  // a unit's gu groups meet at most ceil(gu / shortest range) + 1 ranges
  const int64_t gu = (d.max_ctx + kStageRows - 1) / kStageRows;
  const int64_t shortest = gu * d.U / nwg;
  return shortest >= 1 && (gu + shortest - 1) / shortest + 1 <= kMaxPartials;
}

void set_partials(void* ws, const Layout& L, int nwg, ScoreArgs* sc, SelectArgs* sa) {
  sc->hist_part = at<uint32_t>(ws, L.hist_part);
  sa->hist_part = sc->hist_part;
  sa->score_nwg = nwg;
}

int run_select_tail(const SelectArgs& a, int units, hipStream_t s) {
  if (a.max_ctx <= kFusedSelectMaxCtx) {
    CKV_TRY_HIP(launch_select_fused(a, units, s), "select launch");
    return CKV_OK;
  }
  CKV_TRY_HIP(launch_filter(a, units, s), "filter launch");
  CKV_TRY_HIP(launch_finish(a, units, s), "finish launch");
  return CKV_OK;
}

// The next step's selection after a pipelined attend-and-score launch, and
// the merge of that launch's attention partials: inside the fused selection
// when it runs (one workgroup per unit, which loads the unit's partials while
// it selects), else by the merge kernel.
int select_and_merge(SelectArgs sa, const AttnArgs& at, const Dims& d, hipStream_t s) {
  if (sa.max_ctx <= kFusedSelectMaxCtx && at.chunks <= kMergeChunks &&
      d.G * kD <= kFinishThreads && !at.q2) {
    sa.mpart = at.part;
    sa.mout = at.out;
    sa.mchunks = at.chunks;
    sa.mG = d.G;
    sa.mHq = d.Hq;
    return run_select_tail(sa, d.U, s);
  }
  int rc = run_select_tail(sa, d.U, s);
  if (rc) return rc;
  CKV_TRY_HIP(launch_combine(at, d.G, d.U, s), "combine launch");
  return CKV_OK;
}

// Workgroups per unit of the same-step selection and attention in one launch
// (0: that launch does not apply and the selection, attention and merge run
// as three kernels).  Two when two workgroups per unit still fit on the
// device's CUs (then every CU has a workgroup to attend with): for an even
// group size with the whole set in one workgroup's LDS, each takes half the
// heads (*heads = 2, no merge); else each takes a share of the rows, and more
// shares when a share would exceed kSelAttnMaxShare rows (*heads = 1).
int select_attn_splits(const Dims& d, int32_t k, const Layout& L, int* heads) {
  *heads = 1;
  if (d.max_ctx > kFusedSelectMaxCtx || d.G > 8) return 0;
  const bool two = 2 * (int64_t)d.U <= device_cus() && k >= 512;
  if (two && d.G % 2 == 0 && k <= kSelAttnMaxShare) {
    *heads = 2;
    return 1;
  }
  int S = two ? 2 : 1;
  while ((((k + S - 1) / S + 15) & ~15) > kSelAttnMaxShare) S *= 2;
  if (S > kSelAttnMaxSplit || S > L.chunks) return 0;
  return S;
}

// Attention of `a` over its set, then the merge of its chunk partials.
int run_attention(const AttnArgs& a, const Dims& d, bool indexed, hipStream_t s) {
  CKV_TRY_HIP(launch_attn(a, d.G, indexed, d.U, s), "attention launch");
  CKV_TRY_HIP(launch_combine(a, d.G, d.U, s), "combine launch");
  return CKV_OK;
}

int check_chunk(int32_t chunk, int32_t k) {
  if (chunk < 1 || chunk > (1 << 20)) return fail(CKV_ESHAPE, "chunk %d outside [1, 2^20]", chunk);
  if (k % chunk) return fail(CKV_ESHAPE, "k %d is not a multiple of chunk %d", k, chunk);
  return CKV_OK;
}

// Scores every chunk landmark of the chunk problem (one entry per chunk,
// budget k / chunk), whose layout fits inside the layout of the row problem
// that the caller's workspace was sized for; sets *sa to that problem's
// selection into chunk_idx / n_chunks and *e to the expansion of its chunks.
int score_chunks(const Dims& d, int32_t chunk, const uint16_t* q_sel,
                 const uint16_t* landmarks, const int32_t* ctx_lens, int32_t k, float scale,
                 int32_t* chunk_idx, int32_t* n_chunks, int32_t* rows, int32_t* n_rows,
                 void* ws, hipStream_t s, SelectArgs* sa, ExpandArgs* e) {
  Dims dc = d;
  dc.max_ctx = (d.max_ctx + chunk - 1) / chunk;
  dc.key_stride = kD;
  const int32_t kc = k / chunk;
  Layout Lc = make_layout(dc, kc, CKV_ENTRY_CRITICAL_KV_ATTN);
  int rc;
  if ((rc = check_grid(dc, Lc))) return rc;
  float* scores = at<float>(ws, Lc.scores);
  *sa = select_args(dc, Lc, ws, scores, ctx_lens, kc, chunk_idx, n_chunks);
  sa->chunk = chunk;
  ScoreArgs sc = score_args(dc, Lc, q_sel, landmarks, ctx_lens, scale, scores, sa);
  sc.chunk = chunk;
  const int nwg = score_blocks(sc, d.G, ScoreKind::kHist);
  if (use_partials(dc, Lc, nwg))
    set_partials(ws, Lc, nwg, &sc, sa);
  else
    CKV_TRY_HIP(launch_zero(ws, Lc.zero_end, s), "zero launch");
  CKV_TRY_HIP(launch_score(sc, d.G, true, nwg, s), "score launch");
  e->chunk_idx = chunk_idx;
  e->n_chunks = n_chunks;
  e->ctx_lens = ctx_lens;
  e->rows = rows;
  e->n_rows = n_rows;
  e->Hkv = d.Hkv;
  e->max_ctx = d.max_ctx;
  e->chunk = chunk;
  e->kc = kc;
  e->k = k;
  return CKV_OK;
}

// Chunk selection into caller arrays: the scoring above, the selection, and
// the expansion to rows.
int run_select_chunks(const Dims& d, int32_t chunk, const uint16_t* q_sel,
                      const uint16_t* landmarks, const int32_t* ctx_lens, int32_t k,
                      float scale, int32_t* chunk_idx, int32_t* n_chunks, int32_t* rows,
                      int32_t* n_rows, void* ws, hipStream_t s) {
  SelectArgs sa;
  ExpandArgs e;
  int rc = score_chunks(d, chunk, q_sel, landmarks, ctx_lens, k, scale, chunk_idx, n_chunks,
                        rows, n_rows, ws, s, &sa, &e);
  if (rc) return rc;
  if ((rc = run_select_tail(sa, d.U, s))) return rc;
  CKV_TRY_HIP(launch_expand(e, d.U, s), "expand launch");
  return CKV_OK;
}

// Whether the same-step chunked call selects, expands and attends in one
// launch (k_select_attn_chunks): the conditions of the head-halves form of
// the fused same-step launch, on the chunk problem's context, with one
// thread per selected chunk.
bool chunk_select_attn(const Dims& d, int32_t chunk, int32_t k) {
  const int64_t cmax = (d.max_ctx + chunk - 1) / chunk;
  return cmax <= kFusedSelectMaxCtx && d.G <= 8 && d.G % 2 == 0 && k >= 512 &&
         k <= kSelAttnMaxShare && k / chunk <= kFinishThreads &&
         2 * (int64_t)d.U <= device_cus();
}

}  // namespace

int ckv::pipelined_layer(const ckv_shape* shape, const PipelinedLayer& p,
                         const int32_t* ctx_lens, int32_t k, float scale, void* ws,
                         size_t ws_bytes, void* stream, LoopLink* link) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  const uint16_t* q_att = p.q_att;
  const uint16_t* q_sel = p.q_sel ? p.q_sel : p.q_att;
  CKV_PTR(q_att);
  CKV_PTR(q_sel);
  CKV_PTR(ctx_lens);
  CKV_PTR(p.idx_out);
  CKV_PTR(p.n_sel_out);
  CKV_PTR(p.out);
  const bool chunked = p.chunk > 1;
  const uint16_t* keys = chunked ? p.landmarks : p.k_score;
  if (chunked) {
    if ((rc = check_chunk(p.chunk, k))) return rc;
    CKV_PTR(p.landmarks);
  } else {
    if (p.chunk < 0) return fail(CKV_ESHAPE, "chunk %d", p.chunk);
    CKV_PTR(p.k_score);
  }
  const bool two = p.out_spec != nullptr;
  if (link && (!two || chunked || p.k_buf))
    return fail(CKV_EINVAL, "a loop link needs a two-token layer read in place");
  if (two) {
    if (d.G > 8)
      return fail(CKV_EUNSUPPORTED, "two tokens need 2G <= 16 head rows (G = %d)", d.G);
    CKV_PTR(p.k_local);
    CKV_PTR(p.v_local);
    CKV_PTR(p.out_spec);
  }
  const bool assembled = p.k_buf != nullptr, in_place = p.idx_in != nullptr;
  if (assembled == in_place)
    return fail(CKV_EINVAL, "exactly one of the assembled buffer and idx_in");
  const uint16_t *k_src = p.k_src, *v_src = p.v_src;
  CKV_PTR(p.n_sel_in);
  if (assembled) {
    CKV_PTR(p.k_buf);
    CKV_PTR(p.v_buf);
  } else {
    CKV_PTR(k_src);
    CKV_PTR(v_src);
    if ((rc = resolve_src(p.src_kind, &k_src, &v_src))) return rc;
  }
  const Layout L = make_layout(d, k, CKV_ENTRY_DECODE_STEP);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, assembled ? nullptr : p.idx_in, p.n_sel_in, k);
  hipStream_t s = (hipStream_t)stream;
  // the selection problem: positions, or chunks (one landmark per chunk rows,
  // budget k / chunk), whose regions lie below the attention partials
  Dims ds = d;
  int32_t ks = k;
  Layout Ls = L;
  if (chunked) {
    ds.max_ctx = (d.max_ctx + p.chunk - 1) / p.chunk;
    ds.key_stride = kD;
    ks = k / p.chunk;
    Ls = make_layout(ds, ks, CKV_ENTRY_CRITICAL_KV_ATTN);
    if ((rc = check_grid(ds, Ls))) return rc;
    if (Ls.part > L.part) return fail(CKV_EWORKSPACE, "chunk selection layout overlaps");
  }
  if (link && link->alt) {  // this layer's scores and slots in the second region
    Ls.scores = L.scores_b;
    Ls.hist_part = L.hist_part_b;
  }
  int32_t* sidx = chunked ? at<int32_t>(ws, L.chunk_idx) : p.idx_out;
  int32_t* sn = chunked ? at<int32_t>(ws, L.n_chunks) : p.n_sel_out;
  float* scores = at<float>(ws, Ls.scores);
  SelectArgs sa = select_args(ds, Ls, ws, scores, ctx_lens, ks, sidx, sn);
  sa.chunk = chunked ? p.chunk : 1;
  ScoreArgs sc = score_args(ds, Ls, q_sel, keys, ctx_lens, scale, scores, &sa);
  sc.chunk = sa.chunk;
  AttnArgs at_ = assembled ? attn_args(d, L, ws, q_att, p.k_buf, p.v_buf, nullptr, p.n_sel_in,
                                       kD, k, scale, p.out)
                           : attn_args(d, L, ws, q_att, k_src, v_src, p.idx_in, p.n_sel_in,
                                       d.kv_stride, k, scale, p.out);
  if (two) {  // the speculative token attends too: its query is the selecting one
    at_.q2 = q_sel;
    at_.out2 = p.out_spec;
    at_.k_local = p.k_local;
    at_.v_local = p.v_local;
  }
  const ScoreKind kind = two ? (in_place ? ScoreKind::kDual2Indexed : ScoreKind::kDual2)
                             : (in_place ? ScoreKind::kDualIndexed : ScoreKind::kDual);
  int nwg = score_blocks(sc, d.G, kind);
  const bool partials = use_partials(ds, Ls, nwg);
  // the previous two-token layer's pending selection joins this launch
  bool fold = false;
  if (link && link->prev) {
    const int nwg_sel = score_blocks(
        sc, d.G, in_place ? ScoreKind::kDual2SelIndexed : ScoreKind::kDual2Sel);
    fold = partials && nwg_sel > 0 && use_partials(ds, Ls, nwg_sel) &&
           d.max_ctx <= kFusedSelectMaxCtx && link->prev->units == d.U;
    if (fold) nwg = nwg_sel;
    else CKV_TRY_HIP(launch_select_fused(*link->prev, link->prev->units, s), "select launch");
  }
  if (partials)
    set_partials(ws, Ls, nwg, &sc, &sa);
  else if (!p.hist_clean)
    CKV_TRY_HIP(launch_zero(ws, Ls.zero_end, s), "zero launch");
  if (fold)
    CKV_TRY_HIP(launch_dual_sel(at_, sc, *link->prev, d.G, in_place, d.U, nwg, s),
                "dual launch");
  else
    CKV_TRY_HIP(launch_dual(at_, sc, d.G, in_place, d.U, nwg, s), "dual launch");
  if (two) {
    if (link && link->next && partials && d.max_ctx <= kFusedSelectMaxCtx) {
      *link->next = sa;  // the next two-token layer's launch selects
      link->deferred = true;
    } else if ((rc = run_select_tail(sa, d.U, s))) {
      return rc;
    }
    CKV_TRY_HIP(launch_combine(at_, 2 * d.G, d.U, s), "combine launch");
  } else if ((rc = select_and_merge(sa, at_, d, s))) {
    return rc;
  }
  if (chunked) {
    ExpandArgs e;
    e.chunk_idx = sidx;
    e.n_chunks = sn;
    e.ctx_lens = ctx_lens;
    e.rows = p.idx_out;
    e.n_rows = p.n_sel_out;
    e.Hkv = d.Hkv;
    e.max_ctx = d.max_ctx;
    e.chunk = p.chunk;
    e.kc = ks;
    e.k = k;
    CKV_TRY_HIP(launch_expand(e, d.U, s), "expand launch");
  }
  return CKV_OK;
}

int ckv::gather_kv_width(const ckv_shape* shape, const uint16_t* k_src, const uint16_t* v_src,
                    int src_kind, const int32_t* idx, const int32_t* n_sel, int32_t k,
                    uint16_t* k_dst, uint16_t* v_dst, int workgroups, void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  CKV_PTR(k_src);
  CKV_PTR(v_src);
  CKV_PTR(idx);
  CKV_PTR(n_sel);
  CKV_PTR(k_dst);
  CKV_PTR(v_dst);
  if (workgroups < 0 || workgroups > kMaxGatherWgs)
    return fail(CKV_EINVAL, "gather width %d outside [0, %d]", workgroups, kMaxGatherWgs);
  if ((rc = resolve_src(src_kind, &k_src, &v_src))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, nullptr, idx, n_sel, k);
  GatherArgs a;
  a.k_src = k_src;
  a.v_src = v_src;
  a.idx = idx;
  a.n_sel = n_sel;
  a.slots = nullptr;
  a.k_dst = k_dst;
  a.v_dst = v_dst;
  a.row_stride = d.kv_stride;
  a.items = (int64_t)d.U * k * 32;
  a.max_ctx = d.max_ctx;
  a.k = k;
  CKV_TRY_HIP(launch_gather(a, workgroups ? workgroups : gather_blocks(src_kind),
                            (hipStream_t)stream),
              "gather launch");
  return CKV_OK;
}

extern "C" {

int ckv_abi_version(void) { return CKV_ABI_VERSION; }

const char* ckv_status_str(int status) {
  switch (status) {
    case CKV_OK: return "ok";
    case CKV_EINVAL: return "invalid argument";
    case CKV_ESHAPE: return "invalid shape";
    case CKV_EUNSUPPORTED: return "unsupported shape";
    case CKV_EWORKSPACE: return "workspace missing or too small";
    case CKV_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* ckv_last_error_detail(void) { return last_detail(); }

int ckv_workspace_bytes(const ckv_shape* shape, int32_t k, int entry, size_t* bytes) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if (!bytes) return fail(CKV_EINVAL, "bytes is NULL");
  if (entry != CKV_ENTRY_SELECT_TOPK && entry != CKV_ENTRY_SPARSE_DECODE_ATTN &&
      entry != CKV_ENTRY_CRITICAL_KV_ATTN && entry != CKV_ENTRY_CORRECTED_ATTN &&
      entry != CKV_ENTRY_DUAL_TOKEN_ATTN && entry != CKV_ENTRY_DECODE_STEP)
    return fail(CKV_EINVAL, "unknown entry %d", entry);
  *bytes = make_layout(d, k, entry).total;
  return CKV_OK;
}

int ckv_score_keys(const ckv_shape* shape, const uint16_t* q, const uint16_t* k_score,
                   const int32_t* ctx_lens, float scale, float* scores, void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_scale(scale))) return rc;
  CKV_PTR(q);
  CKV_PTR(k_score);
  CKV_PTR(ctx_lens);
  CKV_PTR(scores);
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, nullptr, nullptr, 1);
  Layout L = make_layout(d, 1, 0);
  if ((rc = check_grid(d, L))) return rc;
  ScoreArgs a = score_args(d, L, q, k_score, ctx_lens, scale, scores, nullptr);
  CKV_TRY_HIP(launch_score(a, d.G, false, score_blocks(a, d.G, ScoreKind::kPlain),
                           (hipStream_t)stream),
              "score launch");
  return CKV_OK;
}

int ckv_select_topk(const ckv_shape* shape, const float* scores, const int32_t* ctx_lens,
                    int32_t k, int32_t* idx, int32_t* n_sel, void* ws, size_t ws_bytes,
                    void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  CKV_PTR(scores);
  CKV_PTR(ctx_lens);
  CKV_PTR(idx);
  CKV_PTR(n_sel);
  Layout L = make_layout(d, k, CKV_ENTRY_SELECT_TOPK);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, nullptr, nullptr, k);
  hipStream_t s = (hipStream_t)stream;
  SelectArgs a = select_args(d, L, ws, scores, ctx_lens, k, idx, n_sel);
  CKV_TRY_HIP(launch_zero(ws, L.zero_end, s), "zero launch");
  CKV_TRY_HIP(launch_hist(a, d.U, s), "hist launch");
  return run_select_tail(a, d.U, s);
}

int ckv_gather_kv(const ckv_shape* shape, const uint16_t* k_src, const uint16_t* v_src,
                  int src_kind, const int32_t* idx, const int32_t* n_sel, int32_t k,
                  uint16_t* k_dst, uint16_t* v_dst, void* stream) {
  return ckv::gather_kv_width(shape, k_src, v_src, src_kind, idx, n_sel, k, k_dst, v_dst, 0,
                              stream);
}

}  // extern "C"

namespace {

// The probe's shape, k and mode checks (the sink size needs all three).
int check_probe(const ckv_shape* shape, int32_t k, int mode, Dims* d) {
  int rc = check_shape(shape, d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if (mode != CKV_PROBE_STANDALONE && mode != CKV_PROBE_ROW_HALVES &&
      mode != CKV_PROBE_HEAD_HALVES)
    return fail(CKV_EINVAL, "probe mode %d unknown", mode);
  if (mode != CKV_PROBE_STANDALONE && k > kSelAttnMaxShare)
    return fail(CKV_ESHAPE, "k %d above %d for the probe's halves", k, kSelAttnMaxShare);
  // work-items per dispatch must stay below 2^32
  const int64_t limit = ((int64_t)1 << 32) / kFinishThreads - 16;
  if ((int64_t)d->U * ((k + kAttnRows - 1) / kAttnRows) > limit || (int64_t)d->U * 2 > limit)
    return fail(CKV_EUNSUPPORTED, "grid too large for this shape");
  return CKV_OK;
}

}  // namespace

extern "C" {

size_t ckv_probe_sink_words(const ckv_shape* shape, int32_t k, int mode) {
  Dims d;
  if (check_probe(shape, k, mode, &d)) return 0;
  return ckv::probe_sink_words(d.U, k, mode);
}

int ckv_probe_read_rows(const ckv_shape* shape, const uint16_t* k_rows,
                        const uint16_t* v_rows, const int32_t* idx, int32_t k, int mode,
                        uint32_t* sink, size_t sink_words, void* stream) {
  Dims d;
  int rc = check_probe(shape, k, mode, &d);
  if (rc) return rc;
  CKV_PTR(k_rows);
  CKV_PTR(v_rows);
  CKV_PTR(idx);
  CKV_PTR(sink);
  const size_t need = ckv::probe_sink_words(d.U, k, mode);
  if (sink_words < need)
    return fail(CKV_EINVAL, "sink of %zu words, %zu needed", sink_words, need);
  if (d.U == 0) return CKV_OK;
  ckv::ProbeArgs a;
  a.k_rows = k_rows;
  a.v_rows = v_rows;
  a.idx = idx;
  a.sink = sink;
  a.row_stride = d.kv_stride;
  a.max_ctx = d.max_ctx;
  a.k = k;
  a.units = d.U;
  CKV_TRY_HIP(ckv::launch_probe(a, mode, (hipStream_t)stream), "probe launch");
  return CKV_OK;
}

int ckv_sparse_decode_attn(const ckv_shape* shape, const uint16_t* q_att,
                           const uint16_t* k_buf, const uint16_t* v_buf,
                           const int32_t* n_sel, int32_t k, float scale, float* out,
                           void* ws, size_t ws_bytes, void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  CKV_PTR(q_att);
  CKV_PTR(k_buf);
  CKV_PTR(v_buf);
  CKV_PTR(n_sel);
  CKV_PTR(out);
  Layout L = make_layout(d, k, CKV_ENTRY_SPARSE_DECODE_ATTN);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, nullptr, nullptr, n_sel, k);
  hipStream_t s = (hipStream_t)stream;
  AttnArgs a = attn_args(d, L, ws, q_att, k_buf, v_buf, nullptr, n_sel, kD, k, scale, out);
  return run_attention(a, d, false, s);
}

int ckv_critical_kv_attn(const ckv_shape* shape, const uint16_t* q_att,
                         const uint16_t* q_sel, const uint16_t* k_score,
                         const int32_t* ctx_lens, int32_t k, float scale,
                         const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                         const int32_t* idx_in, const uint16_t* k_buf, const uint16_t* v_buf,
                         const int32_t* n_sel_in, int32_t* idx_out, int32_t* n_sel_out,
                         float* out, void* ws, size_t ws_bytes, void* stream) {
  return ckv::critical_impl(shape, q_att, q_sel, k_score, ctx_lens, k, scale, k_src, v_src,
                            src_kind, idx_in, k_buf, v_buf, n_sel_in, idx_out, n_sel_out, out,
                            ws, ws_bytes, stream, false);
}

}  // extern "C"

int ckv::critical_impl(const ckv_shape* shape, const uint16_t* q_att, const uint16_t* q_sel,
                       const uint16_t* k_score, const int32_t* ctx_lens, int32_t k, float scale,
                       const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                       const int32_t* idx_in, const uint16_t* k_buf, const uint16_t* v_buf,
                       const int32_t* n_sel_in, int32_t* idx_out, int32_t* n_sel_out,
                       float* out, void* ws, size_t ws_bytes, void* stream, bool hist_clean,
                       LoopLink* link) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  CKV_PTR(q_att);
  if (!q_sel) q_sel = q_att;
  CKV_PTR(q_sel);
  CKV_PTR(k_score);
  CKV_PTR(ctx_lens);
  CKV_PTR(idx_out);
  CKV_PTR(n_sel_out);
  CKV_PTR(out);
  if (idx_in && k_buf)
    return fail(CKV_EINVAL, "idx_in and k_buf are exclusive (rows in place or assembled)");
  // pipelined: the attended set was selected one step earlier, either
  // assembled in k_buf/v_buf or read in place through idx_in
  const bool assembled = k_buf != nullptr, in_place = idx_in != nullptr;
  if (assembled) {
    CKV_PTR(k_buf);
    CKV_PTR(v_buf);
    CKV_PTR(n_sel_in);
  } else {
    CKV_PTR(k_src);
    CKV_PTR(v_src);
    if (in_place) CKV_PTR(n_sel_in);
    if ((rc = resolve_src(src_kind, &k_src, &v_src))) return rc;
  }
  Layout L = make_layout(d, k, CKV_ENTRY_CRITICAL_KV_ATTN);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  const bool pipelined = assembled || in_place;
  if (link && !pipelined) return fail(CKV_EINVAL, "a loop link needs a pipelined call");
  if (link && link->alt) {  // this layer's scores and slots in the second region
    const Layout Ls = make_layout(d, k, CKV_ENTRY_DECODE_STEP);
    if ((rc = check_ws(ws, ws_bytes, Ls))) return rc;
    L.scores = Ls.scores_b;
    L.hist_part = Ls.hist_part_b;
  }
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, idx_in, n_sel_in, k);
  hipStream_t s = (hipStream_t)stream;
  float* scores = at<float>(ws, L.scores);
  SelectArgs sa = select_args(d, L, ws, scores, ctx_lens, k, idx_out, n_sel_out);
  ScoreArgs sc = score_args(d, L, q_sel, k_score, ctx_lens, scale, scores, &sa);
  int nwg = score_blocks(
      sc, d.G, !pipelined ? ScoreKind::kHist : in_place ? ScoreKind::kDualIndexed : ScoreKind::kDual);
  bool partials = use_partials(d, L, nwg);
  // the previous layer's pending selection joins this launch when this
  // launch is the one-token kernel with static ranges and slots
  bool fold = false;
  if (link && link->prev) {
    const int nwg_sel = score_blocks(
        sc, d.G, in_place ? ScoreKind::kDualSelIndexed : ScoreKind::kDualSel);
    fold = partials && nwg_sel > 0 && use_partials(d, L, nwg_sel) &&
           d.max_ctx <= kFusedSelectMaxCtx && link->prev->units == d.U;
    if (fold) nwg = nwg_sel;
    else CKV_TRY_HIP(launch_select_fused(*link->prev, link->prev->units, s), "select launch");
  }
  // a pipelined call whose caller knows the histograms clear (the previous
  // selection on this workspace left them so) skips the clearing kernel
  if (partials)
    set_partials(ws, L, nwg, &sc, &sa);
  else if (!(pipelined && hist_clean))
    CKV_TRY_HIP(launch_zero(ws, L.zero_end, s), "zero launch");
  if (pipelined) {
    AttnArgs at_ = assembled ? attn_args(d, L, ws, q_att, k_buf, v_buf, nullptr, n_sel_in, kD,
                                         k, scale, out)
                             : attn_args(d, L, ws, q_att, k_src, v_src, idx_in, n_sel_in,
                                         d.kv_stride, k, scale, out);
    if (fold)
      CKV_TRY_HIP(launch_dual_sel(at_, sc, *link->prev, d.G, in_place, d.U, nwg, s),
                  "dual launch");
    else
      CKV_TRY_HIP(launch_dual(at_, sc, d.G, in_place, d.U, nwg, s), "dual launch");
    if (link && link->next && partials && d.max_ctx <= kFusedSelectMaxCtx) {
      // the next layer's launch selects this layer's sets; the partials are
      // merged now
      CKV_TRY_HIP(launch_combine(at_, d.G, d.U, s), "combine launch");
      *link->next = sa;
      link->deferred = true;
    } else if ((rc = select_and_merge(sa, at_, d, s))) {
      return rc;
    }
  } else {
    AttnArgs at_ = attn_args(d, L, ws, q_att, k_src, v_src, idx_out, n_sel_out,
                             d.kv_stride, k, scale, out);
    int heads;
    int S = select_attn_splits(d, k, L, &heads);
    const int one = g_one_launch.load();
    // row halves need a partial per half in the attention partials
    const bool rows = one == CKV_ONE_LAUNCH_ROW_HALVES && L.chunks >= 2;
    if (S == 1 && heads == 2 && partials && L.flags && one &&
        critical_blocks(d.G, d.U, nwg, rows)) {
      // scoring, selection and attention in one launch, XCD-affine slots
      sa.affine = 1;
      const FusedSync fs{at<uint64_t>(ws, L.flags), at<uint64_t>(ws, L.merge), next_fused_tag()};
      CKV_TRY_HIP(launch_critical(sc, sa, at_, fs, d.G, nwg, rows, s), "same-step launch");
      return CKV_OK;
    }
    CKV_TRY_HIP(launch_score(sc, d.G, true, nwg, s), "score launch");
    if (S) {
      // each workgroup selects its unit's set and attends over its share of
      // the rows, or over the whole set with its share of the heads.  Two
      // workgroups per unit attend over half of the rows each and merge in
      // the launch, unless head halves are asked for (where they apply) or
      // the layout has no merge flags.
      const bool merge2 = (S == 2 || (S == 1 && heads == 2 && one != CKV_ONE_LAUNCH_HEAD_HALVES)) &&
                          L.merge > 0 && L.chunks >= 2;
      if (merge2) {
        S = 2;
        heads = 1;
      }
      at_.chunks = S;
      const FusedSync fs{nullptr, merge2 ? at<uint64_t>(ws, L.merge) : nullptr, next_fused_tag()};
      CKV_TRY_HIP(launch_select_attn(sa, at_, d.G, S, heads, merge2 ? &fs : nullptr, s),
                  "select-attention launch");
      if (S > 1 && !merge2) CKV_TRY_HIP(launch_combine(at_, d.G, d.U, s), "combine launch");
    } else {
      if ((rc = run_select_tail(sa, d.U, s))) return rc;
      if ((rc = run_attention(at_, d, true, s))) return rc;
    }
  }
  return CKV_OK;
}

extern "C" {

int ckv_set_one_launch_same_step(int on) {
  g_one_launch.store(on == CKV_ONE_LAUNCH_HEAD_HALVES ? CKV_ONE_LAUNCH_HEAD_HALVES
                     : on                             ? CKV_ONE_LAUNCH_ROW_HALVES
                                                      : CKV_ONE_LAUNCH_OFF);
  return CKV_OK;
}

int ckv_critical_kv_attn_noalloc(const ckv_shape* shape, const uint16_t* q_att,
                                 const uint16_t* q_sel, const uint16_t* k_score,
                                 const int32_t* ctx_lens, int32_t k, float scale,
                                 const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                                 const int32_t* idx_in, const uint16_t* k_buf,
                                 const uint16_t* v_buf, const int32_t* n_sel_in,
                                 int32_t* idx_out, int32_t* n_sel_out, float* out,
                                 void* stream) {
  // the size check first: an oversized shape is refused before any runtime call
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  const size_t need = make_layout(d, k, CKV_ENTRY_CRITICAL_KV_ATTN).total;
  if (need > CKV_NOALLOC_SCRATCH_BYTES)
    return fail(CKV_EWORKSPACE,
                "this shape needs %zu bytes of workspace; the fixed scratch holds %zu "
                "(use ckv_critical_kv_attn with a workspace)",
                need, (size_t)CKV_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((rc = noalloc_scratch(&ws))) return rc;
  return ckv_critical_kv_attn(shape, q_att, q_sel, k_score, ctx_lens, k, scale, k_src, v_src,
                              src_kind, idx_in, k_buf, v_buf, n_sel_in, idx_out, n_sel_out, out,
                              ws, CKV_NOALLOC_SCRATCH_BYTES, stream);
}

int ckv_dual_token_attn(const ckv_shape* shape, const uint16_t* q_cur, const uint16_t* q_spec,
                        const uint16_t* k_buf, const uint16_t* v_buf, const int32_t* n_sel,
                        const uint16_t* k_local, const uint16_t* v_local, int32_t k,
                        float scale, float* out_cur, float* out_spec, void* ws, size_t ws_bytes,
                        void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  if (d.G > 8)
    return fail(CKV_EUNSUPPORTED, "two tokens need 2G <= 16 head rows (G = %d)", d.G);
  CKV_PTR(q_cur);
  CKV_PTR(q_spec);
  CKV_PTR(k_buf);
  CKV_PTR(v_buf);
  CKV_PTR(n_sel);
  CKV_PTR(k_local);
  CKV_PTR(v_local);
  CKV_PTR(out_cur);
  CKV_PTR(out_spec);
  Layout L = make_layout(d, k, CKV_ENTRY_DUAL_TOKEN_ATTN);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, nullptr, nullptr, n_sel, k);
  hipStream_t s = (hipStream_t)stream;
  AttnArgs a = attn_args(d, L, ws, q_cur, k_buf, v_buf, nullptr, n_sel, kD, k, scale, out_cur);
  a.q2 = q_spec;
  a.out2 = out_spec;
  a.k_local = k_local;
  a.v_local = v_local;
  if (2 * (int64_t)d.U <= device_cus() && k >= 512) {
    // a workgroup per token and unit, each over all of the unit's rows
    CKV_TRY_HIP(launch_dual_token_wg(a, d.G, d.U, s), "dual-token attention launch");
    return CKV_OK;
  }
  // one launch reads each selected row once for the 2G head rows of both tokens
  CKV_TRY_HIP(launch_attn(a, 2 * d.G, false, d.U, s), "attention launch");
  CKV_TRY_HIP(launch_combine(a, 2 * d.G, d.U, s), "combine launch");
  return CKV_OK;
}

int ckv_chunk_landmarks(const ckv_shape* shape, int32_t chunk, const uint16_t* keys,
                        const int32_t* ctx_lens, uint16_t* landmarks, void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_chunk(chunk, chunk))) return rc;
  CKV_PTR(keys);
  CKV_PTR(ctx_lens);
  CKV_PTR(landmarks);
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, nullptr, nullptr, 1);
  LandmarkArgs a;
  a.keys = keys;
  a.ctx_lens = ctx_lens;
  a.landmarks = landmarks;
  a.key_stride = d.key_stride;
  a.Hkv = d.Hkv;
  a.max_ctx = d.max_ctx;
  a.chunk = chunk;
  a.cmax = (d.max_ctx + chunk - 1) / chunk;
  a.items = (int64_t)d.U * a.cmax * 16;
  CKV_TRY_HIP(launch_landmarks(a, (hipStream_t)stream), "landmarks launch");
  return CKV_OK;
}

int ckv_select_chunks(const ckv_shape* shape, int32_t chunk, const uint16_t* q_sel,
                      const uint16_t* landmarks, const int32_t* ctx_lens, int32_t k,
                      float scale, int32_t* chunk_idx, int32_t* n_chunks, int32_t* rows,
                      int32_t* n_rows, void* ws, size_t ws_bytes, void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_chunk(chunk, k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  CKV_PTR(q_sel);
  CKV_PTR(landmarks);
  CKV_PTR(ctx_lens);
  CKV_PTR(chunk_idx);
  CKV_PTR(n_chunks);
  CKV_PTR(rows);
  CKV_PTR(n_rows);
  Layout L = make_layout(d, k, CKV_ENTRY_CRITICAL_KV_ATTN);
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, nullptr, nullptr, k);
  return run_select_chunks(d, chunk, q_sel, landmarks, ctx_lens, k, scale, chunk_idx,
                           n_chunks, rows, n_rows, ws, (hipStream_t)stream);
}

int ckv_chunked_kv_attn(const ckv_shape* shape, int32_t chunk, const uint16_t* q_att,
                        const uint16_t* q_sel, const uint16_t* landmarks,
                        const int32_t* ctx_lens, int32_t k, float scale,
                        const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                        int32_t* chunk_idx, int32_t* n_chunks, int32_t* rows,
                        int32_t* n_rows, float* out, void* ws, size_t ws_bytes,
                        void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_chunk(chunk, k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  CKV_PTR(q_att);
  if (!q_sel) q_sel = q_att;
  CKV_PTR(q_sel);
  CKV_PTR(landmarks);
  CKV_PTR(ctx_lens);
  CKV_PTR(k_src);
  CKV_PTR(v_src);
  CKV_PTR(chunk_idx);
  CKV_PTR(n_chunks);
  CKV_PTR(rows);
  CKV_PTR(n_rows);
  CKV_PTR(out);
  if ((rc = resolve_src(src_kind, &k_src, &v_src))) return rc;
  Layout L = make_layout(d, k, CKV_ENTRY_CRITICAL_KV_ATTN);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, nullptr, nullptr, k);
  hipStream_t s = (hipStream_t)stream;
  // the partials live past everything the chunk selection used
  AttnArgs at_ = attn_args(d, L, ws, q_att, k_src, v_src, rows, n_rows, d.kv_stride, k, scale,
                           out);
  if (chunk > 1 && chunk_select_attn(d, chunk, k)) {
    SelectArgs sa;
    ExpandArgs e;
    if ((rc = score_chunks(d, chunk, q_sel, landmarks, ctx_lens, k, scale, chunk_idx, n_chunks,
                           rows, n_rows, ws, s, &sa, &e)))
      return rc;
    CKV_TRY_HIP(launch_select_attn_chunks(sa, at_, e, d.G, s), "chunk select-attention launch");
    return CKV_OK;
  }
  if ((rc = run_select_chunks(d, chunk, q_sel, landmarks, ctx_lens, k, scale, chunk_idx,
                              n_chunks, rows, n_rows, ws, s)))
    return rc;
  return run_attention(at_, d, true, s);
}

}  // extern "C"

bool ckv::loop_defers(const ckv_shape* shape, int32_t k, size_t ws_bytes) {
  Dims d;
  if (!shape || check_shape(shape, &d) != CKV_OK || k < 1) return false;
  return ws_bytes >= make_layout(d, k, CKV_ENTRY_DECODE_STEP).total;
}

// rank == 0: misses fetched whole; else their keys rebuilt from u_fac/w_fac
int ckv::corrected_impl(const ckv_shape* shape, const uint16_t* q_att, const uint16_t* q_sel,
                        const uint16_t* k_score, const int32_t* ctx_lens, int32_t k,
                        float scale, const uint16_t* k_src, const uint16_t* v_src,
                        int src_kind, int32_t rank, const uint16_t* u_fac,
                        const uint16_t* w_fac, const int32_t* idx_pred, const int32_t* n_pred,
                        uint16_t* k_buf, uint16_t* v_buf, int32_t* idx_true, int32_t* n_true,
                        int32_t* hits, int32_t* idx_next, int32_t* n_next, float* out,
                        void* ws, size_t ws_bytes, void* stream, bool hist_clean) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_scale(scale))) return rc;
  CKV_PTR(q_att);
  if (!q_sel) q_sel = q_att;
  CKV_PTR(q_sel);
  CKV_PTR(k_score);
  CKV_PTR(ctx_lens);
  if (rank > 0) {
    if ((rc = check_rank(rank))) return rc;
    CKV_PTR(u_fac);
    CKV_PTR(w_fac);
    if (!k_src) k_src = v_src;  // not read
  }
  CKV_PTR(k_src);
  CKV_PTR(v_src);
  CKV_PTR(idx_pred);
  CKV_PTR(n_pred);
  CKV_PTR(k_buf);
  CKV_PTR(v_buf);
  CKV_PTR(idx_true);
  CKV_PTR(n_true);
  CKV_PTR(hits);
  CKV_PTR(idx_next);
  CKV_PTR(n_next);
  CKV_PTR(out);
  if ((rc = resolve_src(src_kind, &k_src, &v_src))) return rc;
  Layout L = make_layout(d, k, CKV_ENTRY_CORRECTED_ATTN);
  if ((rc = check_grid(d, L))) return rc;
  if ((rc = check_ws(ws, ws_bytes, L))) return rc;
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, ctx_lens, idx_pred, n_pred, k);
  hipStream_t s = (hipStream_t)stream;
  float* scores = at<float>(ws, L.scores);
  // 1. the current token's own selection
  SelectArgs s1 = select_args(d, L, ws, scores, ctx_lens, k, idx_true, n_true);
  ScoreArgs c1 = score_args(d, L, q_att, k_score, ctx_lens, scale, scores, &s1);
  // the next step's selection (4. below) is scored by the dual kernel
  SelectArgs s2 = select_args(d, L, ws, scores, ctx_lens, k, idx_next, n_next);
  s2.hist = at<uint32_t>(ws, L.hist2);
  s2.coarse = at<uint32_t>(ws, L.coarse2);
  s2.ctrl = at<uint32_t>(ws, L.ctrl2);
  ScoreArgs c2 = score_args(d, L, q_sel, k_score, ctx_lens, scale, scores, &s2);
  // static ranges: beside this call's own gather of the misses, claims made
  // the long-context loop slower (137.2 against 136.7 ms per step)
  c2.claim = nullptr;
  const int nwg1 = score_blocks(c1, d.G, ScoreKind::kHist);
  const int nwg2 = score_blocks(c2, d.G, ScoreKind::kDualIndexed);
  if (use_partials(d, L, nwg1) && use_partials(d, L, nwg2)) {
    // both selections use the slots in turn: the first reads them before the
    // dual launch writes them again
    set_partials(ws, L, nwg1, &c1, &s1);
    set_partials(ws, L, nwg2, &c2, &s2);
  } else if (!hist_clean) {
    CKV_TRY_HIP(launch_zero(ws, L.zero_end, s), "zero launch");
  }
  CKV_TRY_HIP(launch_score(c1, d.G, true, nwg1, s), "score launch");
  if ((rc = run_select_tail(s1, d.U, s))) return rc;
  // 2. hits and misses against the predicted set; misses into free slots
  MissArgs m;
  m.idx_true = idx_true;
  m.n_true = n_true;
  m.idx_pred = idx_pred;
  m.n_pred = n_pred;
  m.slot_of = at<int32_t>(ws, L.slot_of);
  m.miss_pos = at<int32_t>(ws, L.miss_pos);
  m.miss_slot = at<int32_t>(ws, L.miss_slot);
  m.n_miss = at<int32_t>(ws, L.n_miss);
  m.hits = hits;
  m.free_slot = L.free_slot ? at<int32_t>(ws, L.free_slot) : nullptr;
  m.k = k;
  CKV_TRY_HIP(launch_miss(m, d.U, s), "miss launch");
  GatherArgs g;
  g.k_src = k_src;
  g.v_src = v_src;
  g.idx = m.miss_pos;
  g.n_sel = m.n_miss;
  g.slots = m.miss_slot;
  g.k_dst = rank > 0 ? nullptr : k_buf;
  g.v_dst = v_buf;
  g.row_stride = d.kv_stride;
  g.items = (int64_t)d.U * k * 32;
  g.max_ctx = d.max_ctx;
  g.k = k;
  if (rank > 0) {
    ReconArgs r = recon_args(d, rank, u_fac, w_fac, m.miss_pos, m.n_miss, m.miss_slot, k,
                             k_buf);
    CKV_TRY_HIP(launch_miss_fill(g, gather_blocks(src_kind), r, s), "miss fill launch");
  } else {
    CKV_TRY_HIP(launch_gather(g, gather_blocks(src_kind), s), "miss gather launch");
  }
  // 3. attention over exactly the selected rows, now all in the buffer (read
  //    through the slot list), in one launch with 4. the next step's scoring
  // the buffer as an indexed source: unit u's slot r is row r of [U][k][d]
  Dims db = d;
  db.max_ctx = k;
  AttnArgs at_ = attn_args(db, L, ws, q_att, k_buf, v_buf, m.slot_of, n_true, kD, k, scale,
                           out);
  CKV_TRY_HIP(launch_dual(at_, c2, d.G, true, d.U, nwg2, s), "dual launch");
  return select_and_merge(s2, at_, d, s);
}

extern "C" {

int ckv_corrected_attn(const ckv_shape* shape, const uint16_t* q_att, const uint16_t* q_sel,
                       const uint16_t* k_score, const int32_t* ctx_lens, int32_t k,
                       float scale, const uint16_t* k_src, const uint16_t* v_src,
                       int src_kind, const int32_t* idx_pred, const int32_t* n_pred,
                       uint16_t* k_buf, uint16_t* v_buf, int32_t* idx_true,
                       int32_t* n_true, int32_t* hits, int32_t* idx_next, int32_t* n_next,
                       float* out, void* ws, size_t ws_bytes, void* stream) {
  return ckv::corrected_impl(shape, q_att, q_sel, k_score, ctx_lens, k, scale, k_src, v_src,
                             src_kind, 0, nullptr, nullptr, idx_pred, n_pred, k_buf, v_buf,
                             idx_true, n_true, hits, idx_next, n_next, out, ws, ws_bytes,
                             stream, false);
}

int ckv_corrected_attn_lowrank(const ckv_shape* shape, const uint16_t* q_att,
                               const uint16_t* q_sel, const uint16_t* k_score,
                               const int32_t* ctx_lens, int32_t k, float scale,
                               const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                               int32_t rank, const uint16_t* u_fac, const uint16_t* w_fac,
                               const int32_t* idx_pred, const int32_t* n_pred,
                               uint16_t* k_buf, uint16_t* v_buf, int32_t* idx_true,
                               int32_t* n_true, int32_t* hits, int32_t* idx_next,
                               int32_t* n_next, float* out, void* ws, size_t ws_bytes,
                               void* stream) {
  int rc = check_rank(rank);
  if (rc) return rc;
  return ckv::corrected_impl(shape, q_att, q_sel, k_score, ctx_lens, k, scale, k_src, v_src,
                             src_kind, rank, u_fac, w_fac, idx_pred, n_pred, k_buf, v_buf,
                             idx_true, n_true, hits, idx_next, n_next, out, ws, ws_bytes,
                             stream, false);
}

int ckv_reconstruct_keys(const ckv_shape* shape, int32_t rank, const uint16_t* u_fac,
                         const uint16_t* w_fac, const int32_t* idx, const int32_t* n_sel,
                         int32_t k, uint16_t* k_dst, void* stream) {
  Dims d;
  int rc = check_shape(shape, &d);
  if (rc) return rc;
  if ((rc = check_k(k))) return rc;
  if ((rc = check_rank(rank))) return rc;
  CKV_PTR(u_fac);
  CKV_PTR(w_fac);
  CKV_PTR(idx);
  CKV_PTR(n_sel);
  CKV_PTR(k_dst);
  if (d.U == 0) return CKV_OK;
  CKV_DEBUG_CHECK(stream, nullptr, idx, n_sel, k);
  ReconArgs r = recon_args(d, rank, u_fac, w_fac, idx, n_sel, nullptr, k, k_dst);
  CKV_TRY_HIP(launch_reconstruct(r, (hipStream_t)stream), "reconstruct launch");
  return CKV_OK;
}

}  // extern "C"
