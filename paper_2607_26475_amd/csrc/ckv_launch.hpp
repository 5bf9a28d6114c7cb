// ckv_launch.hpp -- host-side launchers of the libckv kernels.
#pragma once

#include "ckv.h"
#include "ckv_device.hpp"

namespace ckv {

// Sets the thread-local detail text of ckv_last_error_detail() and returns
// code; hip_fail reports a failed HIP call as CKV_EHIP.
int fail(int code, const char* fmt, ...);
int hip_fail(hipError_t e, const char* what);
const char* last_detail();

// The read-rate probe: the rows idx[u][0 .. k) of each unit, read with the
// access pattern of one attention launch (mode: CKV_PROBE_*) and no
// arithmetic; sink gets one checksum per thread.
struct ProbeArgs {
  const uint16_t* k_rows;
  const uint16_t* v_rows;
  const int32_t* idx;   // [units][k]
  uint32_t* sink;       // probe_sink_words(units, k, mode) words
  int64_t row_stride;   // elements between a unit's rows
  int max_ctx, k, units;
};
size_t probe_sink_words(int64_t units, int k, int mode);

// Debug mode's check of an entry's device-side inputs (each may be null):
// 0 <= ctx_lens[b] <= max_ctx; 0 <= n_sel[u] <= k; idx[u][i] for i below
// n_sel[u] (below k without n_sel) is -1 or in [0, n_b) (n_b = max_ctx
// without ctx_lens).  *flag: the smallest violation code, kind << 40 | item
// (kind 1: ctx_lens[b], 2: n_sel[u], 3: idx entry u*k + i), or all ones.
struct CheckArgs {
  const int32_t* ctx_lens;
  const int32_t* idx;
  const int32_t* n_sel;
  unsigned long long* flag;
  int B, Hkv, max_ctx, k;
};
hipError_t launch_check(const CheckArgs& a, hipStream_t s);
// In debug mode, checks those inputs on the device, synchronising `s`;
// CKV_EINVAL names the first violation.  Otherwise returns CKV_OK at once.
int debug_check(hipStream_t s, const int32_t* ctx_lens, const int32_t* idx,
                const int32_t* n_sel, int B, int Hkv, int max_ctx, int k);
hipError_t launch_probe(const ProbeArgs& a, int mode, hipStream_t s);

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_fill(void* p, size_t bytes, uint32_t pattern, hipStream_t s);
// The kernel that runs a scoring pass: scores only, scores with the
// first-digit histogram (chunk landmarks when a.chunk > 1), or the scoring
// role of the one-launch attend-and-score kernel (buffer or rows in place).
// kDual2*: the same with the two tokens' 2G head rows attending (G <= 8).
enum class ScoreKind {
  kPlain, kHist, kDual, kDualIndexed, kDual2, kDual2Indexed, kDualSel, kDualSelIndexed,
  kDual2Sel, kDual2SelIndexed
};
// Workgroups of that scoring pass for these arguments.  A call computes it
// once and passes the same value to the launcher and to the selection, whose
// histogram slots depend on it.
int score_blocks(const ScoreArgs& a, int G, ScoreKind kind);
hipError_t launch_score(const ScoreArgs& a, int G, bool hist, int nwg, hipStream_t s);
hipError_t launch_hist(const SelectArgs& a, int units, hipStream_t s);
hipError_t launch_filter(const SelectArgs& a, int units, hipStream_t s);
hipError_t launch_finish(const SelectArgs& a, int units, hipStream_t s);
hipError_t launch_select_fused(const SelectArgs& a, int units, hipStream_t s);
hipError_t launch_attn(const AttnArgs& a, int G, bool indexed, int units, hipStream_t s);
// same-step selection and attention in one launch: heads == 1, nsplit shares
// of rows per unit (partials [U][nsplit][G] for k_combine when nsplit > 1);
// heads == 2 (G even, nsplit 1), two workgroups per unit attending with half
// the heads each over the whole set, outputs written directly.  merge (heads
// 1, nsplit 2 only): the two row shares merge in the launch through
// merge->merge and at.part, written directly too (no k_combine)
hipError_t launch_select_attn(const SelectArgs& sa, const AttnArgs& at, int G, int nsplit,
                              int heads, const FusedSync* merge, hipStream_t s);
// the same-step layer in one launch (k_critical): scoring on nwg workgroups
// with XCD-affine ranges and slots (sa.affine set, sa.score_nwg = nwg), then
// the selection and attention by two workgroups per unit, with half the
// heads each or (rows) with half the rows each, merged in the launch through
// fs.merge and at.part; 0 workgroups when the launch does not apply (G odd or
// above 8, U or nwg not multiples of 8, or more scoring workgroups than fit on
// the device at once).
int critical_blocks(int G, int units, int nwg, bool rows);
hipError_t launch_critical(const ScoreArgs& sc, const SelectArgs& sa, const AttnArgs& at,
                           const FusedSync& fs, int G, int nwg, bool rows, hipStream_t s);
// the same over chunks (sa: the chunk problem, k / chunk <= kFinishThreads;
// e: the rows written as k_expand writes them; G even, k <= kSelAttnMaxShare)
hipError_t launch_select_attn_chunks(const SelectArgs& sa, const AttnArgs& at,
                                    const ExpandArgs& e, int G, hipStream_t s);
hipError_t launch_combine(const AttnArgs& a, int G, int units, hipStream_t s);
// co-batched dual-token attention over the assembled buffer, two workgroups
// per unit (one per token), outputs written directly (G heads per token)
hipError_t launch_dual_token_wg(const AttnArgs& a, int G, int units, hipStream_t s);
// The one-launch attend-and-score kernel: attention over the buffer or rows in
// place (indexed) with G head rows, or with the 2G rows of two tokens when
// at.q2 is set; scoring with G heads on nwg workgroups.
hipError_t launch_dual(const AttnArgs& at, const ScoreArgs& sc, int G, bool indexed,
                       int units, int nwg, hipStream_t s);
// The same (static scoring ranges with per-workgroup histogram slots; one
// token, or two when at.q2 is set) with the previous layer's selection `sel`
// (its own slots, n_b <= kFusedSelectMaxCtx) as a third role: sel.units
// workgroups first; nwg from score_blocks with ScoreKind::kDual(2)Sel(Indexed).
hipError_t launch_dual_sel(const AttnArgs& at, const ScoreArgs& sc, const SelectArgs& sel,
                           int G, bool indexed, int units, int nwg, hipStream_t s);
hipError_t launch_miss(const MissArgs& a, int units, hipStream_t s);
hipError_t launch_landmarks(const LandmarkArgs& a, hipStream_t s);
hipError_t launch_expand(const ExpandArgs& a, int units, hipStream_t s);
hipError_t launch_reconstruct(const ReconArgs& a, hipStream_t s);
// value fetch (gather with k_dst NULL) and key rebuild of the misses in one launch
hipError_t launch_miss_fill(const GatherArgs& g, int fetch_blocks, const ReconArgs& r,
                            hipStream_t s);
hipError_t launch_gather(const GatherArgs& a, int max_blocks, hipStream_t s);

// Compute units of the current device (queried once per device).
int device_cus();

// Device address of the current device's fixed scratch array
// (CKV_NOALLOC_SCRATCH_BYTES), asked of the runtime on the first call per
// device.
int noalloc_scratch(void** ptr);

// One pipelined layer of the decode loop (Sec. 4.1, Sec. 5.2-5.4): attention
// of q_att over the set selected one step earlier (assembled in k_buf/v_buf,
// or rows idx_in of k_src/v_src in place, n_sel_in rows) and, in the same
// launch, the scoring of the next step's selection with q_sel (NULL: q_att):
// of the keys k_score, or, with chunk > 1, of the chunk landmarks, whose k /
// chunk best chunks are expanded to rows; idx_out/n_sel_out get the rows.
// With out_spec set, the speculative token (query q_sel) attends in the same
// launch over the same rows and the two tokens' own rows k_local/v_local
// ([B][Hkv][2][d], causal), as ckv_dual_token_attn.  Workspace:
// CKV_ENTRY_DECODE_STEP.
struct PipelinedLayer {
  const uint16_t* q_att;
  const uint16_t* q_sel;
  const uint16_t* k_score;
  int32_t chunk;
  const uint16_t* landmarks;
  const uint16_t* k_src;
  const uint16_t* v_src;
  int src_kind;
  const int32_t* idx_in;
  const uint16_t* k_buf;
  const uint16_t* v_buf;
  const int32_t* n_sel_in;
  int32_t* idx_out;
  int32_t* n_sel_out;
  float* out;
  const uint16_t* k_local;
  const uint16_t* v_local;
  float* out_spec;
  bool hist_clean;  // the workspace's selection histograms are known clear
};
struct LoopLink;
// link (two-token layers of the loop without buffers; see LoopLink): this
// layer's scores and slots in the decode step layout's second region when
// link->alt, the previous two-token layer's pending selection folded into
// this launch, this layer's selection left to the next one.
int pipelined_layer(const ckv_shape* shape, const PipelinedLayer& p, const int32_t* ctx_lens,
                    int32_t k, float scale, void* ws, size_t ws_bytes, void* stream,
                    LoopLink* link = nullptr);

// Plain pipelined layers of the decode loop without buffers: a layer may leave
// its selection (its sets for the next step) to the next layer's launch,
// which runs it as a third role.  alt: this layer's scores and histogram
// slots go to the decode step layout's second region (consecutive layers
// alternate, so the previous layer's stay intact); prev: the previous
// layer's pending selection, run by this call (in its launch when it can);
// next (may be null): where this layer leaves its own selection if it
// defers it (then *deferred is set and its attention partials are merged by
// a merge launch instead).  The caller runs a pending selection itself
// (launch_select_fused) before anything else uses the workspace.
struct LoopLink {
  bool alt = false;
  const SelectArgs* prev = nullptr;
  SelectArgs* next = nullptr;
  bool deferred = false;
};
// Whether a workspace of ws_bytes holds the second region (the decode step
// layout's), so that the loop may defer selections.
bool loop_defers(const ckv_shape* shape, int32_t k, size_t ws_bytes);

// ckv_critical_kv_attn and ckv_corrected_attn(_lowrank: rank > 0), for
// callers that run several calls in order on one workspace: with hist_clean
// a pipelined call skips the clearing of the selection histograms, which a
// selection whose histograms were counted atomically leaves clear (the
// previous call on the same workspace layout).
int critical_impl(const ckv_shape* shape, const uint16_t* q_att, const uint16_t* q_sel,
                  const uint16_t* k_score, const int32_t* ctx_lens, int32_t k, float scale,
                  const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                  const int32_t* idx_in, const uint16_t* k_buf, const uint16_t* v_buf,
                  const int32_t* n_sel_in, int32_t* idx_out, int32_t* n_sel_out, float* out,
                  void* ws, size_t ws_bytes, void* stream, bool hist_clean,
                  LoopLink* link = nullptr);
int corrected_impl(const ckv_shape* shape, const uint16_t* q_att, const uint16_t* q_sel,
                   const uint16_t* k_score, const int32_t* ctx_lens, int32_t k, float scale,
                   const uint16_t* k_src, const uint16_t* v_src, int src_kind, int32_t rank,
                   const uint16_t* u_fac, const uint16_t* w_fac, const int32_t* idx_pred,
                   const int32_t* n_pred, uint16_t* k_buf, uint16_t* v_buf, int32_t* idx_true,
                   int32_t* n_true, int32_t* hits, int32_t* idx_next, int32_t* n_next,
                   float* out, void* ws, size_t ws_bytes, void* stream, bool hist_clean);

// Largest gather grid a caller may ask for.
constexpr int kMaxGatherWgs = 4096;
// ckv_gather_kv with an explicit grid: `workgroups` (0: the default for
// src_kind) bounds the workgroups that stream the rows.
int gather_kv_width(const ckv_shape* shape, const uint16_t* k_src, const uint16_t* v_src,
                    int src_kind, const int32_t* idx, const int32_t* n_sel, int32_t k,
                    uint16_t* k_dst, uint16_t* v_dst, int workgroups, void* stream);

}  // namespace ckv
