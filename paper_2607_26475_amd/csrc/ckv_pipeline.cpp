// ckv_pipeline.cpp -- the two-buffer decode loop: compute stream and copy
// stream ordered by fill and release events.
#include <hip/hip_runtime.h>

#include <new>

#include "ckv.h"
#include "ckv_launch.hpp"

struct ckv_pipeline {
  hipEvent_t filled[2];  // buffer i holds the rows of the layer about to use it
  hipEvent_t freed[2];   // the attention that read buffer i has been enqueued before this
  unsigned long long filled_capture[2];  // capture filled[i] was last recorded in (0: none)
  int parity;            // buffer of the next layer to compute
  int gather_wgs;        // workgroups of each refill (0: the gather's default)
  unsigned checks;       // CKV_PIPE_CHECK_* flags (tests of the event protocol)
};

namespace {

// A layer that the plain entries do not cover: chunk landmarks or two tokens.
bool special_layer(const ckv_layer& L) { return L.chunk > 1 || L.out_spec != nullptr; }

// Which workspace layout a layer's selections use: consecutive layers with
// the same layout find the selection histograms as the previous layer left
// them (clear), so only the first of them clears.
int layout_of(const ckv_layer& L) {
  if (L.chunk > 1) return 1000 + L.chunk;  // the chunk problem's layout
  if (L.out_spec) return 3;                // the decode step's layout
  return L.idx_true ? 2 : 1;               // corrected, or the fused entry's
}

int run_special(const ckv_shape* shape, const ckv_layer& L, const int32_t* ctx_lens,
                int32_t k, float scale, int src_kind, const uint16_t* k_buf,
                const uint16_t* v_buf, void* ws, size_t ws_bytes, void* stream,
                bool hist_clean, ckv::LoopLink* link = nullptr) {
  ckv::PipelinedLayer p;
  p.q_att = L.q_att;
  p.q_sel = L.q_sel;
  p.k_score = L.k_score;
  p.chunk = L.chunk;
  p.landmarks = L.landmarks;
  p.k_src = L.k_src;
  p.v_src = L.v_src;
  p.src_kind = src_kind;
  p.idx_in = k_buf ? nullptr : L.idx_prev;  // no buffers: rows read in place
  p.k_buf = k_buf;
  p.v_buf = v_buf;
  p.n_sel_in = L.n_sel_prev;
  p.idx_out = L.idx_next;
  p.n_sel_out = L.n_sel_next;
  p.out = L.out;
  p.k_local = L.k_local;
  p.v_local = L.v_local;
  p.out_spec = L.out_spec;
  p.hist_clean = hist_clean;
  return ckv::pipelined_layer(shape, p, ctx_lens, k, scale, ws, ws_bytes, stream, link);
}

// Id of the stream capture s takes part in, 0 if it is not capturing.
unsigned long long capture_id(hipStream_t s) {
  hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
  unsigned long long id = 0;
  if (hipStreamGetCaptureInfo(s, &st, &id) != hipSuccess) return 0;
  return st == hipStreamCaptureStatusActive ? id : 0;
}

// Refill grid when the caller set none.  A gather reading pinned host memory
// with one workgroup per CU slows the compute stream's kernels several-fold
// while it runs; a narrow one (80 workgroups carry most of the link's rate)
// leaves them most of their speed.  The compute stream reads about
// max_ctx/(2k) times the bytes the link carries per layer (the scoring
// pass's keys against the selected K|V rows); from a ratio of 32 on, its
// slowed kernels, not the link, would set the step time.
constexpr int kNarrowRefillWgs = 80;

int refill_width(const ckv_pipeline* p, const ckv_shape* shape, int32_t k, int src_kind) {
  if (p->gather_wgs || src_kind != CKV_SRC_HOST_PINNED || !shape || k < 1) return p->gather_wgs;
  return (int64_t)shape->max_ctx >= 64 * (int64_t)k ? kNarrowRefillWgs : 0;
}

int gather_layer(const ckv_pipeline* p, const ckv_shape* shape, int32_t k, const ckv_layer& L,
                 const int32_t* idx, const int32_t* n_sel, int src_kind, uint16_t* kb,
                 uint16_t* vb, void* stream) {
  return ckv::gather_kv_width(shape, L.k_src, L.v_src, src_kind, idx, n_sel, k, kb, vb,
                              refill_width(p, shape, k, src_kind), stream);
}

}  // namespace

extern "C" {

int ckv_pipeline_create(ckv_pipeline** pipe) {
  if (!pipe) return ckv::fail(CKV_EINVAL, "pipe is NULL");
  ckv_pipeline* p = new (std::nothrow) ckv_pipeline();
  if (!p) return ckv::fail(CKV_EINVAL, "out of host memory");
  for (int i = 0; i < 2; ++i) {
    hipError_t e = hipEventCreateWithFlags(&p->filled[i], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&p->freed[i], hipEventDisableTiming);
    if (e != hipSuccess) {
      delete p;
      return ckv::hip_fail(e, "pipeline event creation");
    }
  }
  p->parity = 0;
  p->gather_wgs = 0;
  p->checks = 0;
  p->filled_capture[0] = p->filled_capture[1] = 0;
  *pipe = p;
  return CKV_OK;
}

int ckv_pipeline_set_gather_width(ckv_pipeline* pipe, int workgroups) {
  if (!pipe) return ckv::fail(CKV_EINVAL, "pipe is NULL");
  if (workgroups < 0 || workgroups > ckv::kMaxGatherWgs)
    return ckv::fail(CKV_EINVAL, "gather width %d outside [0, %d]", workgroups,
                     ckv::kMaxGatherWgs);
  pipe->gather_wgs = workgroups;
  return CKV_OK;
}

int ckv_pipeline_set_checks(ckv_pipeline* pipe, unsigned flags) {
  if (!pipe) return ckv::fail(CKV_EINVAL, "pipe is NULL");
  if (flags & ~(unsigned)(CKV_PIPE_CHECK_NO_FILL_WAIT | CKV_PIPE_CHECK_NO_RELEASE_WAIT |
                          CKV_PIPE_CHECK_POISON | CKV_PIPE_CHECK_NO_DEFER))
    return ckv::fail(CKV_EINVAL, "unknown check flags 0x%x", flags);
  pipe->checks = flags;
  return CKV_OK;
}

int ckv_pipeline_destroy(ckv_pipeline* pipe) {
  if (!pipe) return CKV_OK;
  for (int i = 0; i < 2; ++i) {
    (void)hipEventDestroy(pipe->filled[i]);
    (void)hipEventDestroy(pipe->freed[i]);
  }
  delete pipe;
  return CKV_OK;
}

int ckv_pipeline_prime(ckv_pipeline* pipe, const ckv_shape* shape, int32_t k,
                       const ckv_layer* layers, int num_layers, int src_kind,
                       uint16_t* const k_buf[2], uint16_t* const v_buf[2],
                       void* copy_stream) {
  if (!pipe || !layers || num_layers < 2 || !k_buf || !v_buf)
    return ckv::fail(CKV_EINVAL, "pipe, layers (at least 2) and both buffers are required");
  pipe->parity = 0;
  for (int l = 0; l < 2; ++l) {
    int rc = gather_layer(pipe, shape, k, layers[l], layers[l].idx_prev, layers[l].n_sel_prev,
                          src_kind, k_buf[l], v_buf[l], copy_stream);
    if (rc) return rc;
    hipError_t e = hipEventRecord(pipe->filled[l], (hipStream_t)copy_stream);
    if (e != hipSuccess) return ckv::hip_fail(e, "fill event record");
    pipe->filled_capture[l] = capture_id((hipStream_t)copy_stream);
  }
  return CKV_OK;
}

int ckv_decode_step(ckv_pipeline* pipe, const ckv_shape* shape, int num_layers,
                    const ckv_layer* layers, const int32_t* ctx_lens, int32_t k,
                    float scale, int src_kind, uint16_t* const k_buf[2],
                    uint16_t* const v_buf[2], void* ws, size_t ws_bytes,
                    void* compute_stream, void* copy_stream) {
  if (!pipe || !layers || num_layers < 1)
    return ckv::fail(CKV_EINVAL, "pipe and layers are required");
  if (!k_buf && !v_buf) {
    // rows read in place through last step's index sets: no buffers, no refills
    for (int l = 0; l < num_layers; ++l)
      if (layers[l].idx_true)
        return ckv::fail(CKV_EINVAL, "layer %d: miss correction needs the two buffers", l);
    // With the decode step's workspace, a plain layer followed by a plain
    // layer, or a two-token layer followed by a two-token layer, leaves its
    // selection (the sets for the next step, not needed before then) to the
    // next layer's launch; consecutive layers of a kind alternate between two
    // regions of scores and histogram slots.  A pending selection runs on its
    // own before a layer of another kind and after the last layer.
    const bool defers =
        ckv::loop_defers(shape, k, ws_bytes) && !(pipe->checks & CKV_PIPE_CHECK_NO_DEFER);
    hipStream_t cs = (hipStream_t)compute_stream;
    ckv::SelectArgs pend, mine;
    bool have = false;
    auto flush = [&]() -> int {
      if (!have) return CKV_OK;
      have = false;
      if (hipError_t e = ckv::launch_select_fused(pend, pend.units, cs))
        return ckv::hip_fail(e, "select launch");
      return CKV_OK;
    };
    // 0: plain, 1: two tokens, 2: chunked (never deferred)
    auto kind_of = [](const ckv_layer& L) { return L.chunk > 1 ? 2 : L.out_spec ? 1 : 0; };
    int pend_kind = -1;
    for (int l = 0; l < num_layers; ++l) {
      const ckv_layer& L = layers[l];
      const int kind = kind_of(L);
      const bool clean = l > 0 && layout_of(L) == layout_of(layers[l - 1]);
      int rc;
      if (have && pend_kind != kind)
        if ((rc = flush())) return rc;
      ckv::LoopLink link;
      link.alt = (l & 1) != 0;
      link.prev = have ? &pend : nullptr;
      link.next = l + 1 < num_layers && kind_of(layers[l + 1]) == kind ? &mine : nullptr;
      ckv::LoopLink* lk = defers && kind != 2 ? &link : nullptr;
      if (kind != 0)
        rc = run_special(shape, L, ctx_lens, k, scale, src_kind, nullptr, nullptr, ws, ws_bytes,
                         compute_stream, clean, lk);
      else
        rc = ckv::critical_impl(shape, L.q_att, L.q_sel, L.k_score, ctx_lens, k, scale, L.k_src,
                                L.v_src, src_kind, L.idx_prev, nullptr, nullptr, L.n_sel_prev,
                                L.idx_next, L.n_sel_next, L.out, ws, ws_bytes, compute_stream,
                                clean, lk);
      if (rc) return rc;
      have = lk && link.deferred;
      if (have) {
        pend = mine;
        pend_kind = kind;
      }
    }
    return flush();
  }
  if (num_layers < 2 || !k_buf || !v_buf)
    return ckv::fail(CKV_EINVAL, "the two-buffer loop needs at least 2 layers and both buffers");
  for (int l = 0; l < num_layers; ++l)
    if (layers[l].idx_true && special_layer(layers[l]))
      return ckv::fail(CKV_EINVAL,
                       "layer %d: miss correction of a chunked or two-token layer", l);
  hipStream_t cs = (hipStream_t)compute_stream, xs = (hipStream_t)copy_stream;
  const unsigned long long capture = capture_id(cs);
  // A graph fixes each layer's buffer at capture time.  Over an odd number of
  // layers the last refills land in the buffers of the other parity, so a
  // second launch of the graph would attend over another layer's rows.
  if (capture && (num_layers & 1))
    return ckv::fail(CKV_EINVAL,
                     "a captured two-buffer step needs an even number of layers (got %d)",
                     num_layers);
  for (int l = 0; l < num_layers; ++l) {
    const int p = pipe->parity;
    const ckv_layer& L = layers[l];
    // attention over buffer p once its gather has landed.  Under stream
    // capture a fill recorded outside this capture cannot be waited for;
    // the graph is then ordered after it by its launch.
    if ((!capture || pipe->filled_capture[p] == capture) &&
        !(pipe->checks & CKV_PIPE_CHECK_NO_FILL_WAIT))
      if (hipError_t e = hipStreamWaitEvent(cs, pipe->filled[p], 0))
        return ckv::hip_fail(e, "wait for a buffer fill");
    // the previous layer of this call on the same workspace layout left the
    // selection histograms clear
    const bool clean = l > 0 && layout_of(L) == layout_of(layers[l - 1]);
    int rc;
    if (special_layer(L)) {  // chunk landmarks or two tokens
      rc = run_special(shape, L, ctx_lens, k, scale, src_kind, k_buf[p], v_buf[p], ws,
                       ws_bytes, compute_stream, clean);
    } else if (L.idx_true) {
      // the current query's own set: misses fetched into buffer p first, their
      // keys rebuilt from the low-rank factors if lr_rank > 0
      rc = ckv::corrected_impl(shape, L.q_att, L.q_sel, L.k_score, ctx_lens, k, scale,
                               L.k_src, L.v_src, src_kind, L.lr_rank > 0 ? L.lr_rank : 0,
                               L.lr_u, L.lr_w, L.idx_prev, L.n_sel_prev, k_buf[p], v_buf[p],
                               L.idx_true, L.n_true, L.hits, L.idx_next, L.n_sel_next, L.out,
                               ws, ws_bytes, compute_stream, clean);
    } else {
      rc = ckv::critical_impl(shape, L.q_att, L.q_sel, L.k_score, ctx_lens, k, scale, nullptr,
                              nullptr, src_kind, nullptr, k_buf[p], v_buf[p], L.n_sel_prev,
                              L.idx_next, L.n_sel_next, L.out, ws, ws_bytes, compute_stream,
                              clean);
    }
    if (rc) return rc;
    if (hipError_t e = hipEventRecord(pipe->freed[p], cs))
      return ckv::hip_fail(e, "release event record");
    // refill buffer p with the layer two ahead (into the next step at the end)
    if (!(pipe->checks & CKV_PIPE_CHECK_NO_RELEASE_WAIT))
      if (hipError_t e = hipStreamWaitEvent(xs, pipe->freed[p], 0))
        return ckv::hip_fail(e, "wait for a buffer release");
    if (pipe->checks & CKV_PIPE_CHECK_POISON) {  // NaN bits where the refill will go
      const size_t bytes = (size_t)shape->batch * shape->num_kv_heads * k * shape->head_dim * 2;
      if (hipError_t e = ckv::launch_fill(k_buf[p], bytes, 0xffffffffu, xs))
        return ckv::hip_fail(e, "poison launch");
      if (hipError_t e = ckv::launch_fill(v_buf[p], bytes, 0xffffffffu, xs))
        return ckv::hip_fail(e, "poison launch");
    }
    const int j = l + 2;
    if (j < num_layers) {
      rc = gather_layer(pipe, shape, k, layers[j], layers[j].idx_prev, layers[j].n_sel_prev,
                        src_kind, k_buf[p], v_buf[p], copy_stream);
    } else {
      const ckv_layer& N = layers[j - num_layers];
      rc = gather_layer(pipe, shape, k, N, N.idx_next, N.n_sel_next, src_kind, k_buf[p], v_buf[p],
                        copy_stream);
    }
    if (rc) return rc;
    if (hipError_t e = hipEventRecord(pipe->filled[p], xs))
      return ckv::hip_fail(e, "fill event record");
    pipe->filled_capture[p] = capture;
    pipe->parity ^= 1;
  }
  return CKV_OK;
}

}  // extern "C"
