/*
 * ckv.h -- C ABI of libckv: critical-KV selection and sparse decode attention
 * for MI355X (gfx950).
 *
 * The operation is the decode-step hot path of DualDecoder (arXiv
 * 2607.26475): for every (request, KV head) the positions of the context are
 * scored against a query (Sec. 2.2 and Sec. 4.1: the retrieval index comes from
 * a query and per-position key summaries; here the summary of a position is
 * its own key), the top-k positions are selected once per KV head for all
 * query heads of its GQA group, the selected K/V rows are gathered from HBM or
 * host-pinned memory into a layer-scoped GPU buffer (Sec. 5.4, GPU-side sparse
 * KV assembly), and softmax attention runs over only those rows (Sec. 5.3:
 * the result must equal attention over the selected entries).  In DualDecoder
 * the selecting query is the speculative token's (Sec. 4.1, retrieval index
 * prediction) and the attending query is the current token's (Sec. 5.2).
 *
 * Conventions shared by every entry point
 *   - Types: bf16 tensors are passed as uint16_t bit patterns; scores and
 *     outputs are fp32; positions and counts are int32.
 *   - Layouts (row-major, dense unless a stride says otherwise):
 *       q, q_att, q_sel   [B][Hq][d]                     bf16, device
 *       k_score           row j of (b,h) at element
 *                         ((b*Hkv + h)*max_ctx + j) * key_row_stride  bf16, device
 *       k_src, v_src      row j of (b,h) at element
 *                         ((b*Hkv + h)*max_ctx + j) * kv_row_stride   bf16,
 *                         device or host-pinned (src_kind); K and V may be
 *                         interleaved per row (kv_row_stride = 2d, v_src =
 *                         k_src + d)
 *       ctx_lens          [B] int32, device; n_b, clamped to [0, max_ctx]
 *       scores            [B][Hkv][max_ctx] fp32, device
 *       idx               [B][Hkv][k] int32, device; ascending positions,
 *                         then -1
 *       n_sel             [B][Hkv] int32, device; m = min(k, n_b)
 *       k_buf, v_buf      [B][Hkv][k][d] bf16, device (slot i = i-th selected)
 *       out               [B][Hq][d] fp32, device
 *     Query head q belongs to KV head q / (Hq/Hkv) (consecutive grouping).
 *   - Supported shapes: head_dim == 128; Hq % Hkv == 0 with group size
 *     G = Hq/Hkv in {1, 2, 4, 8, 16}; 1 <= max_ctx <= 2^30; 1 <= k <= 2^20;
 *     row strides >= 128 and multiples of 8 elements; every tensor pointer
 *     16-byte aligned.
 *   - Ownership: every buffer belongs to the caller; the library never
 *     allocates or frees caller memory.  Scratch memory is a caller-provided
 *     workspace of at least ckv_workspace_bytes() bytes, 256-byte aligned; its
 *     contents on entry do not matter and are undefined on return.
 *   - Streams: every call only enqueues work on `stream` (a hipStream_t; NULL
 *     is the legacy default stream) and returns without synchronising.  Calls
 *     that share a workspace must be ordered on one stream.
 *   - Errors: each call returns a ckv_status.  Argument errors are detected on
 *     the host before anything is enqueued; CKV_EHIP reports a failed launch
 *     (the HIP error code is in the detail text).  Faults during kernel
 *     execution surface at the caller's next synchronisation.  No C++
 *     exception crosses this interface.  ckv_last_error_detail() gives a
 *     thread-local description of the last failure.
 *   - Device-side preconditions (not checked, values are clamped so that no
 *     access leaves the caller's buffers): 0 <= n_b <= max_ctx; gathered idx
 *     entries lie in [0, max_ctx) (slots whose idx is outside are skipped).
 *   - Scores are compared by their fp32 value (-0 equals +0); equal scores
 *     rank the lower position first.  Inputs must be finite; scores may be
 *     -inf or +inf but not NaN (a NaN score, which finite inputs can only
 *     give through fp32 overflow, leaves the selected set unspecified while
 *     every write stays inside the caller's buffers).
 */
#ifndef CKV_H
#define CKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CKV_ABI_VERSION 9

typedef enum ckv_status {
  CKV_OK = 0,
  CKV_EINVAL = 1,        /* null pointer, misaligned pointer or bad value   */
  CKV_ESHAPE = 2,        /* Hq % Hkv != 0, k < 1, max_ctx < 1, bad stride    */
  CKV_EUNSUPPORTED = 3,  /* head_dim != 128, group size not in {1,2,4,8,16}  */
  CKV_EWORKSPACE = 4,    /* workspace NULL or smaller than required          */
  CKV_EHIP = 5           /* a HIP runtime call or kernel launch failed       */
} ckv_status;

typedef enum ckv_src_kind {
  CKV_SRC_DEVICE = 0,      /* K/V rows in device memory (HBM)                */
  CKV_SRC_HOST_PINNED = 1  /* K/V rows in host memory from hipHostMalloc or   */
                           /* torch pin_memory; read by the GPU over the host */
                           /* link, no staging copy                           */
} ckv_src_kind;

typedef enum ckv_entry {
  CKV_ENTRY_SELECT_TOPK = 1,
  CKV_ENTRY_SPARSE_DECODE_ATTN = 2,
  CKV_ENTRY_CRITICAL_KV_ATTN = 3,
  CKV_ENTRY_CORRECTED_ATTN = 4,
  CKV_ENTRY_DUAL_TOKEN_ATTN = 5,
  CKV_ENTRY_DECODE_STEP = 6  /* ckv_decode_step with any kind of layer */
} ckv_entry;

typedef struct ckv_shape {
  int32_t batch;          /* B: requests in the decode batch                  */
  int32_t num_q_heads;    /* Hq                                               */
  int32_t num_kv_heads;   /* Hkv                                              */
  int32_t head_dim;       /* d (must be 128)                                  */
  int32_t max_ctx;        /* rows stored per (request, KV head)               */
  int32_t reserved;       /* must be 0                                        */
  int64_t key_row_stride; /* elements between consecutive rows of k_score     */
  int64_t kv_row_stride;  /* elements between consecutive rows of k_src/v_src */
} ckv_shape;

/* Version of this interface (CKV_ABI_VERSION of the built library). */
int ckv_abi_version(void);

/* Static text for a status code (never NULL). */
const char* ckv_status_str(int status);

/* Thread-local description of the last failed call on this thread ("" if
 * none).  Valid until the next call on the same thread. */
const char* ckv_last_error_detail(void);

/* Workspace that `entry` needs for this shape and budget k, in bytes, stored
 * in *bytes.  Entry points not listed in ckv_entry need none. */
int ckv_workspace_bytes(const ckv_shape* shape, int32_t k, int entry,
                        size_t* bytes);

/* Sec. 2.2 / Sec. 4.1 -- retrieval scores.  For every request b, KV head h and
 * position j < n_b:
 *   scores[b][h][j] = max over the G query heads g of h's group of
 *                     scale * sum_c q[b][h*G+g][c] * k_score(b,h,j)[c]
 * computed from bf16 inputs with fp32 accumulation; positions
 * n_b <= j < max_ctx get -inf.  scale > 0 (normally 1/sqrt(d)). */
int ckv_score_keys(const ckv_shape* shape, const uint16_t* q,
                   const uint16_t* k_score, const int32_t* ctx_lens,
                   float scale, float* scores, void* stream);

/* Sec. 2.2 -- critical-entry selection within the sparse budget.  For every
 * (b, h) the m = min(k, n_b) largest scores[b][h][0..n_b), ties broken by lower
 * position, are written to idx[b][h][0..m) in ascending position order, the
 * remaining k - m slots get -1, and n_sel[b][h] = m.  One index set per KV
 * head serves all G query heads of its group.  Workspace:
 * CKV_ENTRY_SELECT_TOPK. */
int ckv_select_topk(const ckv_shape* shape, const float* scores,
                    const int32_t* ctx_lens, int32_t k, int32_t* idx,
                    int32_t* n_sel, void* ws, size_t ws_bytes, void* stream);

/* Sec. 5.4 -- GPU-side sparse KV assembly.  For i < n_sel[b][h]:
 *   k_dst[b][h][i] = K row idx[b][h][i] of (b,h) in k_src,
 *   v_dst[b][h][i] = V row idx[b][h][i] of (b,h) in v_src,
 * copied bit-exactly; slots i >= n_sel (and slots whose idx is outside
 * [0, max_ctx)) are not written.  src_kind says where k_src/v_src live; with
 * CKV_SRC_HOST_PINNED the GPU reads the rows straight from pinned host memory.
 * k_dst/v_dst are device buffers of [B][Hkv][k][d]. */
int ckv_gather_kv(const ckv_shape* shape, const uint16_t* k_src,
                  const uint16_t* v_src, int src_kind, const int32_t* idx,
                  const int32_t* n_sel, int32_t k, uint16_t* k_dst,
                  uint16_t* v_dst, void* stream);

/* Sec. 5.3 / Sec. 5.4 -- attention over the assembled sparse set.  For every
 * query head g of KV head h, with m = n_sel[b][h] (clamped to [0, k]):
 *   l_i = scale * q_att[b][g] . k_buf[b][h][i],  p = softmax(l_0..l_{m-1}),
 *   out[b][g] = sum_i p_i v_buf[b][h][i],
 * fp32 logits, weights and accumulation; out = 0 when m = 0.  Workspace:
 * CKV_ENTRY_SPARSE_DECODE_ATTN. */
int ckv_sparse_decode_attn(const ckv_shape* shape, const uint16_t* q_att,
                           const uint16_t* k_buf, const uint16_t* v_buf,
                           const int32_t* n_sel, int32_t k, float scale,
                           float* out, void* ws, size_t ws_bytes,
                           void* stream);

/* Fused decode step of one layer (Sec. 4.1, Sec. 5.2-5.4).  The selecting
 * query q_sel (the speculative token's; NULL means q_att) scores k_score and
 * picks idx_out / n_sel_out exactly as ckv_score_keys + ckv_select_topk.
 *   Same-step mode (idx_in == NULL, k_buf == NULL): out = attention of q_att
 *     over the rows idx_out of k_src / v_src (read in place, src_kind says
 *     where), i.e. ckv_sparse_decode_attn applied to ckv_gather_kv(idx_out).
 *     Where it applies, the scoring, the selection and the attention run as
 *     one launch (see ckv_set_one_launch_same_step), with the same results.
 *   Pipelined modes (Sec. 4.1: the set attended at step t was selected at
 *   step t-1 from the speculative token's query): out = attention of q_att
 *   over the set selected one step earlier, and in the same launch the
 *   context is scored with q_sel for the next step's idx_out / n_sel_out.
 *   The earlier set is either
 *     assembled (k_buf != NULL): k_buf/v_buf rows [0, n_sel_in), as
 *       ckv_gather_kv left them; k_src/v_src and idx_in are not read; or
 *     in place (idx_in != NULL): rows idx_in[b][h][0..n_sel_in[b][h]) of
 *       k_src / v_src, read where they are (the HBM-resident cache needs no
 *       buffer); idx_in must not alias idx_out.
 *   idx_in and k_buf together are CKV_EINVAL.
 * Workspace: CKV_ENTRY_CRITICAL_KV_ATTN. */
int ckv_critical_kv_attn(const ckv_shape* shape, const uint16_t* q_att,
                         const uint16_t* q_sel, const uint16_t* k_score,
                         const int32_t* ctx_lens, int32_t k, float scale,
                         const uint16_t* k_src, const uint16_t* v_src,
                         int src_kind, const int32_t* idx_in,
                         const uint16_t* k_buf, const uint16_t* v_buf,
                         const int32_t* n_sel_in, int32_t* idx_out,
                         int32_t* n_sel_out, float* out, void* ws,
                         size_t ws_bytes, void* stream);

/* ---- the fused step for callers that cannot allocate -----------------------
 * For callers that cannot allocate device memory or hold a workspace: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  ckv_critical_kv_attn, with the same arguments and results,
 * whose workspace is a fixed array of CKV_NOALLOC_SCRATCH_BYTES bytes of
 * device memory, one per device, that the library holds from its load until
 * the process ends.  The call allocates and frees nothing; the caller still
 * passes every input and output.  A shape whose workspace
 * (ckv_workspace_bytes, CKV_ENTRY_CRITICAL_KV_ATTN) is larger than
 * CKV_NOALLOC_SCRATCH_BYTES is CKV_EWORKSPACE, before anything is enqueued.
 * All calls on a device share that device's array, which keeps the last
 * call's contents (each call clears what it needs cleared): calls on one
 * device that may overlap in time (on different streams, or from threads
 * without ordering) race on it, so the caller orders them, e.g. on one
 * stream. */
#define CKV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

int ckv_critical_kv_attn_noalloc(const ckv_shape* shape, const uint16_t* q_att,
                                 const uint16_t* q_sel, const uint16_t* k_score,
                                 const int32_t* ctx_lens, int32_t k, float scale,
                                 const uint16_t* k_src, const uint16_t* v_src,
                                 int src_kind, const int32_t* idx_in,
                                 const uint16_t* k_buf, const uint16_t* v_buf,
                                 const int32_t* n_sel_in, int32_t* idx_out,
                                 int32_t* n_sel_out, float* out, void* stream);

/* Sec. 5.3 (prioritized missing KV transfer) and Sec. 5.4 (GPU-side sparse KV
 * assembly with deferred reordering) -- one layer of a pipelined decode step
 * whose attention uses the current token's own selection, not the
 * prediction.  On entry k_buf/v_buf hold, in slot order, the rows of the
 * predicted set idx_pred/n_pred: the selection made one step earlier from the
 * speculative query and gathered ahead of time.  The call
 *   1. selects idx_true/n_true from q_att exactly as ckv_score_keys +
 *      ckv_select_topk;
 *   2. gathers every row of idx_true that is missing from idx_pred from
 *      k_src/v_src (src_kind says where) into a buffer slot whose predicted
 *      row is not in idx_true, or a slot past n_pred: the buffer then holds
 *      every row of idx_true.  hits[b][h] = |idx_true ∩ idx_pred|;
 *   3. computes out = attention of q_att over exactly the rows of idx_true,
 *      the same-step result of ckv_critical_kv_attn with q_sel = q_att;
 *   4. in the same launch as that attention, selects idx_next/n_next from
 *      q_sel (the speculative query; NULL means q_att): the prediction for
 *      the next step.
 * idx_pred must be ascending in [0, max_ctx) and -1 padded, as
 * ckv_select_topk writes it; n_pred is clamped to [0, k].  k_buf/v_buf are
 * modified: slots of mispredicted rows are overwritten.  All streams run at
 * the default priority; the misses are fetched on `stream` ahead of the
 * attention that needs them.  Workspace: CKV_ENTRY_CORRECTED_ATTN. */
int ckv_corrected_attn(const ckv_shape* shape, const uint16_t* q_att,
                       const uint16_t* q_sel, const uint16_t* k_score,
                       const int32_t* ctx_lens, int32_t k, float scale,
                       const uint16_t* k_src, const uint16_t* v_src,
                       int src_kind, const int32_t* idx_pred,
                       const int32_t* n_pred, uint16_t* k_buf, uint16_t* v_buf,
                       int32_t* idx_true, int32_t* n_true, int32_t* hits,
                       int32_t* idx_next, int32_t* n_next, float* out,
                       void* ws, size_t ws_bytes, void* stream);

/* ---- adaptive key reconstruction -------------------------------------------
 * Sec. 5.3 (adaptive key reconstruction): for layers where the prediction
 * misses many rows, the keys of the missing rows are rebuilt on the GPU from
 * a low-rank key cache, and only their values come from k_src/v_src's
 * memory.  Factors per (b, h), bf16 on the device:
 *   u_fac [B][Hkv][max_ctx][rank]   w_fac [B][Hkv][rank][d]
 * Key row p of (b, h) is rebuilt as
 *   K'[p][c] = sum_{j < rank} u_fac[b][h][p][j] * w_fac[b][h][j][c],
 * summed in fp64 in ascending j (each product is exact) and rounded once to
 * bf16, nearest, ties to even.  rank is in [1, CKV_MAX_RANK]. */
#define CKV_MAX_RANK 4096

/* For i < n_sel[b][h] (clamped to [0, k]) writes K'[idx[b][h][i]] to
 * k_dst[b][h][i] ([B][Hkv][k][d]).  Entries whose idx is outside
 * [0, max_ctx), and slots i >= n_sel, are not written. */
int ckv_reconstruct_keys(const ckv_shape* shape, int32_t rank, const uint16_t* u_fac,
                         const uint16_t* w_fac, const int32_t* idx, const int32_t* n_sel,
                         int32_t k, uint16_t* k_dst, void* stream);

/* ckv_corrected_attn for a layer with key reconstruction: the same, except
 * that the key of every row of idx_true missing from idx_pred is rebuilt into
 * its slot as ckv_reconstruct_keys rebuilds it, in the same launch that
 * fetches its value from v_src (k_src is not read and may be NULL).  out is
 * the attention of q_att over the rows of idx_true, with the prefetched keys
 * for hits and the rebuilt keys for misses.  Workspace:
 * CKV_ENTRY_CORRECTED_ATTN. */
int ckv_corrected_attn_lowrank(const ckv_shape* shape, const uint16_t* q_att,
                               const uint16_t* q_sel, const uint16_t* k_score,
                               const int32_t* ctx_lens, int32_t k, float scale,
                               const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                               int32_t rank, const uint16_t* u_fac, const uint16_t* w_fac,
                               const int32_t* idx_pred, const int32_t* n_pred,
                               uint16_t* k_buf, uint16_t* v_buf, int32_t* idx_true,
                               int32_t* n_true, int32_t* hits, int32_t* idx_next,
                               int32_t* n_next, float* out, void* ws, size_t ws_bytes,
                               void* stream);

/* Sec. 5.2 (dual-token decoding, co-batched attention) -- the current token
 * T_i and the speculative token T'_{i+1} of every request attend together,
 * as two consecutive positions after the selected rows, with the causal mask
 * that hides T'_{i+1} from T_i.  k_local/v_local [B][Hkv][2][d] bf16 hold
 * the two tokens' own rows (row 0: T_i, row 1: T'_{i+1}).  With m = n_sel
 * (clamped to [0, k]):
 *   out_cur[b][g]  = attention of q_cur[b][g]  over k_buf/v_buf rows [0, m)
 *                    and local row 0,
 *   out_spec[b][g] = attention of q_spec[b][g] over the same m rows and
 *                    local rows 0 and 1,
 * fp32 as in ckv_sparse_decode_attn.  One launch reads each selected row
 * once for both tokens' 2G head rows, so G <= 8 (CKV_EUNSUPPORTED else).
 * Workspace: CKV_ENTRY_DUAL_TOKEN_ATTN. */
int ckv_dual_token_attn(const ckv_shape* shape, const uint16_t* q_cur,
                        const uint16_t* q_spec, const uint16_t* k_buf,
                        const uint16_t* v_buf, const int32_t* n_sel,
                        const uint16_t* k_local, const uint16_t* v_local, int32_t k,
                        float scale, float* out_cur, float* out_spec, void* ws,
                        size_t ws_bytes, void* stream);

/* ---- chunk landmarks --------------------------------------------------------
 * Sec. 2.2: adjacent KV entries are segmented into chunks, each with a small
 * GPU-resident landmark; the query selects chunks by their landmarks and the
 * selected chunks' entries are retrieved.  Sec. 4.1: the landmarks are built
 * before decoding and stay fixed.  A chunk holds `chunk` consecutive rows
 * (chunk >= 1; chunk 1 is the per-position path above); a unit with n_b rows
 * has ceil(n_b / chunk) chunks, the last possibly partial.
 *   landmarks   [B][Hkv][ceil(max_ctx / chunk)][d] bf16, device
 *   chunk_idx   [B][Hkv][k / chunk] int32: ascending chunk numbers, -1 padded
 *   n_chunks    [B][Hkv] int32
 *   rows        [B][Hkv][k] int32: the selected chunks' rows below n_b in
 *               ascending order, -1 padded (the idx of the other entries)
 *   n_rows      [B][Hkv] int32 */

/* Landmark c of every (b, h), for c < ceil(n_b / chunk): the mean of key rows
 * [c*chunk, min(c*chunk + chunk, n_b)) of `keys` (key_row_stride), summed in
 * fp64 in row order, divided by the row count and rounded once to bf16
 * (nearest, ties to even).  Later landmarks are not written. */
int ckv_chunk_landmarks(const ckv_shape* shape, int32_t chunk, const uint16_t* keys,
                        const int32_t* ctx_lens, uint16_t* landmarks, void* stream);

/* Chunk selection: every landmark is scored against q_sel exactly as
 * ckv_score_keys scores a key (max over the group's heads), the k / chunk
 * best chunks are selected as ckv_select_topk selects positions (ties to the
 * lower chunk; all chunks if there are fewer), and expanded to rows.  k must
 * be a multiple of chunk.  Workspace: CKV_ENTRY_CRITICAL_KV_ATTN for this
 * shape and k. */
int ckv_select_chunks(const ckv_shape* shape, int32_t chunk, const uint16_t* q_sel,
                      const uint16_t* landmarks, const int32_t* ctx_lens, int32_t k,
                      float scale, int32_t* chunk_idx, int32_t* n_chunks, int32_t* rows,
                      int32_t* n_rows, void* ws, size_t ws_bytes, void* stream);

/* Same-step decode of one layer over chunks: ckv_select_chunks with q_sel
 * (NULL means q_att), then out = attention of q_att over the rows `rows` of
 * k_src/v_src read in place (src_kind says where), i.e.
 * ckv_sparse_decode_attn over ckv_gather_kv(rows, n_rows).  Workspace:
 * CKV_ENTRY_CRITICAL_KV_ATTN for this shape and k. */
int ckv_chunked_kv_attn(const ckv_shape* shape, int32_t chunk, const uint16_t* q_att,
                        const uint16_t* q_sel, const uint16_t* landmarks,
                        const int32_t* ctx_lens, int32_t k, float scale,
                        const uint16_t* k_src, const uint16_t* v_src, int src_kind,
                        int32_t* chunk_idx, int32_t* n_chunks, int32_t* rows,
                        int32_t* n_rows, float* out, void* ws, size_t ws_bytes,
                        void* stream);

/* ---- layer pipeline --------------------------------------------------------
 * The decode loop of Sec. 5.3 (layer-aware transfer overlap) and Sec. 5.4
 * (two-layer ping-pong buffer): the set selected for a layer at step t-1 is
 * gathered into one of two layer-scoped buffers on a copy stream while the
 * compute stream works on the previous layer; the gather for layer l+2 starts
 * as soon as the attention of layer l has released its buffer.  The compute
 * stream waits for a buffer's fill event before attending over it (no
 * read-after-write hazard) and the copy stream waits for its release event
 * before refilling it (no write-after-read hazard).  Layer g of the decode
 * (counting layers across steps) uses buffer g % 2.
 *
 * Per layer the caller provides: */
typedef struct ckv_layer {
  const uint16_t* q_att;      /* [B][Hq][d] query of the current token         */
  const uint16_t* q_sel;      /* [B][Hq][d] query of the speculative token,    */
                              /* NULL => q_att                                 */
  const uint16_t* k_score;    /* scoring keys (device, key_row_stride)          */
  const uint16_t* k_src;      /* K rows gathered into the buffer (src_kind,     */
  const uint16_t* v_src;      /* kv_row_stride); V rows likewise                */
  const int32_t* idx_prev;    /* [B][Hkv][k] set selected at the previous step  */
  const int32_t* n_sel_prev;  /* [B][Hkv]                                       */
  int32_t* idx_next;          /* [B][Hkv][k] written: selected at this step     */
  int32_t* n_sel_next;        /* [B][Hkv] written                               */
  float* out;                 /* [B][Hq][d] written: attention output           */
  int32_t* idx_true;          /* NULL: attention over the predicted set.  Else  */
  int32_t* n_true;            /* the layer runs ckv_corrected_attn: [B][Hkv][k], */
  int32_t* hits;              /* [B][Hkv] and [B][Hkv] written                   */
  int32_t lr_rank;            /* > 0 (with idx_true set): misses' keys rebuilt  */
  const uint16_t* lr_u;       /* from these factors, ckv_corrected_attn_lowrank */
  const uint16_t* lr_w;       /* (u_fac, w_fac); 0/NULL otherwise               */
  int32_t chunk;              /* > 1: a chunked layer (Sec. 2.2 chunk landmarks) */
  const uint16_t* landmarks;  /* as ckv_chunk_landmarks writes them, [B][Hkv]    */
                              /* [ceil(max_ctx/chunk)][d]: its selection scores */
                              /* these with q_sel, keeps the k/chunk best chunks */
                              /* and expands them to rows (ckv_select_chunks):  */
                              /* idx_prev/idx_next hold rows; k_score unused.   */
                              /* 0/1 and NULL: one score per position           */
  const uint16_t* k_local;    /* non-NULL out_spec: two tokens (Sec. 5.2): the  */
  const uint16_t* v_local;    /* current and the speculative token attend in   */
  float* out_spec;            /* one launch, as ckv_dual_token_attn, with their */
                              /* own rows k_local/v_local [B][Hkv][2][d]; the   */
                              /* speculative token's query is q_sel and its     */
                              /* output goes to out_spec [B][Hq][d] (G <= 8)    */
} ckv_layer;

typedef struct ckv_pipeline ckv_pipeline; /* events of one decode loop */

/* Creates the events of one decode loop on the current device. */
int ckv_pipeline_create(ckv_pipeline** pipe);
int ckv_pipeline_destroy(ckv_pipeline* pipe);

/* Workgroups of every refill this loop launches on its copy stream.  A
 * gather that reads pinned host memory slows kernels on other streams while
 * it runs; a narrower one (80 workgroups carry most of the link's rate)
 * leaves the compute stream most of its speed, for loops where that stream,
 * not the link, sets the step time.  0 (the default) chooses by shape: 80
 * workgroups for pinned sources when max_ctx >= 64 k (the scoring pass then
 * reads at least 32 times the bytes the link carries per layer), else what
 * ckv_gather_kv uses (256 for pinned sources).  0 <= workgroups <= 4096,
 * else CKV_EINVAL. */
int ckv_pipeline_set_gather_width(ckv_pipeline* pipe, int workgroups);

/* For tests of the event protocol only, never for serving: breaks the
 * loop's ordering on purpose, so that a test can show that it would see a
 * missing wait (CKV_PIPE_CHECK_NO_DEFER only changes where selections run:
 * every plain layer of the loop without buffers runs its own selection, as
 * with a smaller workspace, for comparing the two forms).  CKV_PIPE_CHECK_NO_FILL_WAIT: the compute stream does not
 * wait for a buffer's fill before attending over it (read-after-write);
 * CKV_PIPE_CHECK_NO_RELEASE_WAIT: the copy stream does not wait for a
 * buffer's release before refilling it (write-after-read);
 * CKV_PIPE_CHECK_POISON: the copy stream overwrites a released buffer with
 * NaN bits before refilling it.  Every access stays inside the buffers; a
 * missing wait only makes an attention read rows of another layer or
 * poison.  0 (the default) restores the normal loop; unknown bits are
 * CKV_EINVAL. */
#define CKV_PIPE_CHECK_NO_FILL_WAIT 1u
#define CKV_PIPE_CHECK_NO_RELEASE_WAIT 2u
#define CKV_PIPE_CHECK_POISON 4u
#define CKV_PIPE_CHECK_NO_DEFER 8u
int ckv_pipeline_set_checks(ckv_pipeline* pipe, unsigned flags);

/* Starts a decode loop: gathers layer 0 (into buffer 0) and layer 1 (into
 * buffer 1) from their idx_prev/n_sel_prev on copy_stream.  Buffers are
 * k_buf[i], v_buf[i], each [B][Hkv][k][d] bf16 on the device. */
int ckv_pipeline_prime(ckv_pipeline* pipe, const ckv_shape* shape, int32_t k,
                       const ckv_layer* layers, int num_layers, int src_kind,
                       uint16_t* const k_buf[2], uint16_t* const v_buf[2],
                       void* copy_stream);

/* One decode step.  With k_buf and v_buf both NULL (a cache resident in
 * device memory), each of num_layers >= 1 layers runs ckv_critical_kv_attn in
 * place on compute_stream: attention of q_att over rows idx_prev/n_sel_prev
 * of the layer's k_src/v_src, selection from q_sel into idx_next; nothing
 * runs on copy_stream (it may be NULL), no prime is needed, and a layer with
 * idx_true set is CKV_EINVAL.  Otherwise the two-buffer loop below.
 *
 * The two-buffer loop, over num_layers >= 2 layers.  For each layer l, on
 * compute_stream: ckv_critical_kv_attn in pipelined mode (attention of q_att
 * over the buffer holding idx_prev's rows, selection from q_sel into
 * idx_next), or, for a layer with idx_true set, ckv_corrected_attn (misses
 * of idx_prev against q_att's own selection fetched into the buffer first,
 * src_kind and the layer's k_src/v_src), ckv_corrected_attn_lowrank if its
 * lr_rank is also > 0; on copy_stream: the refill of the
 * released buffer with layer l+2, or, for the last two layers, with the next
 * step's layers 0 and 1 from this step's idx_next.  Before the next step the
 * caller swaps idx_prev and idx_next.  ws is the workspace of
 * CKV_ENTRY_CRITICAL_KV_ATTN, or of CKV_ENTRY_CORRECTED_ATTN if any layer
 * has idx_true set, or of CKV_ENTRY_DECODE_STEP (which serves every layer
 * kind) if any layer is chunked or has two tokens; it is used on the compute
 * stream only.  Without buffers and with the workspace of
 * CKV_ENTRY_DECODE_STEP, a plain layer followed by a plain layer, or a
 * two-token layer followed by a two-token layer, leaves its selection
 * (idx_next, n_sel_next: not read before the next step) to the next layer's
 * launch, which runs it beside that layer's attention and scoring; a plain
 * layer's own attention partials are then merged by a merge launch.  A
 * pending selection runs before the call returns and before a layer of
 * another kind.  Results are the same either way.  A chunked or two-token layer runs the same pipelined step
 * (one launch attends over the previous set and scores for the next one) with
 * its selection over chunk landmarks or its second token; such a layer with
 * idx_true set is CKV_EINVAL.
 *
 * Steps can be captured into a HIP graph on compute_stream (whole steps: the
 * copy stream joins the capture at its first wait and the caller joins it
 * back before the capture ends).  A fill recorded outside the capture (by
 * the prime or an eager step) is not waited for inside it, so the caller
 * orders each launch of the graph after the copy stream's earlier work
 * (e.g. compute_stream waits for copy_stream before the first launch).  A
 * captured two-buffer step must have an even number of layers, so that the
 * graph leaves the buffers as it found them for its next launch; an odd
 * number under capture is CKV_EINVAL. */
int ckv_decode_step(ckv_pipeline* pipe, const ckv_shape* shape, int num_layers,
                    const ckv_layer* layers, const int32_t* ctx_lens, int32_t k,
                    float scale, int src_kind, uint16_t* const k_buf[2],
                    uint16_t* const v_buf[2], void* ws, size_t ws_bytes,
                    void* compute_stream, void* copy_stream);

/* ---- kernel timing -------------------------------------------------------
 * For benchmarks and profiling, not for serving: between ckv_profile_begin()
 * and ckv_profile_end(), every kernel the library launches carries a pair of
 * HIP events stamped by the dispatch itself (start and end of that kernel on
 * the caller's stream), so timing adds no packets to the stream.  The state
 * is process-wide and guarded by a lock; calls on several threads are
 * accumulated together. */
typedef enum ckv_kernel_id {
  CKV_K_ZERO = 0,     /* workspace clear                                    */
  CKV_K_SCORE = 1,    /* scoring pass (with first-digit histogram if fused) */
  CKV_K_HIST = 2,     /* first-digit histogram of given scores              */
  CKV_K_FILTER = 3,   /* selection: above-bin positions and candidates      */
  CKV_K_FINISH = 4,   /* selection: exact threshold, ordered output         */
  CKV_K_ATTN = 5,     /* attention partials over selected rows              */
  CKV_K_COMBINE = 6,  /* merge of attention partials                        */
  CKV_K_DUAL = 7,     /* one launch: attention (buffer) + scoring           */
  CKV_K_GATHER = 8,   /* sparse K/V assembly                                */
  CKV_K_MISS = 9,     /* predicted vs selected set: hits, misses, slots     */
  CKV_K_LANDMARKS = 10, /* chunk landmarks (mean keys)                      */
  CKV_K_EXPAND = 11,  /* selected chunks -> their rows                      */
  CKV_K_RECONSTRUCT = 12, /* low-rank key rebuild (with the misses' V fetch)  */
  CKV_K_SELECT_ATTN = 13, /* same-step selection and attention in one launch */
  CKV_K_PROBE = 14,   /* read-rate probe (ckv_probe_read_rows)              */
  CKV_K_CRITICAL = 15, /* same-step scoring, selection and attention in one launch */
  CKV_K_COUNT = 16
} ckv_kernel_id;

#define CKV_K_ALL ((1u << CKV_K_COUNT) - 1u)

typedef struct ckv_kernel_stats {
  int64_t launches;   /* dispatches of this kernel class                    */
  double total_ms;    /* sum of their durations                             */
  double max_ms;      /* longest single dispatch                            */
} ckv_kernel_stats;

/* Static name of a kernel class ("" for an unknown id). */
const char* ckv_kernel_name(int id);

/* Start recording the kernel classes whose bit (1 << ckv_kernel_id) is set
 * in kernel_mask; other kernels launch unstamped.  Drops anything recorded
 * before. */
int ckv_profile_begin(uint32_t kernel_mask);

/* ckv_profile_begin, stamping only launches 0, every, 2*every, ... of each
 * recorded class (every >= 1, else CKV_EINVAL).  A stamped dispatch costs a
 * few microseconds of stream time more than a plain one, so a timed loop
 * that also measures one kernel's duration stamps a sample of its launches. */
int ckv_profile_begin_sampled(uint32_t kernel_mask, uint32_t every);

/* Stop recording, wait for the recorded kernels to finish and write one
 * entry per ckv_kernel_id into stats[0 .. CKV_K_COUNT). */
int ckv_profile_end(ckv_kernel_stats* stats);

/* ---- debug mode -----------------------------------------------------------
 * For development, not for serving (on: nonzero; process-wide; off by default,
 * on by default in a library built with -DCKV_DEBUG).  In debug mode every
 * entry first checks its device-side inputs on the device and synchronises
 * the caller's stream, returning CKV_EINVAL with the first violation in
 * ckv_last_error_detail():
 *   0 <= ctx_lens[b] <= max_ctx;
 *   0 <= n_sel[u] <= k for an input count (n_sel, n_sel_in, n_pred);
 *   entries 0 .. n_sel[u] - 1 of an input index set (idx, idx_in, idx_pred;
 *   all k without a count) are -1 or positions below the unit's context
 *   length (below max_ctx where the entry takes no ctx_lens).
 * Outside debug mode these are the caller's preconditions, and kernels only
 * clamp what they read.  Every kernel launch then also synchronises its
 * stream, so that a failing kernel is reported by the entry that launched it
 * (CKV_EHIP).  Debug mode synchronises, so it is not for graph capture. */
int ckv_set_debug(int on);

/* ---- the same-step layer in one launch ---------------------------------------
 * Where it applies, a same-step call of ckv_critical_kv_attn (or of
 * ckv_critical_kv_attn_noalloc) scores, selects and attends in one launch:
 * the group size is 2, 4 or 8, the batch has a multiple of 8 units with two
 * workgroups per unit fitting on the device, 512 <= k <= 2048, max_ctx <=
 * 65536, and the per-workgroup histogram slots apply (at least about 40
 * units).  Each unit's selection
 * and attention then start as soon as that unit's scores are complete (Sec. 2.2
 * selection inside the step, with the attention of Sec. 5.3-5.4), not after
 * the whole scoring pass.  The launch hands each unit's scores over through
 * flags in the workspace, which are zero again when it ends.  Each of a
 * unit's two workgroups selects the unit's set; by default each then attends
 * over half of the set's rows with all of the group's heads, and the second
 * merges the first's partial (handed over through a per-unit flag) into the
 * output.  Otherwise, or with this setting off, the call runs the scoring
 * launch, then the selection and attention launch, whose two workgroups per
 * unit attend and merge the same way.
 *   on = CKV_ONE_LAUNCH_OFF: two launches; the same bits as one launch.
 *   on = CKV_ONE_LAUNCH_HEAD_HALVES: one launch (or, where it does not
 *        apply, two) whose two workgroups per unit attend over the whole set
 *        with half of the heads each.  The index sets and counts are those
 *        of the other forms bit for bit; the outputs add the same terms in
 *        another order (fp32 rounding only).
 *   any other value: one launch with row halves (the default).
 * The setting is process-wide and for comparing the forms; calls already
 * launched keep their form. */
enum { CKV_ONE_LAUNCH_OFF = 0, CKV_ONE_LAUNCH_ROW_HALVES = 1, CKV_ONE_LAUNCH_HEAD_HALVES = 2 };
int ckv_set_one_launch_same_step(int on);

/* ---- read-rate probe -------------------------------------------------------
 * For measurement, not for serving: reads the K and V rows that idx selects
 * with the access pattern of one of the attention launches and no
 * arithmetic, so that its duration is what the memory system gives that
 * pattern (the attention's floor).  Per unit (request b, KV head h) it reads
 * rows idx[b][h][0 .. k) of k_rows and v_rows (the layout of
 * ckv_sparse_decode_attn's in-place sources: unit rows at stride
 * shape->kv_row_stride elements, max_ctx rows per unit; entries outside
 * [0, max_ctx), such as -1 padding, read row 0 or max_ctx - 1), 16 bytes per
 * lane, 4 rows per load, in blocks of 16 rows with the next block in flight:
 *   CKV_PROBE_STANDALONE: the standalone attention's grid, one 256-thread
 *     workgroup per 256 selected rows, indices read from idx;
 *   CKV_PROBE_ROW_HALVES: two 1024-thread workgroups per unit (each holding
 *     the fused same-step launch's LDS, so one per CU), each over half the
 *     set, positions staged in LDS; a unit's two go to one XCD;
 *   CKV_PROBE_HEAD_HALVES: the same, both over the whole set (the fused
 *     launch's head halves: the second read of each row from the L2).
 * k: 1 .. 2^20 for the standalone grid, 1 .. 2048 for the halves
 * (CKV_ESHAPE beyond).  sink: device, at least ckv_probe_sink_words() 32-bit
 * words; one checksum per thread is written there so that no load is
 * dropped.  Pointers 16-byte aligned.  Launched as kernel class CKV_K_PROBE. */
#define CKV_PROBE_STANDALONE 0
#define CKV_PROBE_ROW_HALVES 1
#define CKV_PROBE_HEAD_HALVES 2
int ckv_probe_read_rows(const ckv_shape* shape, const uint16_t* k_rows,
                        const uint16_t* v_rows, const int32_t* idx, int32_t k, int mode,
                        uint32_t* sink, size_t sink_words, void* stream);

/* Words of sink that ckv_probe_read_rows needs for this shape, k and mode
 * (0 for an invalid shape, k or mode). */
size_t ckv_probe_sink_words(const ckv_shape* shape, int32_t k, int mode);

#ifdef __cplusplus
}
#endif
#endif /* CKV_H */
