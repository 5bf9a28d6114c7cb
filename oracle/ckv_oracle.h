/*
 * ckv_oracle.h -- plain CPU oracle for critical-KV selection and sparse
 * decode attention (DualDecoder, arXiv 2607.26475).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link
 * or call this code: only the tests, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or helper
 * with the HIP library; the two meet only through the seeded input
 * generators, which hold none of the method's arithmetic.
 *
 * Everything is computed in fp64 from bf16 bit patterns decoded exactly.
 * The arithmetic follows the paper's statement of the decode step:
 *   - Sec. 2.2 / Sec. 4.1: the retrieval index of a decoding step is computed
 *     from a query and GPU-resident key summaries ("landmarks"); here the
 *     landmark of a position is its own key (chunk size 1).
 *   - Sec. 4.1 (retrieval index prediction): the index used at step i+1 is
 *     computed at step i from the speculative token's query.
 *   - Sec. 5.3 / Sec. 5.4: attention must equal the result computed over the
 *     KV entries of the selected index, assembled in the attention layout.
 * Readings where the paper is silent (GQA aggregation = max over the group's
 * heads, tie-break on lower position, ascending output order, -1 padding,
 * fp32 scale widened to fp64) are listed in the design notes of the repo.
 *
 * Parity pinning: the paper prints no worked example, closed-form output or
 * kernel value.  Each function is pinned by closed forms, brute force on tiny
 * inputs, special cases reducing to library routines and invariants (the CPU
 * test suite), not by any value printed in the paper.
 */
#ifndef CKV_ORACLE_H
#define CKV_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same meaning as the library's shape descriptor; declared separately on
 * purpose (the oracle shares no header with the product). */
typedef struct ckvref_shape {
  int32_t batch;          /* B                                            */
  int32_t num_q_heads;    /* Hq                                           */
  int32_t num_kv_heads;   /* Hkv; query head q belongs to KV head q/(Hq/Hkv) */
  int32_t head_dim;       /* d                                            */
  int32_t max_ctx;        /* rows stored per (request, KV head)           */
  int32_t reserved;
  int64_t key_row_stride; /* elements between rows of the scoring keys    */
  int64_t kv_row_stride;  /* elements between rows of the K/V source      */
} ckvref_shape;

/* Exact decode of a bf16 bit pattern. */
double ckvref_bf16_to_f64(uint16_t bits);

/* ---- single (request, KV head) unit ------------------------------------ */

/* S[j] = max over g < G of scale * sum_c q[g*d + c] * keys[j*stride + c],
 * j < n.  q holds the G query heads of the group, row-major [G][d]. */
void ckvref_unit_scores(int G, int d, int n, const uint16_t* q,
                        const uint16_t* keys, int64_t key_row_stride,
                        float scale, double* S);

/* Top-m of S[0..n) by (S descending, position ascending), m = min(k, n);
 * idx[0..m) in ascending position order, idx[m..k) = -1.  Returns m. */
int ckvref_unit_select(int n, const double* S, int k, int32_t* idx);

/* out[g*d + c] = sum_i p_gi * v_rows[i*d + c] with p_g = softmax over i < m of
 * scale * q[g] . k_rows[i]; out = 0 when m == 0.  k_rows/v_rows are dense
 * [m][d] (already gathered).  If p != NULL it receives p[g*m + i]. */
void ckvref_unit_attn(int G, int d, int m, const uint16_t* q,
                      const uint16_t* k_rows, const uint16_t* v_rows,
                      float scale, double* out, double* p);

/* ---- whole-batch functions, one per library entry point --------------- */
/* All buffers are host memory with the library's dense layouts:
 *   q         [B][Hq][d] bf16            ctx_lens  [B] int32
 *   keys      row (b,h,j) at ((b*Hkv+h)*max_ctx + j) * row_stride
 *   scores    [B][Hkv][max_ctx] (fp64 here; -inf for j >= n_b)
 *   idx       [B][Hkv][k] int32          n_sel     [B][Hkv] int32
 *   k/v buf   [B][Hkv][k][d] bf16        out       [B][Hq][d] (fp64 here)
 * nthreads > 1 splits the independent (request, KV head) units over
 * pthreads; the arithmetic per unit is unchanged.  Return 0 on success,
 * -1 on a malformed shape. */
int ckvref_score_keys(const ckvref_shape* s, const uint16_t* q,
                      const uint16_t* k_score, const int32_t* ctx_lens,
                      float scale, double* scores, int nthreads);

int ckvref_select_topk(const ckvref_shape* s, const double* scores,
                       const int32_t* ctx_lens, int k, int32_t* idx,
                       int32_t* n_sel, int nthreads);

int ckvref_gather_kv(const ckvref_shape* s, const uint16_t* k_src,
                     const uint16_t* v_src, const int32_t* idx,
                     const int32_t* n_sel, int k, uint16_t* k_dst,
                     uint16_t* v_dst);

int ckvref_sparse_decode_attn(const ckvref_shape* s, const uint16_t* q_att,
                              const uint16_t* k_buf, const uint16_t* v_buf,
                              const int32_t* n_sel, int k, float scale,
                              double* out, int nthreads);

/* Selection from q_sel (the speculative token's query; NULL => q_att), then
 * attention of q_att over the selected rows of k_src/v_src. */
int ckvref_critical_kv_attn(const ckvref_shape* s, const uint16_t* q_att,
                            const uint16_t* q_sel, const uint16_t* k_score,
                            const uint16_t* k_src, const uint16_t* v_src,
                            const int32_t* ctx_lens, int k, float scale,
                            int32_t* idx, int32_t* n_sel, double* out,
                            int nthreads);

/* ---- chunk landmarks ---------------------------------------------------
 * Sec. 2.2 (adjacent KV entries segmented into chunks, one compressed
 * landmark per chunk, chunks selected by the query) and Sec. 4.1 (the
 * landmarks are fixed before decoding).  The landmark of a chunk is the mean
 * of its keys, rounded once to bf16. */

/* Nearest bf16 to x, ties to the even significand; the bit pattern. */
uint16_t ckvref_f64_to_bf16(double x);

/* For every (b, h) and chunk c < ceil(n_b / chunk): landmark row c =
 * bf16(mean of key rows [c*chunk, min(c*chunk + chunk, n_b))), the mean
 * summed in fp64 in row order and divided by the row count.  Chunks at or
 * past ceil(n_b / chunk) are not written.  keys use s->key_row_stride;
 * landmarks are dense [B][Hkv][ceil(max_ctx / chunk)][d]. */
int ckvref_chunk_landmarks(const ckvref_shape* s, int chunk, const uint16_t* keys,
                           const int32_t* ctx_lens, uint16_t* landmarks);

/* The rows of m selected chunks (ascending chunk indices): rows[i] =
 * chunk_idx[i / chunk] * chunk + i % chunk for the rows below n, in that
 * order; -1 after, up to k.  Returns the row count. */
int ckvref_expand_chunks(int chunk, int m, const int32_t* chunk_idx, int n, int k,
                         int32_t* rows);

/* Chunk selection: every landmark scored against q_sel (ckvref_score_keys on
 * the landmarks, ceil(n_b / chunk) chunks per unit), the k / chunk best
 * chunks selected (ckvref_select_topk) and expanded to rows.  chunk_idx
 * [B][Hkv][k/chunk], n_chunks [B][Hkv], rows [B][Hkv][k], n_rows [B][Hkv].
 * k must be a multiple of chunk. */
int ckvref_select_chunks(const ckvref_shape* s, int chunk, const uint16_t* q_sel,
                         const uint16_t* landmarks, const int32_t* ctx_lens, int k,
                         float scale, int32_t* chunk_idx, int32_t* n_chunks,
                         int32_t* rows, int32_t* n_rows, int nthreads);

/* ---- dual-token attention ----------------------------------------------
 * Sec. 5.2 (dual-token decoding): the current token T_i and the speculative
 * token T'_{i+1} of a request run as two consecutive positions of one
 * sequence, causally masked: T_i never sees T'_{i+1}.  Over the sparse set
 * both tokens attend to the same selected rows; the tokens' own new rows
 * (k_local/v_local [B][Hkv][2][d]: row 0 = T_i, row 1 = T'_{i+1}) follow
 * them.  Per unit with m = n_sel (clamped to [0, k]):
 *   out_cur[b][g]  = attention of q_cur[b][g]  over buffer rows [0, m) + local row 0
 *   out_spec[b][g] = attention of q_spec[b][g] over buffer rows [0, m) + local rows 0, 1 */
int ckvref_dual_token_attn(const ckvref_shape* s, const uint16_t* q_cur,
                           const uint16_t* q_spec, const uint16_t* k_buf,
                           const uint16_t* v_buf, const int32_t* n_sel,
                           const uint16_t* k_local, const uint16_t* v_local, int k,
                           float scale, double* out_cur, double* out_spec, int nthreads);

/* ---- low-rank key reconstruction --------------------------------------
 * Sec. 5.3 (adaptive key reconstruction, after ShadowKV): for layers whose
 * prediction misses often, selected keys are rebuilt on the GPU from a
 * low-rank key cache instead of being fetched; values are still fetched.
 * The cache of a unit is K ~ U . W with U [max_ctx][rank] and W [rank][d]
 * (bf16).  For i < n_sel (clamped to [0, k]):
 *   k_dst[b][h][i][c] = bf16(sum over j < rank, ascending, of
 *                            U[idx_i][j] * W[j][c])   (fp64 sum, rounded once)
 * Slots i >= n_sel are not written. */
int ckvref_reconstruct_keys(const ckvref_shape* s, int rank, const uint16_t* u_fac,
                            const uint16_t* w_fac, const int32_t* idx, const int32_t* n_sel,
                            int k, uint16_t* k_dst);

#ifdef __cplusplus
}
#endif
#endif /* CKV_ORACLE_H */
