// abi_checks.cpp -- host-side checks of libckv's C ABI, built with the host
// code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU needed).
//
// Every entry point is called with rejected arguments (NULL, misaligned,
// bad shapes, budgets, strides, kinds, workspaces) and with a batch of 0,
// which runs the whole validation and workspace layout of the call and then
// returns before any launch.  Workspace sizes are computed over a grid of
// shapes up to the header's limits.  Exit status 0 iff every status matches.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "ckv.h"

namespace {

int g_failures = 0;
uint16_t* const F16 = reinterpret_cast<uint16_t*>(0x100000);  // never dereferenced
int32_t* const FI = reinterpret_cast<int32_t*>(0x100000);
float* const FF = reinterpret_cast<float*>(0x100000);
void* const FW = reinterpret_cast<void*>(0x100000);

void expect(int got, int want, const char* what, int line) {
  if (got != want) {
    std::fprintf(stderr, "line %d: %s: status %d, expected %d (%s)\n", line, what, got, want,
                 ckv_last_error_detail());
    ++g_failures;
  }
  if (want != CKV_OK && std::strlen(ckv_last_error_detail()) == 0) {
    std::fprintf(stderr, "line %d: %s: no error detail\n", line, what);
    ++g_failures;
  }
}
#define EXPECT(call, want) expect((call), (want), #call, __LINE__)

ckv_shape shape(int B, int Hq, int Hkv, int n, int64_t ks = 128, int64_t vs = 128) {
  ckv_shape s;
  std::memset(&s, 0, sizeof s);
  s.batch = B;
  s.num_q_heads = Hq;
  s.num_kv_heads = Hkv;
  s.head_dim = 128;
  s.max_ctx = n;
  s.key_row_stride = ks;
  s.kv_row_stride = vs;
  return s;
}

size_t ws_of(const ckv_shape& s, int k, int entry) {
  size_t b = 0;
  EXPECT(ckv_workspace_bytes(&s, k, entry, &b), CKV_OK);
  return b;
}

}  // namespace

int main() {
  // status text
  for (int st = 0; st <= 6; ++st)
    if (!ckv_status_str(st) || !*ckv_status_str(st)) ++g_failures;
  if (ckv_abi_version() != CKV_ABI_VERSION) ++g_failures;

  // workspace sizes over a grid of shapes, each entry, up to large sizes
  const int entries[] = {CKV_ENTRY_SELECT_TOPK, CKV_ENTRY_SPARSE_DECODE_ATTN,
                         CKV_ENTRY_CRITICAL_KV_ATTN, CKV_ENTRY_CORRECTED_ATTN,
                         CKV_ENTRY_DUAL_TOKEN_ATTN};
  const int ctxs[] = {1, 31, 4096, 65536, 65537, 1 << 20, (1 << 20) + 3, 1 << 26};
  const int ks[] = {1, 256, 2048, 8192, 9000, 1 << 20};
  for (int e : entries)
    for (int n : ctxs)
      for (int k : ks)
        for (int G : {1, 4, 16}) {
          const ckv_shape s = shape(2, 8 * G, 8, n);
          size_t b = 0;
          const int rc = ckv_workspace_bytes(&s, k, e, &b);
          if (rc != CKV_OK || b % 256 != 0) {
            std::fprintf(stderr, "workspace e=%d n=%d k=%d G=%d: rc %d bytes %zu\n", e, n, k,
                         G, rc, b);
            ++g_failures;
          }
        }
  {
    const ckv_shape s = shape(2, 8, 2, 64);
    size_t b = 0;
    EXPECT(ckv_workspace_bytes(&s, 16, 42, &b), CKV_EINVAL);
    EXPECT(ckv_workspace_bytes(&s, 16, CKV_ENTRY_SELECT_TOPK, nullptr), CKV_EINVAL);
    EXPECT(ckv_workspace_bytes(&s, 0, CKV_ENTRY_SELECT_TOPK, &b), CKV_ESHAPE);
    EXPECT(ckv_workspace_bytes(&s, (1 << 20) + 1, CKV_ENTRY_SELECT_TOPK, &b), CKV_ESHAPE);
    EXPECT(ckv_workspace_bytes(nullptr, 16, CKV_ENTRY_SELECT_TOPK, &b), CKV_EINVAL);
  }

  // shape validation
  {
    ckv_shape s = shape(2, 6, 4, 64);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_ESHAPE);
    s = shape(2, 8, 2, 64);
    s.head_dim = 64;
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_EUNSUPPORTED);
    s = shape(2, 6, 2, 64);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_EUNSUPPORTED);
    s = shape(2, 64, 2, 64);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_EUNSUPPORTED);
    s = shape(2, 8, 2, 0);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_ESHAPE);
    s = shape(2, 8, 2, (1 << 30) + 1);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_ESHAPE);
    s = shape(2, 8, 2, 64, 100);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_ESHAPE);
    s = shape(2, 8, 2, 64, 128, 132);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_ESHAPE);
    s = shape(-1, 8, 2, 64);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_ESHAPE);
    s = shape(1 << 24, 8, 8, 64);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_EUNSUPPORTED);
    s = shape(2, 8, 2, 64);
    s.reserved = 3;
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_EINVAL);
    s = shape(2, 8, 2, 64);
    EXPECT(ckv_score_keys(&s, nullptr, F16, FI, 0.1f, FF, nullptr), CKV_EINVAL);
    EXPECT(ckv_score_keys(&s, F16 + 2, F16, FI, 0.1f, FF, nullptr), CKV_EINVAL);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.f, FF, nullptr), CKV_EINVAL);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, -2.f, FF, nullptr), CKV_EINVAL);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, __builtin_nanf(""), FF, nullptr), CKV_EINVAL);
    EXPECT(ckv_score_keys(&s, F16, F16, FI, __builtin_inff(), FF, nullptr), CKV_EINVAL);
  }

  // batch 0: full validation and layout, no launch
  for (int n : {64, 70000, 1 << 21})
    for (int k : {16, 2048, 9000}) {
      const ckv_shape s = shape(0, 32, 8, n, 256, 256);
      const size_t wsel = ws_of(s, k, CKV_ENTRY_SELECT_TOPK);
      const size_t wat = ws_of(s, k, CKV_ENTRY_SPARSE_DECODE_ATTN);
      const size_t wcr = ws_of(s, k, CKV_ENTRY_CRITICAL_KV_ATTN);
      const size_t wco = ws_of(s, k, CKV_ENTRY_CORRECTED_ATTN);
      const size_t wdt = ws_of(s, k, CKV_ENTRY_DUAL_TOKEN_ATTN);
      EXPECT(ckv_score_keys(&s, F16, F16, FI, 0.1f, FF, nullptr), CKV_OK);
      EXPECT(ckv_select_topk(&s, FF, FI, k, FI, FI, FW, wsel, nullptr), CKV_OK);
      EXPECT(ckv_gather_kv(&s, F16, F16 + 128, CKV_SRC_DEVICE, FI, FI, k, F16, F16, nullptr),
             CKV_OK);
      EXPECT(ckv_sparse_decode_attn(&s, F16, F16, F16, FI, k, 0.1f, FF, FW, wat, nullptr),
             CKV_OK);
      EXPECT(ckv_critical_kv_attn(&s, F16, nullptr, F16, FI, k, 0.1f, F16, F16, CKV_SRC_DEVICE,
                                  nullptr, nullptr, nullptr, nullptr, FI, FI, FF, FW, wcr,
                                  nullptr),
             CKV_OK);
      EXPECT(ckv_critical_kv_attn(&s, F16, F16, F16, FI, k, 0.1f, F16, F16, CKV_SRC_DEVICE, FI,
                                  nullptr, nullptr, FI, FI, FI, FF, FW, wcr, nullptr),
             CKV_OK);
      EXPECT(ckv_critical_kv_attn(&s, F16, F16, F16, FI, k, 0.1f, nullptr, nullptr, 0, nullptr,
                                  F16, F16, FI, FI, FI, FF, FW, wcr, nullptr),
             CKV_OK);
      EXPECT(ckv_corrected_attn(&s, F16, nullptr, F16, FI, k, 0.1f, F16, F16, CKV_SRC_DEVICE,
                                FI, FI, F16, F16, FI, FI, FI, FI, FI, FF, FW, wco, nullptr),
             CKV_OK);
      EXPECT(ckv_corrected_attn_lowrank(&s, F16, nullptr, F16, FI, k, 0.1f, nullptr, F16,
                                        CKV_SRC_DEVICE, 32, F16, F16, FI, FI, F16, F16, FI,
                                        FI, FI, FI, FI, FF, FW, wco, nullptr),
             CKV_OK);
      EXPECT(ckv_dual_token_attn(&s, F16, F16, F16, F16, FI, F16, F16, k, 0.1f, FF, FF, FW,
                                 wdt, nullptr),
             CKV_OK);
      EXPECT(ckv_reconstruct_keys(&s, 32, F16, F16, FI, FI, k, F16, nullptr), CKV_OK);
      EXPECT(ckv_chunk_landmarks(&s, 8, F16, FI, F16, nullptr), CKV_OK);
      if (k % 8 == 0) {
        EXPECT(ckv_select_chunks(&s, 8, F16, F16, FI, k, 0.1f, FI, FI, FI, FI, FW, wcr,
                                 nullptr),
               CKV_OK);
        EXPECT(ckv_chunked_kv_attn(&s, 8, F16, nullptr, F16, FI, k, 0.1f, F16, F16,
                                   CKV_SRC_DEVICE, FI, FI, FI, FI, FF, FW, wcr, nullptr),
               CKV_OK);
      }
    }

  // one byte short of each workspace (a non-empty batch: the check comes
  // before anything is launched)
  for (int n : {64, 70000, 1 << 21})
    for (int k : {16, 2048, 9000}) {
      const ckv_shape s = shape(3, 32, 8, n, 256, 256);
      const size_t wsel = ws_of(s, k, CKV_ENTRY_SELECT_TOPK);
      const size_t wat = ws_of(s, k, CKV_ENTRY_SPARSE_DECODE_ATTN);
      const size_t wcr = ws_of(s, k, CKV_ENTRY_CRITICAL_KV_ATTN);
      const size_t wco = ws_of(s, k, CKV_ENTRY_CORRECTED_ATTN);
      const size_t wdt = ws_of(s, k, CKV_ENTRY_DUAL_TOKEN_ATTN);
      EXPECT(ckv_select_topk(&s, FF, FI, k, FI, FI, FW, wsel - 1, nullptr), CKV_EWORKSPACE);
      EXPECT(ckv_critical_kv_attn(&s, F16, nullptr, F16, FI, k, 0.1f, F16, F16, CKV_SRC_DEVICE,
                                  nullptr, nullptr, nullptr, nullptr, FI, FI, FF, FW, wcr - 1,
                                  nullptr),
             CKV_EWORKSPACE);
      EXPECT(ckv_corrected_attn(&s, F16, nullptr, F16, FI, k, 0.1f, F16, F16, CKV_SRC_DEVICE,
                                FI, FI, F16, F16, FI, FI, FI, FI, FI, FF, FW, wco - 1, nullptr),
             CKV_EWORKSPACE);
      EXPECT(ckv_dual_token_attn(&s, F16, F16, F16, F16, FI, F16, F16, k, 0.1f, FF, FF, FW,
                                 wdt - 1, nullptr),
             CKV_EWORKSPACE);
      EXPECT(ckv_sparse_decode_attn(&s, F16, F16, F16, FI, k, 0.1f, FF, FW, wat - 1, nullptr),
             CKV_EWORKSPACE);
      EXPECT(ckv_select_topk(&s, FF, FI, k, FI, FI, nullptr, wsel, nullptr), CKV_EWORKSPACE);
      EXPECT(ckv_critical_kv_attn(&s, F16, nullptr, F16, FI, k, 0.1f, F16, F16, CKV_SRC_DEVICE,
                                  nullptr, nullptr, nullptr, nullptr, FI, FI, FF,
                                  static_cast<char*>(FW) + 16, wcr, nullptr),
             CKV_EWORKSPACE);  // not 256-byte aligned
    }

  // the read-rate probe: sizes, refusals, and an empty batch (no launch)
  {
    uint32_t* const FU = reinterpret_cast<uint32_t*>(0x100000);
    const ckv_shape s = shape(16, 32, 8, 32768);
    if (ckv_probe_sink_words(&s, 2048, CKV_PROBE_STANDALONE) != (size_t)128 * 8 * 256) ++g_failures;
    if (ckv_probe_sink_words(&s, 2048, CKV_PROBE_HEAD_HALVES) != (size_t)256 * 1024) ++g_failures;
    if (ckv_probe_sink_words(&s, 4096, CKV_PROBE_ROW_HALVES) != 0) ++g_failures;
    if (ckv_probe_sink_words(&s, 16, 3) != 0) ++g_failures;
    EXPECT(ckv_probe_read_rows(&s, F16, F16, FI, 16, 3, FU, 1 << 20, nullptr), CKV_EINVAL);
    EXPECT(ckv_probe_read_rows(&s, F16, F16, FI, 4096, CKV_PROBE_HEAD_HALVES, FU, 1 << 20,
                               nullptr),
           CKV_ESHAPE);
    EXPECT(ckv_probe_read_rows(&s, F16, F16, FI, 2048, CKV_PROBE_STANDALONE, FU, 1000, nullptr),
           CKV_EINVAL);  // sink too small
    EXPECT(ckv_probe_read_rows(&s, nullptr, F16, FI, 16, CKV_PROBE_STANDALONE, FU, 1 << 20,
                               nullptr),
           CKV_EINVAL);
    const ckv_shape e = shape(0, 32, 8, 32768);
    for (int mode : {CKV_PROBE_STANDALONE, CKV_PROBE_ROW_HALVES, CKV_PROBE_HEAD_HALVES})
      EXPECT(ckv_probe_read_rows(&e, F16, F16, FI, 2048, mode, FU, 0, nullptr), CKV_OK);
  }

  // argument errors of the other entries
  {
    const ckv_shape s = shape(2, 8, 2, 64);
    const size_t w = ws_of(s, 16, CKV_ENTRY_CRITICAL_KV_ATTN);
    EXPECT(ckv_gather_kv(&s, F16, F16, 7, FI, FI, 16, F16, F16, nullptr), CKV_EINVAL);
    EXPECT(ckv_gather_kv(&s, F16, F16, CKV_SRC_DEVICE, FI, FI, 0, F16, F16, nullptr),
           CKV_ESHAPE);
    EXPECT(ckv_critical_kv_attn(&s, F16, nullptr, F16, FI, 16, 0.1f, F16, F16, 0, FI, F16, F16,
                                FI, FI, FI, FF, FW, w, nullptr),
           CKV_EINVAL);  // idx_in and k_buf together
    EXPECT(ckv_select_chunks(&s, 8, F16, F16, FI, 18, 0.1f, FI, FI, FI, FI, FW, w, nullptr),
           CKV_ESHAPE);
    EXPECT(ckv_chunk_landmarks(&s, 0, F16, FI, F16, nullptr), CKV_ESHAPE);
    EXPECT(ckv_reconstruct_keys(&s, 0, F16, F16, FI, FI, 16, F16, nullptr), CKV_ESHAPE);
    EXPECT(ckv_reconstruct_keys(&s, CKV_MAX_RANK + 1, F16, F16, FI, FI, 16, F16, nullptr),
           CKV_ESHAPE);
    const ckv_shape s16 = shape(2, 32, 2, 64);
    EXPECT(ckv_dual_token_attn(&s16, F16, F16, F16, F16, FI, F16, F16, 16, 0.1f, FF, FF, FW,
                               1u << 30, nullptr),
           CKV_EUNSUPPORTED);
  }

  // the fixed-scratch entry refuses a shape whose workspace does not fit,
  // before any runtime call
  {
    const ckv_shape s = shape(8, 32, 8, 131072);
    EXPECT(ckv_critical_kv_attn_noalloc(&s, F16, nullptr, F16, FI, 4096, 0.1f, F16, F16,
                                        CKV_SRC_DEVICE, nullptr, nullptr, nullptr, nullptr, FI,
                                        FI, FF, nullptr),
           CKV_EWORKSPACE);
    EXPECT(ckv_critical_kv_attn_noalloc(&s, F16, nullptr, F16, FI, 0, 0.1f, F16, F16,
                                        CKV_SRC_DEVICE, nullptr, nullptr, nullptr, nullptr, FI,
                                        FI, FF, nullptr),
           CKV_ESHAPE);
  }

  // pipeline object: creation needs the device (events); argument checks do not
  {
    const ckv_shape s = shape(2, 8, 2, 64);
    ckv_layer layers[2];
    std::memset(layers, 0, sizeof layers);
    uint16_t* bufs[2] = {F16, F16};
    EXPECT(ckv_pipeline_create(nullptr), CKV_EINVAL);
    EXPECT(ckv_pipeline_destroy(nullptr), CKV_OK);
    EXPECT(ckv_pipeline_set_gather_width(nullptr, 64), CKV_EINVAL);
    EXPECT(ckv_pipeline_prime(nullptr, &s, 16, layers, 2, 0, bufs, bufs, nullptr), CKV_EINVAL);
    EXPECT(ckv_decode_step(nullptr, &s, 2, layers, FI, 16, 0.1f, 0, bufs, bufs, FW, 1 << 20,
                           nullptr, nullptr),
           CKV_EINVAL);
  }

  // timing state without any launch
  {
    ckv_kernel_stats st[CKV_K_COUNT];
    EXPECT(ckv_profile_begin_sampled(CKV_K_ALL, 0), CKV_EINVAL);
    EXPECT(ckv_profile_begin_sampled(CKV_K_ALL, 3), CKV_OK);
    EXPECT(ckv_profile_end(st), CKV_OK);
    for (int i = 0; i < CKV_K_COUNT; ++i)
      if (st[i].launches != 0 || !*ckv_kernel_name(i)) ++g_failures;
    EXPECT(ckv_profile_end(nullptr), CKV_EINVAL);
  }

  if (g_failures) {
    std::fprintf(stderr, "%d failures\n", g_failures);
    return 1;
  }
  std::printf("abi checks ok\n");
  return 0;
}
