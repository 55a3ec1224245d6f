// C ABI of libipdv: argument validation, workspace sizing, error reporting and
// dispatch to the gfx950 kernels.  Declarations and the full contract are in
// include/ipdv.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <unordered_map>
#include <vector>

#include "../../include/ipdv.h"
#include "kernels.h"

// The kernels see their own copies of the public constants (kernels.h does not
// include the C header); these keep the two in step.
static_assert(IPDV_MAX_K == IPDV_MAX_K_DEV, "top-K limit");
static_assert(IPDV_MAX_GATHER == IPDV_MAX_GATHER_DEV, "gather limit");
static_assert(IPDV_NOALLOC_SCRATCH_BYTES == IPDV_NOALLOC_SCRATCH_BYTES_DEV, "scratch size");
static_assert(IPDV_DRIVER_S == IPDV_DRIVER_S_DEV, "driver code");
static_assert(IPDV_SRC_S == IPDV_SRC_S_DEV && IPDV_SRC_T == IPDV_SRC_T_DEV, "source labels");
static_assert(IPDV_TAKE_COVERAGE == IPDV_TAKE_COVERAGE_DEV &&
                  IPDV_TAKE_ENTROPY == IPDV_TAKE_ENTROPY_DEV, "takeover rules");
static_assert(IPDV_HAND_COVERAGE == IPDV_HAND_COVERAGE_DEV &&
                  IPDV_HAND_FIXED_ONE == IPDV_HAND_FIXED_ONE_DEV &&
                  IPDV_HAND_ENTROPY == IPDV_HAND_ENTROPY_DEV, "handback rules");
static_assert(IPDV_SUPPORT_UNION == IPDV_SUPPORT_UNION_DEV &&
                  IPDV_SUPPORT_STUDENT == IPDV_SUPPORT_STUDENT_DEV &&
                  IPDV_SUPPORT_TEACHER == IPDV_SUPPORT_TEACHER_DEV &&
                  IPDV_SUPPORT_INTERSECTION == IPDV_SUPPORT_INTERSECTION_DEV, "supports");
static_assert(IPDV_LOSS_IPD_SPLIT == IPDV_LOSS_IPD_SPLIT_DEV &&
                  IPDV_LOSS_PURE_REVERSE == IPDV_LOSS_PURE_REVERSE_DEV &&
                  IPDV_LOSS_PURE_FORWARD == IPDV_LOSS_PURE_FORWARD_DEV &&
                  IPDV_LOSS_INVERSE_SPLIT == IPDV_LOSS_INVERSE_SPLIT_DEV, "loss modes");

namespace {

thread_local char g_err[512] = "";
thread_local void* const* g_trace = nullptr;
thread_local int g_trace_cap = 0;
thread_local int g_trace_n = 0;

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_err[0] = '\0';
  return IPDV_OK;
}

int hip_fail(const char* what, hipError_t e) {
  return fail(IPDV_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

}  // namespace

namespace ipdv {

void trace_begin(hipStream_t st) { trace_mark(st); }

void trace_mark(hipStream_t st) {
  if (g_trace && g_trace_n < g_trace_cap) {
    // A bad handle must not turn into a launch failure: clear its error.
    if (hipEventRecord(reinterpret_cast<hipEvent_t>(g_trace[g_trace_n]), st) != hipSuccess)
      (void)hipGetLastError();
    ++g_trace_n;
  }
}

}  // namespace ipdv

extern "C" {

int ipdv_trace_events(void* const* events, int capacity) {
  g_trace = (events && capacity > 0) ? events : nullptr;
  g_trace_cap = g_trace ? capacity : 0;
  g_trace_n = 0;
  return IPDV_OK;
}

int ipdv_trace_count(void) { return g_trace_n; }

const char* ipdv_last_error(void) { return g_err; }

const char* ipdv_version(void) { return "ipdv 0.1 gfx950"; }

static int attn_shape_check(int n_seq, int Hq, int Hkv, int D, int max_q, int max_pages,
                            int page_size) {
  if (n_seq < 0) return fail(IPDV_EINVAL, "n_seq must be >= 0 (got %d)", n_seq);
  if (Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0)
    return fail(IPDV_EINVAL, "Hq (%d) must be a positive multiple of Hkv (%d)", Hq, Hkv);
  if (max_q < 1) return fail(IPDV_EINVAL, "max_q must be >= 1 (got %d)", max_q);
  if (max_pages < 1) return fail(IPDV_EINVAL, "max_pages_per_seq must be >= 1 (got %d)", max_pages);
  if (D != 64 && D != 128) return fail(IPDV_EUNSUPPORTED, "head dim D=%d not in {64, 128}", D);
  if (!is_pow2(page_size) || page_size < 16 || page_size > 64)
    return fail(IPDV_EUNSUPPORTED, "page_size=%d not in {16, 32, 64}", page_size);
  if ((long)n_seq * Hkv > 65535) return fail(IPDV_EUNSUPPORTED, "n_seq * Hkv exceeds 65535");
  if ((long)max_q * (Hq / Hkv) > 64L * 65535) return fail(IPDV_EUNSUPPORTED, "max_q * Hq/Hkv too large");
  return IPDV_OK;
}

size_t ipdv_attn_workspace_size(int n_seq, int Hq, int Hkv, int D, int max_q,
                                int max_pages_per_seq, int page_size) {
  if (attn_shape_check(n_seq, Hq, Hkv, D, max_q, max_pages_per_seq, page_size) != IPDV_OK) return 0;
  return ipdv::attn_plan(n_seq, Hq, Hkv, D, max_q, max_pages_per_seq, page_size).workspace_bytes;
}

// Argument checks shared by both attention entry points (everything but the
// workspace).  Returns IPDV_OK with *empty set when there is nothing to launch.
static int attn_args_check(const void* q, const void* k_new, const void* v_new, void* k_cache,
                           void* v_cache, const int32_t* page_table, int max_pages_per_seq,
                           const int32_t* ctx_lens, const int32_t* cu_q, int n_seq, int max_q,
                           void* out, int Hq, int Hkv, int D, int page_size, int num_pages,
                           float scale, int dtype, bool* empty) {
  *empty = false;
  int st = attn_shape_check(n_seq, Hq, Hkv, D, max_q, max_pages_per_seq, page_size);
  if (st != IPDV_OK) return st;
  if (dtype != IPDV_F32 && dtype != IPDV_BF16) return fail(IPDV_EUNSUPPORTED, "dtype %d", dtype);
  if (dtype == IPDV_F32 && D != 64) return fail(IPDV_EUNSUPPORTED, "fp32 attention supports D=64 only");
  if (num_pages < 1) return fail(IPDV_EINVAL, "num_pages must be >= 1 (got %d)", num_pages);
  if (!std::isfinite(scale) || !(scale > 0.f)) return fail(IPDV_EINVAL, "scale must be positive and finite");
  if (n_seq == 0) {
    *empty = true;
    return IPDV_OK;
  }
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !page_table || !ctx_lens || !cu_q || !out)
    return fail(IPDV_EINVAL, "null required pointer");
  return IPDV_OK;
}

int verify_attn_paged(const void* q, const void* k_new, const void* v_new, void* k_cache,
                      void* v_cache, const int32_t* page_table, int max_pages_per_seq,
                      const int32_t* ctx_lens, const int32_t* cu_q, const int32_t* seq_ids,
                      int n_seq, int max_q, void* out, int Hq, int Hkv, int D, int page_size,
                      int num_pages, float scale, int dtype, void* workspace,
                      size_t workspace_bytes, void* hip_stream) {
  bool empty;
  int st = attn_args_check(q, k_new, v_new, k_cache, v_cache, page_table, max_pages_per_seq,
                           ctx_lens, cu_q, n_seq, max_q, out, Hq, Hkv, D, page_size, num_pages,
                           scale, dtype, &empty);
  if (st != IPDV_OK) return st;
  if (empty) return ok();
  const ipdv::AttnPlan pl = ipdv::attn_plan(n_seq, Hq, Hkv, D, max_q, max_pages_per_seq, page_size);
  if (!workspace || workspace_bytes < pl.workspace_bytes)
    return fail(IPDV_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", pl.workspace_bytes,
                workspace ? workspace_bytes : (size_t)0);
  ipdv::AttnLaunch L{q, k_new, v_new, k_cache, v_cache, page_table, max_pages_per_seq,
                     ctx_lens, cu_q, seq_ids, n_seq, out, Hq, Hkv, D, page_size, num_pages,
                     scale, dtype == IPDV_BF16, workspace};
  hipError_t e = ipdv::launch_verify_attn(L, pl, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("verify_attn_paged launch", e);
  return ok();
}

int verify_attn_paged_noalloc(const void* q, const void* k_new, const void* v_new, void* k_cache,
                              void* v_cache, const int32_t* page_table, int max_pages_per_seq,
                              const int32_t* ctx_lens, const int32_t* cu_q, const int32_t* seq_ids,
                              int n_seq, int max_q, void* out, int Hq, int Hkv, int D,
                              int page_size, int num_pages, float scale, int dtype,
                              void* hip_stream) {
  bool empty;
  int st = attn_args_check(q, k_new, v_new, k_cache, v_cache, page_table, max_pages_per_seq,
                           ctx_lens, cu_q, n_seq, max_q, out, Hq, Hkv, D, page_size, num_pages,
                           scale, dtype, &empty);
  if (st != IPDV_OK) return st;
  if (empty) return ok();
  const ipdv::AttnPlan pl = ipdv::attn_plan(n_seq, Hq, Hkv, D, max_q, max_pages_per_seq, page_size);
  if (pl.workspace_bytes > IPDV_NOALLOC_SCRATCH_BYTES)
    return fail(IPDV_EUNSUPPORTED,
                "this call needs %zu bytes of split-KV scratch; the allocation-free entry point "
                "holds %zu (use verify_attn_paged with a workspace)",
                pl.workspace_bytes, (size_t)IPDV_NOALLOC_SCRATCH_BYTES);
  ipdv::AttnLaunch L{q, k_new, v_new, k_cache, v_cache, page_table, max_pages_per_seq,
                     ctx_lens, cu_q, seq_ids, n_seq, out, Hq, Hkv, D, page_size, num_pages,
                     scale, dtype == IPDV_BF16, nullptr};
  hipError_t e = ipdv::launch_verify_attn_noalloc(L, pl, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("verify_attn_paged_noalloc", e);
  return ok();
}

int ipdv_check_page_table(const int32_t* page_table, int B, int max_pages, const int32_t* ctx_lens,
                          const int32_t* cu_q, const int32_t* seq_ids, int n_seq, int max_q,
                          int page_size, int num_pages, int32_t* bad_seq) {
  if (bad_seq) *bad_seq = -1;
  if (!page_table || !ctx_lens || !cu_q) return fail(IPDV_EINVAL, "null required pointer");
  if (B < 0 || n_seq < 0 || max_pages < 1 || page_size < 1 || num_pages < 1)
    return fail(IPDV_EINVAL, "bad sizes (B %d, n_seq %d, max_pages %d, page_size %d, num_pages %d)",
                B, n_seq, max_pages, page_size, num_pages);
  if (!seq_ids && n_seq > B) return fail(IPDV_EINVAL, "n_seq %d exceeds B %d", n_seq, B);
  auto bad = [&](int b, const char* fmt, ...) {
    if (bad_seq) *bad_seq = b;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return IPDV_EINVAL;
  };
  if (B > 0 && cu_q[0] != 0) return bad(0, "cu_q[0] = %d, must be 0", cu_q[0]);
  for (int b = 0; b < B; ++b)
    if (cu_q[b + 1] < cu_q[b]) return bad(b, "cu_q decreases at sequence %d", b);
  // page -> the handled sequence that writes it (window pages), and the
  // handled sequences that see each page
  std::unordered_map<int32_t, int> writer;
  std::vector<char> handled(B, 0);
  for (int i = 0; i < n_seq; ++i) {
    const int b = seq_ids ? seq_ids[i] : i;
    if (b < 0 || b >= B) return bad(-1, "seq_ids[%d] = %d is not in [0, %d)", i, b, B);
    if (handled[b]) return bad(b, "sequence %d is listed twice in seq_ids", b);
    handled[b] = 1;
    const long L = ctx_lens[b], k = (long)cu_q[b + 1] - cu_q[b];
    if (L < 0) return bad(b, "sequence %d: ctx_len %ld < 0", b, L);
    if (k > max_q) return bad(b, "sequence %d: window of %ld rows exceeds max_q %d", b, k, max_q);
    if (L + k > (long)max_pages * page_size)
      return bad(b, "sequence %d: %ld positions do not fit %d pages of %d", b, L + k, max_pages,
                 page_size);
    const long n_pages = (L + k + page_size - 1) / page_size;
    for (long j = 0; j < n_pages; ++j) {
      const int32_t pg = page_table[(size_t)b * max_pages + j];
      if (pg < 0 || pg >= num_pages)
        return bad(b, "sequence %d: page_table[%d][%ld] = %d is not in [0, %d)", b, b, j, pg,
                   num_pages);
    }
    for (long j = L / page_size; k > 0 && j < n_pages; ++j) {
      const int32_t pg = page_table[(size_t)b * max_pages + j];
      auto it = writer.find(pg);
      if (it != writer.end() && it->second != b)
        return bad(b, "page %d is written by the windows of sequences %d and %d", pg, it->second, b);
      writer[pg] = b;
    }
  }
  for (int i = 0; i < n_seq && !writer.empty(); ++i) {
    const int b = seq_ids ? seq_ids[i] : i;
    const long L = ctx_lens[b], k = (long)cu_q[b + 1] - cu_q[b];
    const long n_pages = (L + k + page_size - 1) / page_size;
    for (long j = 0; j < n_pages; ++j) {
      const int32_t pg = page_table[(size_t)b * max_pages + j];
      auto it = writer.find(pg);
      if (it != writer.end() && it->second != b)
        return bad(b, "page %d is written by sequence %d's window and read by sequence %d", pg,
                   it->second, b);
    }
  }
  return ok();
}

static int lm_shape_check(int M, int Hd, int V, int K) {
  if (M < 0) return fail(IPDV_EINVAL, "M must be >= 0 (got %d)", M);
  if (V < 1) return fail(IPDV_EINVAL, "V must be >= 1 (got %d)", V);
  if (K < 1 || K > IPDV_MAX_K || K > V)
    return fail(IPDV_EINVAL, "K=%d must satisfy 1 <= K <= min(%d, V=%d)", K, IPDV_MAX_K, V);
  if (Hd < 64 || Hd % 64 != 0) return fail(IPDV_EUNSUPPORTED, "Hd=%d must be a positive multiple of 64", Hd);
  if (V > 262144) return fail(IPDV_EUNSUPPORTED, "V=%d exceeds 262144", V);
  if (Hd > 4096) return fail(IPDV_EUNSUPPORTED, "Hd=%d exceeds 4096", Hd);
  if (M > 2147483647 / 2) return fail(IPDV_EUNSUPPORTED, "M too large");
  return IPDV_OK;
}

// The `dtype` argument of the calls that read W: IPDV_F32 or IPDV_BF16, with
// IPDV_W_TILED set when W was packed by lmhead_pack_w (bf16 only).
static int w_dtype(int dtype, bool* bf16, bool* tiled) {
  const int base = dtype & ~IPDV_W_TILED;
  *tiled = (dtype & IPDV_W_TILED) != 0;
  if (base != IPDV_F32 && base != IPDV_BF16) return fail(IPDV_EUNSUPPORTED, "dtype %d", dtype);
  if (*tiled && base != IPDV_BF16) return fail(IPDV_EUNSUPPORTED, "tiled W is bf16 only");
  *bf16 = base == IPDV_BF16;
  return IPDV_OK;
}

size_t ipdv_lmhead_workspace_size(int M, int Hd, int V, int K) {
  if (lm_shape_check(M, Hd, V, K) != IPDV_OK) return 0;
  return ipdv::lm_plan(M, Hd, V, K, true).workspace_bytes;
}

size_t ipdv_workspace_size(int which, const int32_t* a, int n) {
  if (!a) {
    fail(IPDV_EINVAL, "host_shape_args is NULL");
    return 0;
  }
  if (which == IPDV_WS_ATTN) {
    if (n != 7) {
      fail(IPDV_EINVAL, "attention workspace query takes 7 shape values (got %d)", n);
      return 0;
    }
    return ipdv_attn_workspace_size(a[0], a[1], a[2], a[3], a[4], a[5], a[6]);
  }
  if (which == IPDV_WS_LMHEAD) {
    if (n != 4) {
      fail(IPDV_EINVAL, "LM-head workspace query takes 4 shape values (got %d)", n);
      return 0;
    }
    return ipdv_lmhead_workspace_size(a[0], a[1], a[2], a[3]);
  }
  fail(IPDV_EINVAL, "unknown workspace kind %d", which);
  return 0;
}

int lmhead_logsoftmax_verify(const void* hidden, const void* W, const int32_t* prop_tok,
                             const int32_t* out_rows, int M, int Hd, int V, int K, float* lse,
                             float* logp_prop, int32_t* argmax, int32_t* topk_idx,
                             float* topk_logp, float* entropy, int dtype, void* workspace,
                             size_t workspace_bytes, void* hip_stream) {
  int st = lm_shape_check(M, Hd, V, K);
  if (st != IPDV_OK) return st;
  bool bf16, tiled;
  if ((st = w_dtype(dtype, &bf16, &tiled)) != IPDV_OK) return st;
  if (M == 0) return ok();
  if (!hidden || !W || !prop_tok || !lse || !logp_prop || !argmax || !topk_idx || !topk_logp)
    return fail(IPDV_EINVAL, "null required pointer");
  const ipdv::LmPlan pl = ipdv::lm_plan(M, Hd, V, K, bf16);
  const size_t need = ipdv::lm_plan(M, Hd, V, K, true).workspace_bytes;
  if (!workspace || workspace_bytes < need)
    return fail(IPDV_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", need,
                workspace ? workspace_bytes : (size_t)0);
  ipdv::LmLaunch L{hidden, W, prop_tok, out_rows, M, Hd, V, K, lse, logp_prop, argmax,
                   topk_idx, topk_logp, entropy, bf16, workspace, tiled};
  hipError_t e = ipdv::launch_lmhead(L, pl, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("lmhead_logsoftmax_verify launch", e);
  return ok();
}

int sample_takeover(const void* hidden, const void* W, int M, int Hd, int V, int K,
                    const void* workspace, size_t workspace_bytes, const int32_t* seq_ids,
                    int n_seq, const int32_t* cu_q, const uint8_t* driver, const int32_t* event_row,
                    const int32_t* row_local, const float* u, int32_t eos_id, int32_t* token,
                    uint8_t* finished, int dtype, void* hip_stream) {
  int st = lm_shape_check(M, Hd, V, K);
  if (st != IPDV_OK) return st;
  bool bf16, tiled;
  if ((st = w_dtype(dtype, &bf16, &tiled)) != IPDV_OK) return st;
  if (n_seq < 0) return fail(IPDV_EINVAL, "n_seq must be >= 0 (got %d)", n_seq);
  if (n_seq > 65535 * 32) return fail(IPDV_EUNSUPPORTED, "n_seq too large");
  if (n_seq == 0) return ok();
  if (!hidden || !W || !cu_q || !driver || !event_row || !u || !token || !finished)
    return fail(IPDV_EINVAL, "null required pointer");
  const ipdv::LmPlan pl = ipdv::lm_plan(M, Hd, V, K, bf16);
  const size_t need = ipdv::lm_plan(M, Hd, V, K, true).workspace_bytes;
  if (!workspace || workspace_bytes < need)
    return fail(IPDV_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", need,
                workspace ? workspace_bytes : (size_t)0);
  ipdv::SampleLaunch L{hidden, W, M, Hd, V, K, workspace, seq_ids, n_seq, cu_q, driver, event_row,
                       row_local, u, eos_id, token, finished, bf16, tiled};
  hipError_t e = ipdv::launch_sample_takeover(L, pl, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("sample_takeover launch", e);
  return ok();
}

int lmhead_sample(const void* hidden, const void* W, int M, int Hd, int V, int K,
                  const void* workspace, size_t workspace_bytes, const float* u, int32_t* token,
                  int dtype, void* hip_stream) {
  int st = lm_shape_check(M, Hd, V, K);
  if (st != IPDV_OK) return st;
  bool bf16, tiled;
  if ((st = w_dtype(dtype, &bf16, &tiled)) != IPDV_OK) return st;
  if (M == 0) return ok();
  if (!hidden || !W || !u || !token) return fail(IPDV_EINVAL, "null required pointer");
  const ipdv::LmPlan pl = ipdv::lm_plan(M, Hd, V, K, bf16);
  const size_t need = ipdv::lm_plan(M, Hd, V, K, true).workspace_bytes;
  if (!workspace || workspace_bytes < need)
    return fail(IPDV_EWORKSPACE, "workspace of %zu bytes needed (got %zu)", need,
                workspace ? workspace_bytes : (size_t)0);
  ipdv::SampleLaunch L{hidden, W, M, Hd, V, K, workspace, nullptr, 0, nullptr, nullptr, nullptr,
                       nullptr, u, -1, token, nullptr, bf16, tiled};
  hipError_t e = ipdv::launch_sample_rows(L, pl, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("lmhead_sample launch", e);
  return ok();
}

int accept_scan_rule(const int32_t* cu_q, const int32_t* prop_tok, const int32_t* topk_idx,
                     int K, const uint8_t* driver, const int32_t* ctx_lens,
                     const int32_t* seq_lens, int32_t eos_id, int32_t max_len, int B,
                     int take_rule, int hand_rule, const float* ent, float tau_take,
                     float tau_hand, int32_t* n_acc, int32_t* event_row, uint8_t* next_driver,
                     uint8_t* finished, int32_t* new_cache_len, uint8_t* src, void* hip_stream) {
  if (B < 0) return fail(IPDV_EINVAL, "B must be >= 0 (got %d)", B);
  if (K < 0 || K > IPDV_MAX_K) return fail(IPDV_EINVAL, "K=%d must be in [0, %d]", K, IPDV_MAX_K);
  if (take_rule != IPDV_TAKE_COVERAGE && take_rule != IPDV_TAKE_ENTROPY)
    return fail(IPDV_EINVAL, "unknown takeover rule %d", take_rule);
  if (hand_rule != IPDV_HAND_COVERAGE && hand_rule != IPDV_HAND_FIXED_ONE &&
      hand_rule != IPDV_HAND_ENTROPY)
    return fail(IPDV_EINVAL, "unknown handback rule %d", hand_rule);
  if (B == 0) return ok();
  const bool uses_cov = take_rule == IPDV_TAKE_COVERAGE || hand_rule == IPDV_HAND_COVERAGE;
  const bool uses_ent = take_rule == IPDV_TAKE_ENTROPY || hand_rule == IPDV_HAND_ENTROPY;
  if (!cu_q || !prop_tok || (K > 0 && uses_cov && !topk_idx) || !driver || !ctx_lens ||
      !seq_lens || !n_acc || !event_row || !next_driver || !finished || !new_cache_len || !src)
    return fail(IPDV_EINVAL, "null required pointer");
  if (uses_ent && !ent) return fail(IPDV_EINVAL, "an entropy rule needs ent");
  ipdv::ScanLaunch L{cu_q, prop_tok, topk_idx, K, driver, ctx_lens, seq_lens, eos_id, max_len,
                     B, n_acc, event_row, next_driver, finished, new_cache_len, src,
                     take_rule, hand_rule, ent, tau_take, tau_hand};
  hipError_t e = ipdv::launch_accept_scan(L, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("accept_scan launch", e);
  return ok();
}

int accept_scan(const int32_t* cu_q, const int32_t* prop_tok, const int32_t* topk_idx, int K,
                const uint8_t* driver, const int32_t* ctx_lens, const int32_t* seq_lens,
                int32_t eos_id, int32_t max_len, int B, int32_t* n_acc, int32_t* event_row,
                uint8_t* next_driver, uint8_t* finished, int32_t* new_cache_len, uint8_t* src,
                void* hip_stream) {
  return accept_scan_rule(cu_q, prop_tok, topk_idx, K, driver, ctx_lens, seq_lens, eos_id,
                          max_len, B, IPDV_TAKE_COVERAGE, IPDV_HAND_COVERAGE, nullptr, 0.f, 0.f,
                          n_acc, event_row, next_driver, finished, new_cache_len, src,
                          hip_stream);
}

int lmhead_logp_gather(const void* hidden, const void* W, int M, int Hd, int V,
                       const float* lse, const int32_t* idx, int n_idx, float* logp, int dtype,
                       void* hip_stream) {
  int st = lm_shape_check(M, Hd, V, 1);
  if (st != IPDV_OK) return st;
  if (n_idx < 0 || n_idx > IPDV_MAX_GATHER)
    return fail(IPDV_EINVAL, "n_idx=%d must be in [0, %d]", n_idx, IPDV_MAX_GATHER);
  bool bf16, tiled;
  if ((st = w_dtype(dtype, &bf16, &tiled)) != IPDV_OK) return st;
  if (M == 0 || n_idx == 0) return ok();
  if (!hidden || !W || !lse || !idx || !logp) return fail(IPDV_EINVAL, "null required pointer");
  ipdv::GatherLaunch L{hidden, W, M, Hd, V, lse, idx, n_idx, logp, bf16, tiled};
  hipError_t e = ipdv::launch_logp_gather(L, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("lmhead_logp_gather launch", e);
  return ok();
}

size_t ipdv_lmhead_packed_w_size(int V, int Hd) {
  if (lm_shape_check(0, Hd, V, 1) != IPDV_OK) return 0;
  return (size_t)((V + 15) / 16) * 16 * Hd * 2;
}

int lmhead_pack_w(const void* W, int V, int Hd, void* W_tiled, int dtype, void* hip_stream) {
  int st = lm_shape_check(0, Hd, V, 1);
  if (st != IPDV_OK) return st;
  if (dtype != IPDV_BF16) return fail(IPDV_EUNSUPPORTED, "tiled W is bf16 only (dtype %d)", dtype);
  if (!W || !W_tiled) return fail(IPDV_EINVAL, "null required pointer");
  if (W == W_tiled) return fail(IPDV_EINVAL, "W_tiled must not alias W");
  hipError_t e = ipdv::launch_pack_w(W, V, Hd, W_tiled, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("lmhead_pack_w launch", e);
  return ok();
}

int source_split_kl(int M, int K, const int32_t* s_idx, const float* s_logp, const float* s_at_t,
                    const int32_t* t_idx, const float* t_logp, const float* t_at_s,
                    const uint8_t* src, int support, int loss_mode, float* kl_rev, float* kl_fwd,
                    float* loss, float* overlap, const int32_t* cu, int B, float* seq_loss,
                    float* t_ratio, void* hip_stream) {
  if (M < 0) return fail(IPDV_EINVAL, "M must be >= 0 (got %d)", M);
  if (K < 1 || K > IPDV_MAX_K) return fail(IPDV_EINVAL, "K=%d must be in [1, %d]", K, IPDV_MAX_K);
  if (support < IPDV_SUPPORT_UNION || support > IPDV_SUPPORT_INTERSECTION)
    return fail(IPDV_EINVAL, "unknown support %d", support);
  if (loss_mode < IPDV_LOSS_IPD_SPLIT || loss_mode > IPDV_LOSS_INVERSE_SPLIT)
    return fail(IPDV_EINVAL, "unknown loss mode %d", loss_mode);
  if (cu && B < 0) return fail(IPDV_EINVAL, "B must be >= 0 (got %d)", B);
  if (M > 0 && (!s_idx || !s_logp || !s_at_t || !t_idx || !t_logp || !t_at_s))
    return fail(IPDV_EINVAL, "null required pointer");
  if ((loss || cu) && !src) return fail(IPDV_EINVAL, "the loss needs src");
  if (cu && B > 0 && !loss) return fail(IPDV_EINVAL, "per-segment values need the row loss");
  ipdv::KlLaunch L{M, K, s_idx, s_logp, s_at_t, t_idx, t_logp, t_at_s, src, support, loss_mode,
                   kl_rev, kl_fwd, loss, overlap, cu, cu ? B : 0, seq_loss, t_ratio};
  hipError_t e = ipdv::launch_source_split_kl(L, reinterpret_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail("source_split_kl launch", e);
  return ok();
}

}  // extern "C"
