// Host-side launch interface between the C ABI (abi.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#define IPDV_MAX_K_DEV 32
#define IPDV_MAX_GATHER_DEV 64
#define IPDV_NOALLOC_SCRATCH_BYTES_DEV (128u << 20)
#define IPDV_DRIVER_S_DEV 0
#define IPDV_TAKE_COVERAGE_DEV 0
#define IPDV_TAKE_ENTROPY_DEV 1
#define IPDV_HAND_COVERAGE_DEV 0
#define IPDV_HAND_FIXED_ONE_DEV 1
#define IPDV_HAND_ENTROPY_DEV 2
#define IPDV_SRC_S_DEV 0
#define IPDV_SRC_T_DEV 1
#define IPDV_SUPPORT_UNION_DEV 0
#define IPDV_SUPPORT_STUDENT_DEV 1
#define IPDV_SUPPORT_TEACHER_DEV 2
#define IPDV_SUPPORT_INTERSECTION_DEV 3
#define IPDV_LOSS_IPD_SPLIT_DEV 0
#define IPDV_LOSS_PURE_REVERSE_DEV 1
#define IPDV_LOSS_PURE_FORWARD_DEV 2
#define IPDV_LOSS_INVERSE_SPLIT_DEV 3

namespace ipdv {

// Timing hook (see ipdv_trace_events): trace_begin() at the start of an entry
// point's launches, trace_mark() after each kernel.
void trace_begin(hipStream_t st);
void trace_mark(hipStream_t st);

// ---- verification-stage attention ----
struct AttnPlan {
  int n_qg;            // 64-row query groups per (sequence, KV head)
  int qt;              // 16-row MFMA tiles per group (1..4)
  int sub;             // keys per wave
  int chunk;           // keys per workgroup
  int max_chunks;      // chunk slots per group (padded to a multiple of 8)
  int sk;              // full 64-row groups of 16-slot D = 128 pages: persistent stream-K kernel (bf16)
  int sk_qt;           // stream-K: 16-row tiles per wave (1: 64-row items, 2: 128-row items)
  int sk_n_qg;         // stream-K: items per (sequence, KV head)
  size_t part_o_bytes, part_lse_bytes, workspace_bytes;
  size_t sk_o_bytes, sk_lse_bytes;   // stream-K partial layout (when sk)
};

struct AttnLaunch {
  const void* q;
  const void* k_new;
  const void* v_new;
  void* k_cache;
  void* v_cache;
  const int32_t* page_table;
  int max_pages;
  const int32_t* ctx_lens;
  const int32_t* cu_q;
  const int32_t* seq_ids;
  int n_seq;
  void* out;
  int Hq, Hkv, D, page_size, num_pages;
  float scale;
  bool dtype_bf16;
  void* workspace;
};

// Compute units of the current device (cached per device; 256 if unknown).
int device_cus();

AttnPlan attn_plan(int n_seq, int Hq, int Hkv, int D, int max_q, int max_pages, int page_size);
hipError_t launch_verify_attn(const AttnLaunch& L, const AttnPlan& pl, hipStream_t st);
// The same launches with the split-KV partials in the library's per-device
// scratch array (L.workspace is ignored); pl.workspace_bytes must not exceed
// IPDV_NOALLOC_SCRATCH_BYTES_DEV.
hipError_t launch_verify_attn_noalloc(const AttnLaunch& L, const AttnPlan& pl, hipStream_t st);

// ---- LM head + log-softmax ----
struct LmPlan {
  int n_groups, n_vt, n_rt, rb;
  int rec_stride;      // record entries per row (n_groups rounded up to a multiple of 4)
  size_t rec_bytes, workspace_bytes;
  size_t hid_off;      // byte offset of the packed hidden copy (bf16) in the workspace
};

struct LmLaunch {
  const void* hidden;
  const void* W;
  const int32_t* prop_tok;
  const int32_t* out_rows;
  int M, Hd, V, K;
  float* lse;
  float* logp_prop;
  int32_t* argmax;
  int32_t* topk_idx;
  float* topk_logp;
  float* entropy;
  bool dtype_bf16;
  void* workspace;
  bool w_tiled = false;        // W packed by lmhead_pack_w
};

LmPlan lm_plan(int M, int Hd, int V, int K, bool bf16);
hipError_t launch_lmhead(const LmLaunch& L, const LmPlan& pl, hipStream_t st);

struct SampleLaunch {
  const void* hidden;
  const void* W;
  int M, Hd, V, K;
  const void* workspace;       // the records of the preceding LM-head call
  const int32_t* seq_ids;      // sequences to draw for (NULL: 0 .. n_seq-1)
  int n_seq;
  const int32_t* cu_q;
  const uint8_t* driver;
  const int32_t* event_row;
  const int32_t* row_local;
  const float* u;
  int32_t eos_id;
  int32_t* token;
  uint8_t* finished;
  bool dtype_bf16;
  bool w_tiled = false;
};

hipError_t launch_sample_takeover(const SampleLaunch& L, const LmPlan& pl, hipStream_t st);
// one draw per hidden row: u [M] and token [M] (the sequence fields unused)
hipError_t launch_sample_rows(const SampleLaunch& L, const LmPlan& pl, hipStream_t st);

// ---- log-probs at given vocabulary indices ----
struct GatherLaunch {
  const void* hidden;
  const void* W;
  int M, Hd, V;
  const float* lse;            // [M], the LM head's
  const int32_t* idx;          // [M, n]
  int n;
  float* logp;                 // [M, n]
  bool dtype_bf16;
  bool w_tiled = false;
};

// ---- W in 16-row x 32-channel blocks (bf16) ----
hipError_t launch_pack_w(const void* W, int V, int Hd, void* W_tiled, hipStream_t st);

hipError_t launch_logp_gather(const GatherLaunch& L, hipStream_t st);

// ---- source-split KL values ----
struct KlLaunch {
  int M, K;
  const int32_t* s_idx;
  const float* s_logp;
  const float* s_at_t;
  const int32_t* t_idx;
  const float* t_logp;
  const float* t_at_s;
  const uint8_t* src;
  int support, loss_mode;
  float* kl_rev;
  float* kl_fwd;
  float* loss;
  float* overlap;
  const int32_t* cu;
  int B;
  float* seq_loss;
  float* t_ratio;
};

hipError_t launch_source_split_kl(const KlLaunch& L, hipStream_t st);

// ---- verdict scan ----
struct ScanLaunch {
  const int32_t* cu_q;
  const int32_t* prop_tok;
  const int32_t* topk_idx;
  int K;
  const uint8_t* driver;
  const int32_t* ctx_lens;
  const int32_t* seq_lens;
  int32_t eos_id, max_len;
  int B;
  int32_t* n_acc;
  int32_t* event_row;
  uint8_t* next_driver;
  uint8_t* finished;
  int32_t* new_cache_len;
  uint8_t* src;
  // rule variants (IPDV_TAKE_*, IPDV_HAND_*); ent is read only by the entropy rules
  int take_rule = 0, hand_rule = 0;
  const float* ent = nullptr;
  float tau_take = 0.f, tau_hand = 0.f;
};

hipError_t launch_accept_scan(const ScanLaunch& L, hipStream_t st);

}  // namespace ipdv
