// Verdict stage for gfx950: the top-K coverage rule of Eq. (9) applied to each
// sequence's window as a first-event scan (Section 3.2.3, verdict stage), and
// the rule variants named after Eq. (9) in Section 3.2.1: an entropy
// threshold in place of either coverage test, the two chosen independently,
// and SKD's fixed one-token handback.
//
// One wave per sequence.  Lane i tests row i of the window in parallel
// (is the draft in the verifier's top-K; is it EOS; does it fit under the
// maximum length), a 64-bit ballot marks the rows that end the scan, and the
// first marked row (find-first-set) decides the verdict -- no serial walk.
#include "common.h"
#include "kernels.h"

namespace ipdv {
namespace {

struct ScanParams {
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
  int take_rule, hand_rule;
  const float* ent;
  float tau_take, tau_hand;
};

__global__ __launch_bounds__(256) void accept_scan_kernel(ScanParams p) {
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= p.B) return;
  const int lane = lane_id();
  const int r0 = p.cu_q[b];
  const int kb = p.cu_q[b + 1] - r0;
  const int drv = p.driver[b];
  const long seq_len = p.seq_lens[b];
  const long max_len = p.max_len;

  int n_acc = kb, event = -1, fin = 0, takeover = 0;
  for (int i0 = 0; i0 < kb; i0 += kWave) {
    const int i = i0 + lane;
    const bool valid = i < kb;
    bool take = false, hand = false, is_eos = false;
    if (valid) {
      const int row = r0 + i;
      const int tok = p.prop_tok[row];
      // coverage: the draft among the verifier's K entries (K = 0: none)
      bool covered = false;
      if (p.take_rule == IPDV_TAKE_COVERAGE_DEV || p.hand_rule == IPDV_HAND_COVERAGE_DEV) {
        const int32_t* tk = p.topk_idx + (size_t)row * p.K;
        for (int kk = 0; kk < p.K; ++kk) covered |= (tk[kk] == tok);
      }
      // entropy thresholds compare as IEEE floats: a NaN passes neither test
      const float e = (p.take_rule == IPDV_TAKE_ENTROPY_DEV || p.hand_rule == IPDV_HAND_ENTROPY_DEV)
                          ? p.ent[row] : 0.f;
      take = p.take_rule == IPDV_TAKE_COVERAGE_DEV ? !covered : e > p.tau_take;
      hand = p.hand_rule == IPDV_HAND_COVERAGE_DEV ? covered
             : p.hand_rule == IPDV_HAND_FIXED_ONE_DEV ? true : e <= p.tau_hand;
      is_eos = tok == p.eos_id;
    }
    const bool allowed = seq_len + i < max_len;
    const bool cap_after = seq_len + i + 1 >= max_len;
    bool stop;
    if (drv == IPDV_DRIVER_S_DEV) stop = !allowed || take || is_eos || cap_after;
    else stop = !allowed || hand || is_eos || cap_after;
    const unsigned long long mask = __ballot(valid && stop);
    if (mask == 0) continue;
    const int first = __builtin_ctzll(mask);
    const int fi = i0 + first;
    // the first stopping lane's flags, read with one readlane (first is wave-uniform)
    const int flags = (allowed ? 1 : 0) | (take ? 2 : 0) | (hand ? 4 : 0) | (is_eos ? 8 : 0) |
                      (cap_after ? 16 : 0);
    const int f = __builtin_amdgcn_readlane(flags, first);
    const bool f_allowed = f & 1, f_take = f & 2, f_hand = f & 4, f_eos = f & 8, f_cap = f & 16;
    if (!f_allowed) {
      n_acc = fi;
      fin = 1;
    } else if (drv == IPDV_DRIVER_S_DEV && f_take) {
      n_acc = fi;
      event = fi;
      takeover = 1;
    } else {
      n_acc = fi + 1;
      if (drv != IPDV_DRIVER_S_DEV && f_hand) event = fi;
      fin = (f_eos || f_cap) ? 1 : 0;
    }
    break;
  }
  const uint8_t label = drv == IPDV_DRIVER_S_DEV ? 0 : 1;
  for (int i = lane; i < kb; i += kWave) p.src[r0 + i] = i < n_acc ? label : (uint8_t)255;
  if (lane == 0) {
    p.n_acc[b] = n_acc;
    p.event_row[b] = event;
    // an event flips the driver, except a takeover under the fixed one-token
    // handback: the replacement is the teacher's only token (SKD)
    const bool flip = event >= 0 && !(takeover && p.hand_rule == IPDV_HAND_FIXED_ONE_DEV);
    p.next_driver[b] = flip ? (uint8_t)(1 - drv) : (uint8_t)drv;
    p.finished[b] = (uint8_t)fin;
    p.new_cache_len[b] = p.ctx_lens[b] + n_acc + takeover;
  }
}

}  // namespace

hipError_t launch_accept_scan(const ScanLaunch& L, hipStream_t st) {
  if (L.B == 0) return hipSuccess;
  ScanParams p{L.cu_q, L.prop_tok, L.topk_idx, L.K, L.driver, L.ctx_lens, L.seq_lens,
               L.eos_id, L.max_len, L.B, L.n_acc, L.event_row, L.next_driver, L.finished,
               L.new_cache_len, L.src, L.take_rule, L.hand_rule, L.ent, L.tau_take,
               L.tau_hand};
  trace_begin(st);
  hipLaunchKernelGGL(accept_scan_kernel, dim3((L.B + 3) / 4), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  trace_mark(st);
  return e;
}

}  // namespace ipdv
