// Source-split KL values for gfx950 (Section 3.2.2): per position, the two
// models' distributions renormalised on the top-K support (Eqs. (5), (6)),
// the reverse and forward KL of Eq. (10), the row's loss by token source, the
// top-K overlap ratio; per trajectory segment, the length-normalised loss of
// Eq. (11) and the teacher-intervention ratio.
//
// One wave per row.  Lanes 0..K-1 hold the student's top-K entries (index,
// its own log-prob, the teacher's log-prob there), lanes 32..32+K-1 the
// teacher's (index, the student's log-prob there, its own log-prob).  K <= 32,
// so a whole row is one wave: membership of each index in the other list is
// 32 shuffles, and every sum is a wave reduction.
#include "common.h"
#include "kernels.h"

namespace ipdv {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// natural-log log-sum-exp over the lanes with `on`; -inf when none is on
__device__ __forceinline__ float wave_lse(float x, bool on) {
  const float mx = wave_max(on ? x : -INFINITY);
  if (mx == -INFINITY) return -INFINITY;
  const float s = wave_sum(on ? fast_exp2((x - mx) * kLog2e) : 0.f);
  return mx + fast_log2(s) * kLn2;
}

__global__ __launch_bounds__(256) void kl_rows_kernel(KlLaunch p) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= p.M) return;
  const int lane = lane_id();
  const int K = p.K;
  const bool sl = lane < 32 && lane < K;               // a student-list lane
  const bool tl = lane >= 32 && lane - 32 < K;         // a teacher-list lane
  const size_t o = (size_t)r * K + (sl ? lane : tl ? lane - 32 : 0);
  const int v = sl ? p.s_idx[o] : tl ? p.t_idx[o] : -1;
  const float lp = sl ? p.s_logp[o] : tl ? p.s_at_t[o] : 0.f;   // log pi(v)
  const float lq = sl ? p.t_at_s[o] : tl ? p.t_logp[o] : 0.f;   // log q(v)
  // is v in the other model's list?
  bool in_other = false;
  for (int j = 0; j < K; ++j) {
    const int vs = __shfl(v, j, kWave);
    const int vt = __shfl(v, 32 + j, kWave);
    in_other |= sl ? (v == vt) : (tl && v == vs);
  }
  // the support; an index in both lists counts once, from the list that
  // defines the support (the student's for the union and the intersection)
  bool on;
  switch (p.support) {
    case IPDV_SUPPORT_UNION_DEV: on = sl || (tl && !in_other); break;
    case IPDV_SUPPORT_STUDENT_DEV: on = sl; break;
    case IPDV_SUPPORT_TEACHER_DEV: on = tl; break;
    default: on = sl && in_other; break;
  }
  const float lse_p = wave_lse(lp, on);
  const float lse_q = wave_lse(lq, on);
  float rev = 0.f, fwd = 0.f;
  if (lse_p != -INFINITY) {            // an empty support gives 0
    const float a = lp - lse_p;        // log pi_bar(v)
    const float b = lq - lse_q;        // log q_bar(v)
    const float pa = on ? fast_exp2(a * kLog2e) : 0.f;
    const float pb = on ? fast_exp2(b * kLog2e) : 0.f;
    rev = wave_sum(pa > 0.f ? pa * (a - b) : 0.f);
    fwd = wave_sum(pb > 0.f ? pb * (b - a) : 0.f);
  }
  const int n_both = __popcll(__ballot(sl && in_other));
  if (lane == 0) {
    if (p.kl_rev) p.kl_rev[r] = rev;
    if (p.kl_fwd) p.kl_fwd[r] = fwd;
    if (p.overlap) p.overlap[r] = (float)n_both / (float)K;
    if (p.loss) {
      const int z = p.src[r];
      const bool s_tok = z == IPDV_SRC_S_DEV;
      float l = 0.f;
      if (z == IPDV_SRC_S_DEV || z == IPDV_SRC_T_DEV) {
        switch (p.loss_mode) {
          case IPDV_LOSS_IPD_SPLIT_DEV: l = s_tok ? rev : fwd; break;
          case IPDV_LOSS_PURE_REVERSE_DEV: l = rev; break;
          case IPDV_LOSS_PURE_FORWARD_DEV: l = fwd; break;
          default: l = s_tok ? fwd : rev; break;
        }
      }
      p.loss[r] = l;
    }
  }
}

// Eq. (11)'s inner term per segment: the mean row loss over emitted tokens
// (src S or T) and the share of teacher tokens among them.  One wave per
// segment, lanes striding over its rows.
__global__ __launch_bounds__(256) void kl_segments_kernel(KlLaunch p) {
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= p.B) return;
  const int lane = lane_id();
  const int r0 = p.cu[b], r1 = p.cu[b + 1];
  float sum = 0.f, n = 0.f, nt = 0.f;
  for (int r = r0 + lane; r < r1; r += kWave) {
    const int z = p.src[r];
    if (z == IPDV_SRC_S_DEV || z == IPDV_SRC_T_DEV) {
      sum += p.loss[r];
      n += 1.f;
      nt += z == IPDV_SRC_T_DEV ? 1.f : 0.f;
    }
  }
  sum = wave_sum(sum);
  n = wave_sum(n);
  nt = wave_sum(nt);
  if (lane == 0) {
    if (p.seq_loss) p.seq_loss[b] = n > 0.f ? sum / n : 0.f;
    if (p.t_ratio) p.t_ratio[b] = n > 0.f ? nt / n : 0.f;
  }
}

}  // namespace

hipError_t launch_source_split_kl(const KlLaunch& L, hipStream_t st) {
  if (L.M == 0 && !(L.cu && L.B > 0)) return hipSuccess;
  trace_begin(st);
  if (L.M > 0) {
    hipLaunchKernelGGL(kl_rows_kernel, dim3((L.M + 3) / 4), dim3(256), 0, st, L);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    trace_mark(st);
  }
  if (L.cu && L.B > 0) {
    hipLaunchKernelGGL(kl_segments_kernel, dim3((L.B + 3) / 4), dim3(256), 0, st, L);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    trace_mark(st);
  }
  return hipSuccess;
}

}  // namespace ipdv
