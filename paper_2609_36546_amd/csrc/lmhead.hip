// LM head + vocabulary log-softmax + top-K support for gfx950, without
// writing the logits to memory.
//
// The verifier's next-token distribution at each window row (temperature 1)
// gives the proposed token's log-prob, the LSE, the argmax, the top-K support
// of the coverage rule (Eq. (5)) and the entropy.
//
// Kernel 1 (GEMM + epilogue).  logits^T = W . hidden^T with
// v_mfma_f32_32x32x16_bf16: A = 32 vocabulary rows of W (read straight from
// HBM into registers: each W element is used by exactly one wave), B = 32
// hidden rows staged through LDS (shared by the four waves).  A workgroup
// owns 256 vocabulary entries x up to 128 hidden rows; wave w owns the
// vocabulary quarter [64w, 64w+64).  In the accumulator layout a lane holds
// one hidden row and 16 vocabulary entries per 32x32 block, so every per-row
// reduction over the vocabulary is in-lane plus one exchange with lane l^32.
// For each (row, 64-entry group) the epilogue emits a 20-byte record: the
// largest logit v1 and its index, the second largest v2 and its index,
// s = sum exp(l - v1) and e = sum exp(l - v1) * l.
//
// Kernel 2 (merge, one workgroup per row).  LSE = M + log sum_g s_g e^(v1_g-M),
// entropy = LSE - (sum_g e_g e^(v1_g-M)) / (sum_g s_g e^(v1_g-M)).  Top-K: the
// K best of the recorded (v1, v2) candidates; a group whose v2 made it into
// that list may hide a third element that belongs too, so such a group's 64
// logits are recomputed exactly and the selection is redone -- the result is
// the exact top-K of all V logits (ties: lower index first).  The proposal's
// logit is one dot product.
#include "common.h"
#include "kernels.h"

namespace ipdv {
namespace {

constexpr int kVT = 256;      // vocabulary entries per workgroup
constexpr int kGroup = 64;    // vocabulary entries per record (one wave's share)
constexpr int kStage = 64;    // hidden channels per pipeline stage
constexpr int kLdsPad = 8;    // elements of padding per LDS row (bank spread)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct LmParams {
  const void* hidden;
  const void* W;
  const int32_t* prop_tok;
  const int32_t* out_rows;
  int M, Hd, V, K;
  int n_groups, n_rt, n_vt;
  float* rec_v1;      // [M][n_groups]
  float* rec_v2;
  float* rec_s;
  float* rec_e;
  int32_t* rec_idx;   // index of v1
  int32_t* rec_i2;    // index of v2
  float* lse;
  float* logp_prop;
  int32_t* argmax;
  int32_t* topk_idx;
  float* topk_logp;
  float* entropy;
};

template <typename DT> struct Mm;

template <> struct Mm<bf16> {
  static constexpr int KSTEPS = kStage / 16;      // MFMA k-steps per stage
  typedef bf16x8 frag;
  __device__ static floatx16 mma(frag a, frag b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mm<float> {
  static constexpr int KSTEPS = kStage / 2;
  typedef float frag;
  __device__ static floatx16 mma(frag a, frag b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// Hidden-channel offset, within a stage, of the value(s) lane half h supplies
// at k-step ks.  Any bijection works as long as A and B agree; these keep each
// lane's loads contiguous.
template <typename DT> __device__ __forceinline__ int koff(int ks, int h);
template <> __device__ __forceinline__ int koff<bf16>(int ks, int h) { return 16 * ks + 8 * h; }
template <> __device__ __forceinline__ int koff<float>(int ks, int h) { return 32 * h + ks; }

template <typename DT>
struct WFrags {
  typename Mm<DT>::frag a[2][Mm<DT>::KSTEPS];
};

template <typename DT>
__device__ __forceinline__ void load_w(const LmParams& p, WFrags<DT>& f, int vbase, int k0) {
  const int lane = lane_id();
  const int h = lane >> 5;
  const DT* W = reinterpret_cast<const DT*>(p.W);
#pragma unroll
  for (int vb = 0; vb < 2; ++vb) {
    const int v = vbase + 32 * vb + (lane & 31);
    const bool ok = v < p.V;
    const DT* row = W + (size_t)(ok ? v : 0) * p.Hd + k0;
    if constexpr (sizeof(DT) == 2) {
#pragma unroll
      for (int ks = 0; ks < Mm<DT>::KSTEPS; ++ks) {
        bf16x8 x = ld16<bf16x8>(row + koff<DT>(ks, h));
        f.a[vb][ks] = ok ? x : bf16x8{};
      }
    } else {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        floatx4 x = ld16<floatx4>(row + 32 * h + 4 * c);
#pragma unroll
        for (int e = 0; e < 4; ++e) f.a[vb][4 * c + e] = ok ? x[e] : 0.f;
      }
    }
  }
}

// Top-2 (value desc, index asc) insertion of (x, ix).
__device__ __forceinline__ void top2_push(float x, int ix, float& v1, int& i1, float& v2, int& i2) {
  const bool c1 = x > v1 || (x == v1 && ix < i1);
  const bool c2 = x > v2 || (x == v2 && ix < i2);
  const float nv2 = c1 ? v1 : (c2 ? x : v2);
  const int ni2 = c1 ? i1 : (c2 ? ix : i2);
  v1 = c1 ? x : v1;
  i1 = c1 ? ix : i1;
  v2 = nv2;
  i2 = ni2;
}

template <typename DT, int RB>
__global__ __launch_bounds__(256) void lmhead_gemm_kernel(LmParams p) {
  // XCD-aware order: the row tiles of one vocabulary tile are consecutive in
  // the dispatch sequence of one XCD (workgroup id % 8), so the W tile they
  // share is fetched from HBM once into that XCD's L2.
  const int id = blockIdx.x;
  const int xcd = id & 7, local = id >> 3;
  const int vt = (local / p.n_rt) * 8 + xcd;
  const int rt = local % p.n_rt;
  if (vt >= p.n_vt) return;
  constexpr int NM = 32 * RB;
  const int m0 = rt * NM;
  const int v0 = vt * kVT;
  const int tid = threadIdx.x;
  const int w = tid >> 6;
  const int lane = lane_id();
  const int h = lane >> 5;
  const int vbase = v0 + kGroup * w;

  constexpr int LDW = kStage + kLdsPad;
  __shared__ DT s_h[2][NM * LDW];

  const DT* hid = reinterpret_cast<const DT*>(p.hidden);
  // Staging of one hidden stage: NM rows x 64 channels, 16 bytes per thread-load.
  constexpr int EPL = 16 / sizeof(DT);            // elements per 16-byte load
  constexpr int LPR = kStage / EPL;               // loads per row
  constexpr int NLD = (NM * LPR + 255) / 256;     // loads per thread
  typedef __attribute__((__vector_size__(16))) int i32x4;
  i32x4 stage_regs[NLD];

  auto load_hidden = [&](int k0) {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int e = tid + 256 * u;
      const int r = e / LPR, c = e % LPR;
      const int m = m0 + r;
      i32x4 x = {0, 0, 0, 0};
      if (r < NM && m < p.M) x = ld16<i32x4>(hid + (size_t)m * p.Hd + k0 + EPL * c);
      stage_regs[u] = x;
    }
  };
  auto store_hidden = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int e = tid + 256 * u;
      const int r = e / LPR, c = e % LPR;
      if (r < NM) *reinterpret_cast<i32x4*>(&s_h[buf][r * LDW + EPL * c]) = stage_regs[u];
    }
  };

  floatx16 acc[2][RB];
#pragma unroll
  for (int vb = 0; vb < 2; ++vb)
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[vb][rb][e] = 0.f;

  const int nst = p.Hd / kStage;
  WFrags<DT> fa, fb;
  load_hidden(0);
  load_w<DT>(p, fa, vbase, 0);
  store_hidden(0);
  for (int st = 0; st < nst; ++st) {
    const bool more = st + 1 < nst;
    if (more) {
      load_hidden((st + 1) * kStage);
      load_w<DT>(p, fb, vbase, (st + 1) * kStage);
    }
    __syncthreads();
    const DT* sb = s_h[st & 1];
#pragma unroll
    for (int ks = 0; ks < Mm<DT>::KSTEPS; ++ks) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const DT* src = sb + (32 * rb + (lane & 31)) * LDW + koff<DT>(ks, h);
        typename Mm<DT>::frag b;
        if constexpr (sizeof(DT) == 2) b = *reinterpret_cast<const bf16x8*>(src);
        else b = *src;
#pragma unroll
        for (int vb = 0; vb < 2; ++vb) acc[vb][rb] = Mm<DT>::mma(fa.a[vb][ks], b, acc[vb][rb]);
      }
    }
    if (more) {
      store_hidden((st + 1) & 1);
      fa = fb;
    }
  }

  // Epilogue: per hidden row (lane column) and this wave's 64 vocabulary
  // entries.  Register e of block vb holds vocabulary entry
  // vbase + 32 vb + 8 (e / 4) + 4 h + e % 4.
  const int g = vt * (kVT / kGroup) + w;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int m = m0 + 32 * rb + (lane & 31);
    float mx = -INFINITY;
#pragma unroll
    for (int vb = 0; vb < 2; ++vb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int v = vbase + 32 * vb + 8 * (e >> 2) + 4 * h + (e & 3);
        if (v >= p.V) acc[vb][rb][e] = -INFINITY;
        mx = fmaxf(mx, acc[vb][rb][e]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float mu = (mx == -INFINITY) ? 0.f : mx;
    const float mub = mu * kLog2e;
    float s = 0.f, ee = 0.f;
    float v1 = -INFINITY, v2 = -INFINITY;
    int i1 = 0x7fffffff, i2 = 0x7fffffff;
#pragma unroll
    for (int vb = 0; vb < 2; ++vb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float x = acc[vb][rb][e];
        const int v = vbase + 32 * vb + 8 * (e >> 2) + 4 * h + (e & 3);
        const float pe = fast_exp2(x * kLog2e - mub);
        s += pe;
        ee += (v < p.V) ? pe * x : 0.f;
        top2_push(x, v, v1, i1, v2, i2);
      }
    s += __shfl_xor(s, 32, kWave);
    ee += __shfl_xor(ee, 32, kWave);
    {
      const float ov1 = __shfl_xor(v1, 32, kWave), ov2 = __shfl_xor(v2, 32, kWave);
      const int oi1 = __shfl_xor(i1, 32, kWave), oi2 = __shfl_xor(i2, 32, kWave);
      top2_push(ov1, oi1, v1, i1, v2, i2);
      top2_push(ov2, oi2, v1, i1, v2, i2);
    }
    if (h == 0 && m < p.M && g < p.n_groups) {
      const size_t r = (size_t)m * p.n_groups + g;
      p.rec_v1[r] = v1;
      p.rec_v2[r] = v2;
      p.rec_s[r] = (mx == -INFINITY) ? 0.f : s;
      p.rec_e[r] = (mx == -INFINITY) ? 0.f : ee;
      p.rec_idx[r] = i1;
      p.rec_i2[r] = i2;
    }
  }
}

// ---------------------------------------------------------------------------
// Merge: one workgroup (256 threads) per row.
// ---------------------------------------------------------------------------

constexpr int kMT = 256;

// (value desc, index asc) order: true if (a, ia) ranks before (b, ib).
__device__ __forceinline__ bool before(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

__device__ float block_sum(float x, float* s) {
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if (lane_id() == 0) s[w] = x;
  __syncthreads();
  float t = 0.f;
  for (int ww = 0; ww < kMT / kWave; ++ww) t += s[ww];
  return t;
}

__device__ float block_max(float x, float* s) {
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, kWave));
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if (lane_id() == 0) s[w] = x;
  __syncthreads();
  float t = -INFINITY;
  for (int ww = 0; ww < kMT / kWave; ++ww) t = fmaxf(t, s[ww]);
  return t;
}

// Candidates per row: two per group plus every element of the groups whose
// second-best made it into the list.  Such a group contributes two entries
// to a K-entry list, so at most K/2 groups are ever recomputed.
constexpr int kMaxSplit = IPDV_MAX_K_DEV / 2;
constexpr int kSplitCand = kMaxSplit * kGroup;

// One wave computes the exact logit of vocabulary entry v for row m.
template <typename DT>
__device__ float wave_dot(const LmParams& p, int m, int v) {
  const DT* hr = reinterpret_cast<const DT*>(p.hidden) + (size_t)m * p.Hd;
  const DT* wr = reinterpret_cast<const DT*>(p.W) + (size_t)v * p.Hd;
  constexpr int EPL = 16 / sizeof(DT);
  float acc = 0.f;
  for (int k = EPL * lane_id(); k < p.Hd; k += EPL * kWave) {
    if constexpr (sizeof(DT) == 2) {
      bf16x8 a = ld16<bf16x8>(hr + k), b = ld16<bf16x8>(wr + k);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = fmaf(static_cast<float>(a[e]), static_cast<float>(b[e]), acc);
    } else {
      floatx4 a = ld16<floatx4>(hr + k), b = ld16<floatx4>(wr + k);
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = fmaf(a[e], b[e], acc);
    }
  }
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, kWave);
  return acc;
}

// Groups per merge thread held in registers: V <= kMT * kMaxGPT * kGroup.
constexpr int kMaxGPT = 16;

// Wave-wide best (value desc, index asc) of one candidate per lane.
__device__ __forceinline__ void wave_best(float& v, int& ix) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(v, o, kWave);
    const int oi = __shfl_xor(ix, o, kWave);
    if (before(ov, oi, v, ix)) { v = ov; ix = oi; }
  }
}

// K picks in order from the lane-held candidates c[0..n) plus extra LDS
// candidates; out_v / out_i receive the wave's top-K (lane 0 writes).
template <int N>
__device__ __forceinline__ void wave_topk(const float (&cv)[N], const int (&ci)[N],
                                          const float* xv, const int* xi, int nx, int K,
                                          float* out_v, int* out_i) {
  float last_v = INFINITY;
  int last_i = -1;
  for (int k = 0; k < K; ++k) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int c = 0; c < N; ++c)
      if (before(last_v, last_i, cv[c], ci[c]) && before(cv[c], ci[c], bv, bi)) { bv = cv[c]; bi = ci[c]; }
    for (int c = lane_id(); c < nx; c += kWave)
      if (before(last_v, last_i, xv[c], xi[c]) && before(xv[c], xi[c], bv, bi)) { bv = xv[c]; bi = xi[c]; }
    wave_best(bv, bi);
    if (lane_id() == 0) { out_v[k] = bv; out_i[k] = bi; }
    last_v = bv;
    last_i = bi;
  }
}

template <typename DT>
__global__ __launch_bounds__(kMT) void lmhead_merge_kernel(LmParams p) {
  const int m = blockIdx.x;
  const int tid = threadIdx.x;
  const int wv = tid >> 6;
  const int G = p.n_groups;
  const int K = p.K;
  const size_t base = (size_t)m * G;
  constexpr int NW = kMT / kWave;
  __shared__ float s_red[8];
  __shared__ float s_wv[NW][IPDV_MAX_K_DEV];
  __shared__ int s_wi[NW][IPDV_MAX_K_DEV];
  __shared__ float s_top_v[IPDV_MAX_K_DEV];
  __shared__ int s_top_i[IPDV_MAX_K_DEV];
  __shared__ int s_split[kMaxSplit];
  __shared__ int s_nsplit;
  __shared__ float s_cv[kSplitCand];   // recomputed logits of split groups
  __shared__ int s_ci[kSplitCand];

  // This thread's groups: tid, tid + kMT, ... (register resident).
  float cv[2 * kMaxGPT];
  int ci[2 * kMaxGPT];
  float mx = -INFINITY;
#pragma unroll
  for (int u = 0; u < kMaxGPT; ++u) {
    const int gi = tid + kMT * u;
    const bool ok = gi < G;
    cv[2 * u] = ok ? p.rec_v1[base + gi] : -INFINITY;
    ci[2 * u] = ok ? p.rec_idx[base + gi] : 0x7fffffff;
    cv[2 * u + 1] = ok ? p.rec_v2[base + gi] : -INFINITY;
    ci[2 * u + 1] = ok ? p.rec_i2[base + gi] : 0x7fffffff;
    mx = fmaxf(mx, cv[2 * u]);
  }

  // Log-sum-exp and entropy sums (group maxima are the v1 records).
  const float M = block_max(mx, s_red);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float S = 0.f, E = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxGPT; ++u) {
    const int gi = tid + kMT * u;
    if (gi < G) {
      const float wgt = fast_exp2((cv[2 * u] - Mu) * kLog2e);
      S += p.rec_s[base + gi] * wgt;
      E += p.rec_e[base + gi] * wgt;
    }
  }
  S = block_sum(S, s_red);
  E = block_sum(E, s_red);
  const float lse = Mu + fast_log2(S) * kLn2;

  // Exact top-K.  Round 0 picks from the recorded (v1, v2) pairs.  A group
  // with two picks may hide a third member, so its 64 logits are recomputed
  // and round 1 picks again from the records of the other groups plus every
  // recomputed value; then each element left out ranks after the K-th pick.
  int nsplit = 0;
  for (int round = 0; round < 2; ++round) {
    wave_topk(cv, ci, s_cv, s_ci, nsplit * kGroup, K, s_wv[wv], s_wi[wv]);
    __syncthreads();
    if (wv == 0) {
      float xv0 = -INFINITY, xv1 = -INFINITY;
      int xi0 = 0x7fffffff, xi1 = 0x7fffffff;
      const int lane = lane_id();
      if (lane < NW * K) { xv0 = s_wv[lane / K][lane % K]; xi0 = s_wi[lane / K][lane % K]; }
      if (lane + kWave < NW * K) {
        xv1 = s_wv[(lane + kWave) / K][(lane + kWave) % K];
        xi1 = s_wi[(lane + kWave) / K][(lane + kWave) % K];
      }
      const float fv[2] = {xv0, xv1};
      const int fi[2] = {xi0, xi1};
      wave_topk(fv, fi, s_cv, s_ci, 0, K, s_top_v, s_top_i);
    }
    __syncthreads();
    if (round == 1) break;
    // Groups picked twice.
    if (tid == 0) {
      int n = 0;
      for (int a = 0; a < K; ++a)
        for (int b2 = a + 1; b2 < K; ++b2)
          if (s_top_i[a] != 0x7fffffff && s_top_i[a] / kGroup == s_top_i[b2] / kGroup) {
            const int gsp = s_top_i[a] / kGroup;
            bool seen = false;
            for (int t = 0; t < n; ++t) seen |= (s_split[t] == gsp);
            if (!seen && n < kMaxSplit) s_split[n++] = gsp;
          }
      s_nsplit = n;
    }
    __syncthreads();
    nsplit = s_nsplit;
    if (nsplit == 0) break;
    for (int c = wv; c < nsplit * kGroup; c += NW) {
      const int v = s_split[c / kGroup] * kGroup + (c % kGroup);
      const bool ok = v < p.V;
      const float x = ok ? wave_dot<DT>(p, m, v) : -INFINITY;
      if (lane_id() == 0) {
        s_cv[c] = x;
        s_ci[c] = ok ? v : 0x7fffffff;
      }
    }
    // drop the split groups' records: their members now come from s_cv
#pragma unroll
    for (int u = 0; u < kMaxGPT; ++u) {
      const int gi = tid + kMT * u;
      bool sp = false;
      for (int t = 0; t < nsplit; ++t) sp |= (s_split[t] == gi);
      if (sp) {
        cv[2 * u] = cv[2 * u + 1] = -INFINITY;
        ci[2 * u] = ci[2 * u + 1] = 0x7fffffff;
      }
    }
    __syncthreads();
  }

  const int orow = p.out_rows ? p.out_rows[m] : m;
  if (tid < K) {
    p.topk_idx[(size_t)orow * K + tid] = s_top_i[tid];
    p.topk_logp[(size_t)orow * K + tid] = s_top_v[tid] - lse;
  }
  if (tid == 0) {
    p.lse[orow] = lse;
    p.argmax[orow] = s_top_i[0];
    if (p.entropy) p.entropy[orow] = lse - E / S;
  }
  // The proposal's logit: one dot product.
  const int pv = p.prop_tok[m];
  const bool pok = pv >= 0 && pv < p.V;
  if (wv == 0) {
    const float lp = wave_dot<DT>(p, m, pok ? pv : 0);
    if (lane_id() == 0) p.logp_prop[orow] = pok ? lp - lse : NAN;
  }
}

template <typename DT, int RB>
hipError_t launch_rb(const LmParams& p, hipStream_t st) {
  const int n_vt_pad = (p.n_vt + 7) / 8 * 8;
  dim3 grid(n_vt_pad * p.n_rt);
  trace_begin(st);
  hipLaunchKernelGGL((lmhead_gemm_kernel<DT, RB>), grid, dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_mark(st);
  hipLaunchKernelGGL((lmhead_merge_kernel<DT>), dim3(p.M), dim3(kMT), 0, st, p);
  e = hipGetLastError();
  trace_mark(st);
  return e;
}

}  // namespace

LmPlan lm_plan(int M, int Hd, int V, int K, bool bf16) {
  LmPlan pl{};
  pl.n_groups = (V + kGroup - 1) / kGroup;
  pl.n_vt = (V + kVT - 1) / kVT;
  const int rows = M < 128 ? M : 128;
  pl.rb = rows <= 32 ? 1 : rows <= 64 ? 2 : rows <= 96 ? 3 : 4;
  if (!bf16) pl.rb = 1;   // fp32 tiles keep their LDS stage under 64 KB
  pl.n_rt = (M + 32 * pl.rb - 1) / (32 * pl.rb);
  const size_t recs = (size_t)M * pl.n_groups;
  pl.rec_bytes = recs * sizeof(float);
  pl.workspace_bytes = 6 * ((pl.rec_bytes + 255) / 256 * 256) + 256;
  (void)Hd;
  (void)K;
  return pl;
}

hipError_t launch_lmhead(const LmLaunch& L, const LmPlan& pl, hipStream_t st) {
  if (L.M == 0) return hipSuccess;
  LmParams p{};
  p.hidden = L.hidden;
  p.W = L.W;
  p.prop_tok = L.prop_tok;
  p.out_rows = L.out_rows;
  p.M = L.M;
  p.Hd = L.Hd;
  p.V = L.V;
  p.K = L.K;
  p.n_groups = pl.n_groups;
  p.n_rt = pl.n_rt;
  p.n_vt = pl.n_vt;
  const size_t stride = (pl.rec_bytes + 255) / 256 * 256;
  char* ws = reinterpret_cast<char*>(L.workspace);
  p.rec_v1 = reinterpret_cast<float*>(ws);
  p.rec_v2 = reinterpret_cast<float*>(ws + stride);
  p.rec_s = reinterpret_cast<float*>(ws + 2 * stride);
  p.rec_e = reinterpret_cast<float*>(ws + 3 * stride);
  p.rec_idx = reinterpret_cast<int32_t*>(ws + 4 * stride);
  p.rec_i2 = reinterpret_cast<int32_t*>(ws + 5 * stride);
  p.lse = L.lse;
  p.logp_prop = L.logp_prop;
  p.argmax = L.argmax;
  p.topk_idx = L.topk_idx;
  p.topk_logp = L.topk_logp;
  p.entropy = L.entropy;
  if (L.dtype_bf16) {
    switch (pl.rb) {
      case 1: return launch_rb<bf16, 1>(p, st);
      case 2: return launch_rb<bf16, 2>(p, st);
      case 3: return launch_rb<bf16, 3>(p, st);
      default: return launch_rb<bf16, 4>(p, st);
    }
  }
  return launch_rb<float, 1>(p, st);
}

}  // namespace ipdv
