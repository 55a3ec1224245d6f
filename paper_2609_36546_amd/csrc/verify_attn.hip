// Verification-stage attention for gfx950: fused window append + split-KV
// multi-token causal grouped-query attention over a paged KV cache, and the
// split combine.
//
// Operation (Section 3.2.3 of the paper: the verifier scores all drafts of
// its sub-batch in one prefill pass over its resident cache, after the
// proposer's tokens are appended to it): for sequence b with L cached tokens
// and a k-row window, row i attends to keys 0 .. L+i of its KV head.
//
// The window's keys and values are appended to the pages first, so the
// attention streams every key, window or cached, the same way: by the
// stream-K kernel itself (each workgroup writes the window positions inside
// its own key blocks before it reads any), or by a small kernel ahead of the
// register kernel.
//
// Work decomposition.  The query rows of one (sequence, KV head) -- k window
// positions x G = Hq/Hkv heads -- are packed position-major into groups of up
// to 64 rows (four 16-row MFMA tiles), so every key byte streamed from HBM
// feeds all G heads of all k positions at once.  A workgroup (4 waves) takes
// one chunk of the key range; each wave streams its quarter in 32-key blocks
// with the next block's loads in flight while the current one is computed:
//
//   S^T[32 keys x 16 rows] = K . Q^T     v_mfma_f32_16x16x32_bf16, A = key rows
//   online softmax in exp2 units on S^T (a lane owns one query row, so the
//   running max / sum and the output rescale need no lane exchange besides
//   the two xor-shuffles of the block max)
//   O^T[d x 16 rows] += V^T . P^T        A = the channel-major value page rows,
//                                        B = P^T straight from the S^T layout
//
// The value pages are channel-major ([page][head][D][slot]), so the A operand
// of the PV product -- 8 consecutive keys of one channel -- is one 16-byte
// load, and P never leaves registers.  The key pages are sliced by 32
// channels ([page][head][D/32][slot][32]) so that every 16-key QK operand load
// reads whole cache lines.  MFMA rows of the QK product are
// permuted (row r <-> key 8(r/4) + 4s + r%4 in sub-tile s) so that each lane
// ends up holding exactly the 8 consecutive keys its PV operand needs.
//
// The four waves of a workgroup merge their partial results through LDS;
// chunks of one (sequence, head group) are merged by a combine kernel in
// log-sum-exp form, unless the sequence fits in one chunk (then the
// workgroup writes the output itself).
//
// bf16 D = 128 heads in 16-token pages (every bf16 workload), when the
// kernel's LDS tables fit, take a second kernel, verify_attn_sk_kernel below:
// persistent workgroups whose waves own one or two 16-row tiles (items of 64
// or 128 rows of one (sequence, KV head)), keys and values streamed through
// an LDS ring with direct-to-LDS loads, and the key blocks of all items split
// evenly between workgroups (stream-K); items split between workgroups are
// merged by attn_combine_sk_kernel.  Both kernels share the block arithmetic
// (attend_block) and the pool layouts.
#include <algorithm>
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace ipdv {
namespace {

constexpr int kWaves = 4;
constexpr int kBlk = 32;      // keys per block
constexpr int kRows = 64;     // packed query rows per workgroup
constexpr float kRescaleSlack = 8.0f;  // log2 units a stale running max may lag
constexpr int kQPad = 8;      // elements of padding per LDS query row (bank spread)

struct AttnParams {
  const void* q;
  const void* k_new;
  const void* v_new;
  void* k_cache;
  void* v_cache;
  const int32_t* page_table;
  const int32_t* ctx_lens;
  const int32_t* cu_q;
  const int32_t* seq_ids;
  void* out;
  float* part_o;      // [slots][kRows][D] (stream-K: [slots][item_rows][D])
  float* part_lse;    // [slots][kRows] (stream-K: [slots][item_rows])
  int max_pages;
  int Hq, Hkv, G;
  int page_size, log2ps, num_pages;
  int chunk, sub;     // keys per workgroup chunk / per wave
  int max_chunks, n_qg, n_seq;
  float scale_log2;   // softmax scale * log2(e)
  int32_t* sk_start;  // stream-K: first block of every item (written by the attention kernel)
  int32_t* sk_ne;     // stream-K: non-empty items before every item (written with sk_start)
  int sk_grid;        // stream-K: persistent workgroups
  int item_rows;      // stream-K: packed query rows per item (64, or 128 with two tiles per wave)
  int sk_first;       // stream-K: workgroups dispatched first on their CU (the CU count)
};

template <typename DT, int D> struct Frags;

template <int D> struct Frags<bf16, D> {
  static constexpr int KS = D / 32;   // k-steps of the QK product
  bf16x8 k[2][KS];                    // A operand: key rows of sub-tiles 0/1
  bf16x8 v[D / 16];                   // A operand: channel rows, 8 keys each
  __device__ __forceinline__ bf16x8 kf(int st, int ks) const { return k[st][ks]; }
  __device__ __forceinline__ bf16x8 vf(int dt) const { return v[dt]; }
};

template <int D> struct Frags<float, D> {
  static constexpr int KS = D / 4;    // v_mfma_f32_16x16x4_f32: one value per lane
  float k[2][KS];
  floatx4 v[D / 16][2];
};

template <typename DT, int D> struct QFrag;
template <int D> struct QFrag<bf16, D> { bf16x8 q[D / 32]; };
template <int D> struct QFrag<float, D> { float q[D / 4]; };

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Loads one 32-key block from the pages (the window has been appended by the
// time this kernel runs).  TAIL: the block reaches past the last visible key
// n_keys; value lanes of those keys are zeroed so that masked probabilities
// never meet stale or poisoned slots (their page-table entries are clamped
// into the pool, so every load stays in bounds).
template <typename DT, int D, bool TAIL>
__device__ __forceinline__ void load_block(const AttnParams& a, Frags<DT, D>& f, int t0, int n_keys,
                                           int g, int my_page, int pbase) {
  const int lane = lane_id();
  const int c16 = lane & 15, j = lane >> 4;
  // K rows: the lane's key for sub-tile s is t0 + 8*(c16/4) + 4s + c16%4; both
  // sub-tiles' keys share one 8-aligned group, hence one page.
  const int kgrp = t0 + 8 * (c16 >> 2);
  const int kpage = __shfl(my_page, clampi((kgrp >> a.log2ps) - pbase, 0, kWave - 1), kWave);
  // Key pages are [D/32][slot][32]: for sub-tile s and k-step ks the 64 lanes
  // read 4 runs of 4 consecutive slots x 64 bytes -- whole cache lines.
  const DT* kbase = reinterpret_cast<const DT*>(a.k_cache) +
                    (size_t)(kpage * a.Hkv + g) * a.page_size * D;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int slot = (kgrp + 4 * s + (c16 & 3)) & (a.page_size - 1);
    if constexpr (sizeof(DT) == 2) {
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        f.k[s][ks] = ld16<bf16x8>(kbase + ((size_t)ks * a.page_size + slot) * 32 + 8 * j);
    } else {
      // fp32: lane group j holds channels j*D/4 .. j*D/4 + D/4 - 1 (one slice run)
      const int d0 = j * (D / 4);
      const DT* row = kbase + ((size_t)(d0 / 32) * a.page_size + slot) * 32 + (d0 & 31);
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        floatx4 v = ld16<floatx4>(row + 4 * c);
        f.k[s][4 * c + 0] = v[0];
        f.k[s][4 * c + 1] = v[1];
        f.k[s][4 * c + 2] = v[2];
        f.k[s][4 * c + 3] = v[3];
      }
    }
  }
  // V^T rows: channel 16*dt + c16, keys t0 + 8j .. t0 + 8j + 7.
  const int vpos = t0 + 8 * j;
  const int vpage = __shfl(my_page, clampi((vpos >> a.log2ps) - pbase, 0, kWave - 1), kWave);
  const DT* vc = reinterpret_cast<const DT*>(a.v_cache) +
                 ((size_t)(vpage * a.Hkv + g) * D) * a.page_size + (vpos & (a.page_size - 1));
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const DT* p = vc + (size_t)(16 * dt + c16) * a.page_size;
    if constexpr (sizeof(DT) == 2) {
      f.v[dt] = ld16<bf16x8>(p);
      if constexpr (TAIL) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (vpos + e >= n_keys) f.v[dt][e] = static_cast<bf16>(0.f);
      }
    } else {
      f.v[dt][0] = ld16<floatx4>(p);
      f.v[dt][1] = ld16<floatx4>(p + 4);
      if constexpr (TAIL) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (vpos + e >= n_keys) f.v[dt][e >> 2][e & 3] = 0.f;
      }
    }
  }
}

// One 32-key block for every query tile: S^T = K Q^T for all tiles first
// (independent MFMA chains), then the online softmax in exp2 units with the
// scale folded into one FMA per score, then O^T += V^T P^T.
// Query fragments: the B operand of the QK product for tile t, k-step ks.
// LdsQ reads them from the group's rows staged in LDS; RegQ holds one tile's
// fragments in registers.
template <typename DT, int D> struct LdsQ;
template <int D> struct LdsQ<bf16, D> {
  const bf16* s_q;
  __device__ __forceinline__ bf16x8 get(int t, int ks) const {
    const int lane = lane_id();
    return *reinterpret_cast<const bf16x8*>(s_q + (16 * t + (lane & 15)) * (D + kQPad) + 8 * (lane >> 4) + 32 * ks);
  }
};
template <int D> struct LdsQ<float, D> {
  const float* s_q;
  __device__ __forceinline__ float get(int t, int ks) const {
    const int lane = lane_id();
    return s_q[(16 * t + (lane & 15)) * (D + kQPad) + (lane >> 4) * (D / 4) + ks];
  }
};
template <int D> struct RegQ {
  bf16x8 q[D / 32];
  __device__ __forceinline__ bf16x8 get(int, int ks) const { return q[ks]; }
};
// QT tiles' fragments in registers.
template <int D, int QT> struct RegQT {
  bf16x8 q[QT][D / 32];
  __device__ __forceinline__ bf16x8 get(int t, int ks) const { return q[t][ks]; }
};


template <typename DT, int D, int QT, bool TAIL, class QS, class FS>
__device__ __forceinline__ void attend_block(const AttnParams& a, const FS& f,
                                             const QS& qs, const int (&qlimit)[QT],
                                             int t0, floatx4 (&acc)[QT][D / 16],
                                             float (&m_run)[QT], float (&l_run)[QT]) {
  const int lane = lane_id();
  const int j = lane >> 4, c16 = lane & 15;
  floatx4 s[QT][2];
#pragma unroll
  for (int t = 0; t < QT; ++t) s[t][0] = s[t][1] = floatx4{0.f, 0.f, 0.f, 0.f};
  if constexpr (sizeof(DT) == 2) {
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        const bf16x8 qv = qs.get(t, ks);
#pragma unroll
        for (int st = 0; st < 2; ++st)
          s[t][st] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.kf(st, ks), qv, s[t][st], 0, 0, 0);
      }
  } else {
#pragma unroll
    for (int ks = 0; ks < D / 4; ++ks)
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        const float qv = qs.get(t, ks);
#pragma unroll
        for (int st = 0; st < 2; ++st)
          s[t][st] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.k[st][ks], qv, s[t][st], 0, 0, 0);
      }
  }
  // s[t][st][e] is the raw score of key t0 + 8j + 4st + e for the lane's row.
  float bm[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    bm[t] = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (TAIL && (t0 + 8 * j + e) >= qlimit[t]) s[t][e >> 2][e & 3] = -INFINITY;
      bm[t] = fmaxf(bm[t], s[t][e >> 2][e & 3]);
    }
  }
#pragma unroll
  for (int t = 0; t < QT; ++t) bm[t] = fmaxf(bm[t], lane_xor16(bm[t]));
#pragma unroll
  for (int t = 0; t < QT; ++t) bm[t] = fmaxf(bm[t], lane_xor32(bm[t]));
  const float c = a.scale_log2;
  float m_use[QT];
  bool rescale = false;
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const float bx = bm[t] * c;
    const float m_old = m_run[t];
    const float m_new = (bx > m_old + kRescaleSlack || m_old == -INFINITY) ? fmaxf(bx, m_old) : m_old;
    m_use[t] = (m_new == -INFINITY) ? 0.f : m_new;
    rescale |= m_new != m_old;
    bm[t] = m_old;          // keep the old running max for the rescale factor
    m_run[t] = m_new;
  }
  if (__any(rescale)) {
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const float alpha = fast_exp2(bm[t] - m_use[t]);
      l_run[t] *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[t][dt] *= alpha;
    }
  }
  if constexpr (sizeof(DT) == 2) {
    // Probabilities of every tile first, then one pass over the value
    // fragments: each fragment read from LDS feeds all QT tiles.
    bf16x8 pf[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = fast_exp2(fmaf(s[t][e >> 2][e & 3], c, -m_use[t]));
        ps += p;
        pf[t][e] = static_cast<bf16>(p);
      }
      l_run[t] += ps;
    }
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const bf16x8 v = f.vf(dt);
#pragma unroll
      for (int t = 0; t < QT; ++t)
        acc[t][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v, pf[t], acc[t][dt], 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float p[8];
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = fast_exp2(fmaf(s[t][e >> 2][e & 3], c, -m_use[t]));
        ps += p[e];
      }
      l_run[t] += ps;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          acc[t][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(f.v[dt][e >> 2][e & 3], p[e],
                                                             acc[t][dt], 0, 0, 0);
    }
  }
}

// Append: the window's keys / values go to this verifier's pages at
// positions L .. L+k-1 (one workgroup per sequence and KV head).
template <typename DT, int D>
__global__ __launch_bounds__(256) void append_window_kernel(AttnParams a) {
  const int slot = blockIdx.x / a.Hkv, g = blockIdx.x % a.Hkv;
  const int b = a.seq_ids ? a.seq_ids[slot] : slot;
  const int L = max(a.ctx_lens[b], 0);
  const int r0 = a.cu_q[b];
  const int kb = a.cu_q[b + 1] - r0;
  const int* pt_row = a.page_table + (size_t)b * a.max_pages;
  DT* kc = reinterpret_cast<DT*>(a.k_cache);
  DT* vc = reinterpret_cast<DT*>(a.v_cache);
  const DT* kn = reinterpret_cast<const DT*>(a.k_new);
  const DT* vn = reinterpret_cast<const DT*>(a.v_new);
  for (int e = threadIdx.x; e < kb * D; e += blockDim.x) {
    const int i = e / D, d = e % D;
    const int pos = L + i;
    const int page = clampi(pt_row[clampi(pos >> a.log2ps, 0, a.max_pages - 1)], 0, a.num_pages - 1);
    const int sl = pos & (a.page_size - 1);
    const size_t src = ((size_t)(r0 + i) * a.Hkv + g) * D + d;
    kc[((size_t)((page * a.Hkv + g) * (D / 32) + d / 32) * a.page_size + sl) * 32 + (d & 31)] = kn[src];
    vc[((size_t)(page * a.Hkv + g) * D + d) * a.page_size + sl] = vn[src];
  }
}

template <typename DT, int D, int QT>
__global__ __launch_bounds__(256) void verify_attn_kernel(AttnParams a) {
  // Grid: x = (sequence, KV head) -- fastest, so consecutive workgroups (which
  // the hardware deals out to the 8 XCDs round-robin) spread every chunk
  // index over all XCDs; y = row group; z = chunk.  x is padded to a
  // multiple of 8, so the row groups of one chunk (ids x apart) share an
  // XCD and its L2.
  if (blockIdx.x >= a.n_seq * a.Hkv) return;
  const int c = blockIdx.z, qg = blockIdx.y;
  const int slot = blockIdx.x / a.Hkv, g = blockIdx.x % a.Hkv;
  const int b = a.seq_ids ? a.seq_ids[slot] : slot;
  const int L = max(a.ctx_lens[b], 0);
  const int r0 = a.cu_q[b];
  const int kb = a.cu_q[b + 1] - r0;
  const int G = a.G;
  const int rows_total = kb * G;
  const int pr0 = qg * kRows;
  if (pr0 >= rows_total) return;
  const int pr_last = min(rows_total, pr0 + kRows) - 1;
  const int n_keys = L + pr_last / G + 1;
  const int n_chunks = min((n_keys + a.chunk - 1) / a.chunk, a.max_chunks);
  const int tid = threadIdx.x;
  const int w = tid / kWave;
  const int lane = lane_id();
  const int c16 = lane & 15, j = lane >> 4;
  const int* pt_row = a.page_table + (size_t)b * a.max_pages;

  if (c >= n_chunks) return;

  // The group's query rows (shared by the four waves) go to LDS; the same
  // buffer later holds the cross-wave merge.
  constexpr int kQBytes = kRows * (D + kQPad) * (int)sizeof(DT);
  constexpr int kAccBytes = 2 * QT * (D / 16) * kWave * (int)sizeof(floatx4);
  __shared__ __attribute__((aligned(16))) char s_buf[kQBytes > kAccBytes ? kQBytes : kAccBytes];
  DT* s_q = reinterpret_cast<DT*>(s_buf);
  {
    constexpr int EPL = 16 / (int)sizeof(DT);
    constexpr int LPR = D / EPL;
    for (int e = tid; e < kRows * LPR; e += blockDim.x) {
      const int r = e / LPR, cc = e % LPR;
      const int pr = pr0 + r;
      typedef __attribute__((__vector_size__(16))) int i32x4;
      i32x4 v = {0, 0, 0, 0};
      if (pr <= pr_last) {
        const int i = pr / G, hl = pr % G;
        v = ld16<i32x4>(reinterpret_cast<const DT*>(a.q) + ((size_t)(r0 + i) * a.Hq + g * G + hl) * D + EPL * cc);
      }
      *reinterpret_cast<i32x4*>(s_q + r * (D + kQPad) + EPL * cc) = v;
    }
  }
  const LdsQ<DT, D> qsrc{s_q};
  int qlimit[QT];   // keys < qlimit are visible to the lane's row of tile t
#pragma unroll
  for (int t = 0; t < QT; ++t) qlimit[t] = L + min(pr0 + 16 * t + c16, pr_last) / G + 1;
  __syncthreads();

  floatx4 acc[QT][D / 16];
  float m_run[QT], l_run[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[t][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  const int t_begin = c * a.chunk + w * a.sub;
  const int t_end = min(t_begin + a.sub, n_keys);
  if (t_begin < t_end) {
    const int pbase = t_begin >> a.log2ps;
    const int my_page = clampi(pt_row[clampi(pbase + lane, 0, a.max_pages - 1)], 0, a.num_pages - 1);
    // Full blocks of cached keys, two register sets in ping-pong: the next
    // block's loads are in flight while the current one is computed.  The
    // prefetch is unconditional (past the end it re-reads the last block,
    // an L1/L2 hit) so that the compiler can wait on exactly the older loads.
    const int main_end = min(t_end, L & ~(kBlk - 1));
    const int nb = main_end > t_begin ? (main_end - t_begin) / kBlk : 0;
    if (nb > 0) {
      Frags<DT, D> fa, fb;
      load_block<DT, D, false>(a, fa, t_begin, n_keys, g, my_page, pbase);
      for (int n = 0; n < nb; n += 2) {
        load_block<DT, D, false>(a, fb, t_begin + kBlk * min(n + 1, nb - 1), n_keys, g, my_page, pbase);
        attend_block<DT, D, QT, false>(a, fa, qsrc, qlimit, t_begin + kBlk * n, acc, m_run, l_run);
        load_block<DT, D, false>(a, fa, t_begin + kBlk * min(n + 2, nb - 1), n_keys, g, my_page, pbase);
        if (n + 1 < nb)
          attend_block<DT, D, QT, false>(a, fb, qsrc, qlimit, t_begin + kBlk * (n + 1), acc, m_run, l_run);
      }
    }
    // The block that reaches past the last visible key, or needs the causal mask.
    for (int t0 = t_begin + kBlk * nb; t0 < t_end; t0 += kBlk) {
      Frags<DT, D> ft;
      load_block<DT, D, true>(a, ft, t0, n_keys, g, my_page, pbase);
      attend_block<DT, D, QT, true>(a, ft, qsrc, qlimit, t0, acc, m_run, l_run);
    }
  }

  // Row sums are partial per lane group: reduce over the 4 groups.
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    l_run[t] += lane_xor16(l_run[t]);
    l_run[t] += lane_xor32(l_run[t]);
  }

  // Merge the four waves' partials.
  __shared__ float s_m[kWaves][kRows];
  __shared__ float s_l[kWaves][kRows];
  typedef floatx4 AccBuf[QT][D / 16][kWave];
  AccBuf* s_acc = reinterpret_cast<AccBuf*>(s_buf);
  __syncthreads();   // every wave is done reading the query rows
  if (j == 0) {
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      s_m[w][16 * t + c16] = m_run[t];
      s_l[w][16 * t + c16] = l_run[t];
    }
  }
  __syncthreads();
  float l_tot[QT], m_tot[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, s_m[ww][16 * t + c16]);
    const float Mu = (M == -INFINITY) ? 0.f : M;
    float Ls = 0.f;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) Ls += s_l[ww][16 * t + c16] * fast_exp2(s_m[ww][16 * t + c16] - Mu);
    const float f = fast_exp2(m_run[t] - Mu);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[t][dt] *= f;
    l_tot[t] = Ls;
    m_tot[t] = M;
  }
  if (w >= 2) {
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) s_acc[w - 2][t][dt][lane] = acc[t][dt];
  }
  __syncthreads();
  if (w < 2) {
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[t][dt] += s_acc[w][t][dt][lane];
  }
  __syncthreads();
  if (w == 1) {
#pragma unroll
    for (int t = 0; t < QT; ++t)
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) s_acc[0][t][dt][lane] = acc[t][dt];
  }
  __syncthreads();
  if (w != 0) return;

  const bool single = n_chunks == 1;
  const size_t pslot = (((size_t)slot * a.Hkv + g) * a.n_qg + qg) * a.max_chunks + c;
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int pr = pr0 + 16 * t + c16;
    const float inv = l_tot[t] > 0.f ? 1.f / l_tot[t] : 0.f;
    floatx4 o[D / 16];
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) o[dt] = (acc[t][dt] + s_acc[0][t][dt][lane]) * inv;
    if (pr > pr_last) continue;
    if (single) {
      const int i = pr / G, hl = pr % G;
      DT* orow = reinterpret_cast<DT*>(a.out) + ((size_t)(r0 + i) * a.Hq + g * G + hl) * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        if constexpr (sizeof(DT) == 2) {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(o[dt][e]);
          *reinterpret_cast<bf16x4*>(orow + 16 * dt + 4 * j) = v;
        } else {
          *reinterpret_cast<floatx4*>(orow + 16 * dt + 4 * j) = o[dt];
        }
      }
    } else {
      float* po = a.part_o + (pslot * kRows + (16 * t + c16)) * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * j) = o[dt];
      if (j == 0)
        a.part_lse[pslot * kRows + 16 * t + c16] =
            l_tot[t] > 0.f ? m_tot[t] + fast_log2(l_tot[t]) : -INFINITY;
    }
  }
}

// ---------------------------------------------------------------------------
// Persistent stream-K variant for full 64-row groups (bf16, D = 128, 16-token
// pages).
//
// The register kernel above holds all four 16-row tiles of a group in every
// wave, so one wave fits per SIMD; and like any kernel of one workgroup per
// key chunk it leaves a CU's load queue idle while a workgroup starts (page
// table, query rows, first block) and finishes (partials), and at the ragged
// end of the grid.  A read-only kernel of the same access pattern (random 4 KB
// pieces) reaches about 5.4-5.7 TB/s.  This kernel's loads alone stream about
// 5.2 TB/s at the teacher shape; with the attention arithmetic interleaved the
// two overlap only in part, and the whole kernel is a few percent faster than
// the register kernel.
//
// Here 2 workgroups per CU stay resident.  The 32-key blocks of all items --
// (sequence, KV head, 64-row group) -- are laid end to end, and workgroup w
// takes the w-th equal share of them, whatever items it spans.  Its 4 waves
// each own one 16-row tile (query fragments in registers).  Everything the
// workgroup reads in its loop arrives through a 3-deep LDS ring of 16 KB
// units with direct-to-LDS loads: an item's query rows (one unit), then its
// key/value blocks, then the next item's query rows, and so on.  Each wave
// issues a quarter of every unit.  The items' lengths and the page ids of the
// workgroup's blocks are read into LDS before the loop, so the loop issues no
// other loads and the ring never drains.  An item split between workgroups
// leaves one partial per piece, at slot item + workgroup, and the combine
// kernel merges them.
//
// LDS image of a key/value unit: [K page 0][K page 1][V page 0][V page 1],
// each a 4 KB page of the pool in its own layout (keys [D/32][slot][32],
// values [D][slot]); of a query unit: 64 rows of 256 bytes.  Within every
// 1 KB piece the 16-byte units are permuted so that the fragment reads of
// eight consecutive lanes hit eight distinct bank groups: unit (slot, q) of a
// key piece sits at 4 slot + (q ^ f(slot)), unit (channel, half) of a value
// piece at 2 channel + (half ^ bit 2 of the channel), unit u of query row r
// at u ^ (r % 8).  A direct-to-LDS load writes lane l's 16 bytes to unit l,
// so the loading lane fetches the global unit that belongs there.
// ---------------------------------------------------------------------------
constexpr int kSkBuf = 3;              // ring depth (units)
constexpr int kSkUnit = 16384;         // bytes per unit
constexpr int kSkMeta = 7680;          // ints of LDS for item tables, sequence data, page ids, unit records
constexpr int kSkGrid = 512;           // persistent workgroups: 2 per CU

__device__ __forceinline__ int kpiece_unit(int slot, int q) {
  return 4 * slot + (q ^ (((slot >> 1) & 1) | ((slot >> 2) & 2)));
}
__device__ __forceinline__ int vpiece_unit(int ch, int h) { return 2 * ch + (h ^ ((ch >> 2) & 1)); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// MFMA operands read from a key/value unit in LDS where they are used, so
// that no full register copy of the block is live.  TAIL: value lanes of keys
// at or past n_keys are zeroed (their pages are clamped stand-ins).
template <bool TAIL> struct LdsFrags {
  const char* buf;
  int k_off0, k_off1, v_off0, vpos, n_keys;
  __device__ __forceinline__ bf16x8 kf(int st, int ks) const {
    return *reinterpret_cast<const bf16x8*>(buf + (st ? k_off1 : k_off0) + 1024 * ks);
  }
  __device__ __forceinline__ bf16x8 vf(int dt) const {
    bf16x8 v = *reinterpret_cast<const bf16x8*>(buf + v_off0 + 512 * dt);
    if constexpr (TAIL) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (vpos + e >= n_keys) v[e] = static_cast<bf16>(0.f);
    }
    return v;
  }
};

// The stream-K split charges each non-empty item's start this many quarter
// blocks on top of its blocks: a piece of an item costs its workgroup the
// item's QT query units and a partial (or output) write besides its key
// blocks (per-workgroup timelines: a share that spans two items ended 4 us
// later at 64-row items and 8 us later at 128-row items).  Four blocks per 64
// rows timed best of 1.5, 2.5, 4 and 6.  Share w is the blocks whose cost
// start lies in [C w / W, C (w + 1) / W), C the total cost, so shares that
// start items take fewer blocks.
__host__ __device__ constexpr int sk_item_cost(int qt) { return 16 * qt; }

// Relative cost spans of the stream-K shares.  The hardware deals workgroup
// ids to the eight XCDs round-robin and gives each CU one workgroup before it
// gives any a second, so workgroup w runs on XCD w % 8, first on its CU when
// w < F (F = the CU count).  With equal shares (per-workgroup timelines, every
// box and shape measured) the odd-numbered XCDs streamed 6-10% slower than the
// even ones, and a CU's second workgroup 5-10% slower than its first, which
// ended first on almost every CU (its waves are the older ones).  Spans:
// kSkSpan = {first even, first odd, second even, second odd}.  Only while the
// shares average at least 8 blocks (and F is even): then no span is shorter
// than one block's cost, so every workgroup between the first and the last
// piece of an item holds a block of it.
struct SkSpan {
  int e1, o1, e2, o2, F;
};
constexpr int kSkSpan[4] = {24, 22, 21, 19};
__host__ __device__ inline SkSpan sk_spans(long blocks, int W, int first) {
  if (blocks >= 8L * W && first > 0 && first % 2 == 0) return {kSkSpan[0], kSkSpan[1], kSkSpan[2], kSkSpan[3], first};
  return {1, 1, 1, 1, 0};
}
__host__ __device__ inline long sk_pre(long v, int e, int o) { return e * ((v + 1) >> 1) + o * (v >> 1); }
// Total span of workgroups 0 .. v-1.
__host__ __device__ inline long sk_span_prefix(long v, const SkSpan& p) {
  return v <= p.F ? sk_pre(v, p.e1, p.o1) : sk_pre(p.F, p.e1, p.o1) + sk_pre(v - p.F, p.e2, p.o2);
}
// The last workgroup (below W) whose span prefix is at most V.
__host__ __device__ inline int sk_span_owner(long V, int W, const SkSpan& p) {
  const long SF = sk_pre(p.F, p.e1, p.o1);
  long w;
  if (p.F >= W || V < SF) {
    const long k = V / (p.e1 + p.o1), r = V % (p.e1 + p.o1);
    w = 2 * k + (r >= p.e1 ? 1 : 0);
  } else {
    const long k = (V - SF) / (p.e2 + p.o2), r = (V - SF) % (p.e2 + p.o2);
    w = p.F + 2 * k + (r >= p.e2 ? 1 : 0);
  }
  return (int)(w < W - 1 ? w : W - 1);
}

// Item `it` = (sequence slot, KV head g, row group qg), it = (slot Hkv + g) n_qg + qg:
// the row groups of one (sequence, head) are neighbours, so the shares that
// read the same keys for them run at the same time and the second read is a
// cache hit.
struct SkItem {
  int slot, g, b, L, r0, pr0, pr_last, n_keys, nb;
};

__device__ __forceinline__ SkItem sk_item(const AttnParams& a, const int* s_seq, int it, int maxblk) {
  SkItem m;
  const int qg = it % a.n_qg;
  const int sg = it / a.n_qg;
  m.g = sg % a.Hkv;
  m.slot = sg / a.Hkv;
  m.b = s_seq[4 * m.slot];
  m.L = s_seq[4 * m.slot + 1];
  m.r0 = s_seq[4 * m.slot + 2];
  const int rows_total = s_seq[4 * m.slot + 3] * a.G;
  m.pr0 = qg * a.item_rows;
  m.pr_last = min(rows_total, m.pr0 + a.item_rows) - 1;
  m.n_keys = m.L + m.pr_last / a.G + 1;
  m.nb = m.pr0 < rows_total ? min((m.n_keys + kBlk - 1) / kBlk, maxblk) : 0;
  return m;
}

template <int QT>
__global__ __launch_bounds__(256, 2) void verify_attn_sk_kernel(AttnParams a) {
  static_assert(QT == 1 || QT == 2, "tiles per wave");
  constexpr int D = 128;
  constexpr int PS = 16;
  constexpr int kRowsI = 64 * QT;      // rows per item: QT query units of 64 rows
  const int tid = threadIdx.x;
  const int t = uni(tid / kWave);      // row tile (wave-uniform)
  const int lane = lane_id();
  const int c16 = lane & 15, j = lane >> 4;
  const int n_it = a.n_seq * a.Hkv * a.n_qg;
  const int maxblk = (a.max_pages * PS + kBlk - 1) / kBlk;

  __shared__ __attribute__((aligned(1024))) char s_ring[kSkBuf * kSkUnit];
  __shared__ int s_meta[kSkMeta];
  __shared__ int s_part[2][256];
  if (2 * (n_it + 1) + 4 * a.n_seq > kSkMeta) return;   // the host sizes every launch to fit
  int* s_start = s_meta;                    // [n_it + 1] first block of each item
  int* s_ne = s_start + n_it + 1;           // [n_it + 1] non-empty items before each item
  int* s_seq = s_ne + n_it + 1;             // [n_seq][4]: b, L, r0, rows
  int* s_pg = s_seq + 4 * a.n_seq;          // [2 per block]: page ids of this workgroup's blocks

  // Sequence data, then every item's block count, and the exclusive scans of
  // the block counts and of the non-empty flags.
  for (int sl = tid; sl < a.n_seq; sl += 256) {
    const int b = a.seq_ids ? a.seq_ids[sl] : sl;
    const int r0 = a.cu_q[b];
    s_seq[4 * sl] = b;
    s_seq[4 * sl + 1] = max(a.ctx_lens[b], 0);
    s_seq[4 * sl + 2] = r0;
    s_seq[4 * sl + 3] = a.cu_q[b + 1] - r0;
  }
  __syncthreads();
  const int per = (n_it + 255) / 256;
  const int i_lo = min(n_it, tid * per), i_hi = min(n_it, (tid + 1) * per);
  const int w = blockIdx.x;
  int B_tot = 0, W = 0, lo = 0, hi = 0;
  {
    // The thread's items' block counts (kept in s_start until their offsets
    // are known), then exclusive scans over the threads, whose order is item
    // order: within each wave with DPP moves, across the four waves' totals.
    int run = 0, cnt = 0;
    for (int i = i_lo; i < i_hi; ++i) {
      const int nb = sk_item(a, s_seq, i, maxblk).nb;
      s_start[i] = nb;
      run += nb;
      cnt += nb > 0;
    }
    const int inc_r = wave_incl_scan_i(run), inc_c = wave_incl_scan_i(cnt);
    if (lane == kWave - 1) {
      s_part[0][t] = inc_r;
      s_part[1][t] = inc_c;
    }
    if (tid == 0) {   // no claim yet: the share's bound is then the last block's end
      s_part[0][4] = s_part[0][5] = -1;
      s_part[1][4] = s_part[1][5] = -1;
    }
    __syncthreads();
    int bs = inc_r - run, ns = inc_c - cnt, NE = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      B_tot += s_part[0][k];
      NE += s_part[1][k];
      if (k < t) {
        bs += s_part[0][k];
        ns += s_part[1][k];
      }
    }
    // Share w: the blocks whose cost start lies in [y_lo, y_hi), in quarter
    // blocks (sk_item_cost), the spans weighted by XCD and CU slot (kSkSpan).
    constexpr int c4 = sk_item_cost(QT);
    W = min((int)gridDim.x, B_tot);
    const int C = 4 * B_tot + c4 * NE;
    const SkSpan sp = sk_spans(B_tot, W, a.sk_first);
    const long SW = sk_span_prefix(W, sp);
    int y_lo = 0, y_hi = 0;
    if (w < W) {
      y_lo = (int)((long)C * sk_span_prefix(w, sp) / SW);
      y_hi = (int)((long)C * sk_span_prefix(w + 1, sp) / SW);
    }
    // Item offsets, and the share's bounds: the first block whose cost start
    // reaches y_lo (y_hi), claimed by the one thread that owns its item.
    // Block x of non-empty item i costs from 4 x + c4 (ne_i + 1); the block
    // before the item's first (the previous non-empty item's last) from
    // 4 bs_i - 4 + c4 ne_i.
    for (int i = i_lo; i < i_hi; ++i) {
      const int nb = s_start[i];
      s_start[i] = bs;
      s_ne[i] = ns;
      if (nb > 0 && w < W) {
        const int cs = 4 * bs + c4 * (ns + 1), ce = cs + 4 * (nb - 1);
        if (y_lo <= ce && (bs == 0 || cs - 4 - c4 < y_lo)) {
          s_part[0][4] = i;
          s_part[0][5] = bs + max(0, (y_lo - cs + 3) >> 2);
        }
        if (y_hi <= ce && (bs == 0 || cs - 4 - c4 < y_hi)) {
          s_part[1][4] = i;
          s_part[1][5] = bs + max(0, (y_hi - cs + 3) >> 2);
        }
      }
      bs += nb;
      ns += nb > 0;
    }
    if (tid == 255) { s_start[n_it] = bs; s_ne[n_it] = ns; }   // thread 255 ends at n_it or owns no items
  }
  __syncthreads();
  if (blockIdx.x == 0)
    for (int i = tid; i <= n_it; i += 256) {
      a.sk_start[i] = s_start[i];
      a.sk_ne[i] = s_ne[i];
    }
  if (w >= W) return;
  lo = uni(s_part[0][5] < 0 ? B_tot : s_part[0][5]);
  hi = uni(s_part[1][5] < 0 ? B_tot : s_part[1][5]);
  if (lo >= hi) return;   // a share of no blocks: its cost span lies in item starts
  // Item of block x among items l0 .. l1: s_start[i] <= x < s_start[i + 1]
  // (empty items never qualify).
  auto item_of = [&](int x, int l0, int l1) {
    while (l0 < l1) {
      const int mid = (l0 + l1 + 1) >> 1;
      if (s_start[mid] <= x) l0 = mid; else l1 = mid - 1;
    }
    return l0;
  };
  // The share's first block lies in the item that claimed it; its last block
  // in that of the block after it or an earlier one.
  const int i_first = uni(s_part[0][4]);
  const int i_last = uni(item_of(hi - 1, i_first, s_part[1][4] >= 0 ? s_part[1][4] : n_it - 1));
  const int n_units = (hi - lo) + QT * (s_ne[i_last + 1] - s_ne[i_first]);
  if (2 * (n_it + 1) + 4 * a.n_seq + 2 * (hi - lo) + n_units > kSkMeta) return;
  int* s_uq = s_pg + 2 * (hi - lo);          // [n_units] the workgroup's units, in order
  // Lane-fixed parts of this wave's loads: key slice t and value channels
  // 32t .. 32t+31 of each page; query rows 16t .. 16t+15, four per load.
  const int ksl = lane >> 2;
  const int k_src = t * (PS * 32) + ksl * 32 + 8 * ((lane & 3) ^ (((ksl >> 1) & 1) | ((ksl >> 2) & 2)));
  const int vch = lane >> 1;
  const int v_src = (32 * t + vch) * PS + 8 * ((lane & 1) ^ ((vch >> 2) & 1));
  const bf16* kc = reinterpret_cast<const bf16*>(a.k_cache);
  const bf16* vc = reinterpret_cast<const bf16*>(a.v_cache);
  const bf16* qp = reinterpret_cast<const bf16*>(a.q);

  // Load side: unit m goes to buffer m % kSkBuf; past the last unit the last
  // one is loaded again, so that every wait below has the same count.  The
  // next unit's record and page ids are read one issue ahead.
  int d_g = 0;                               // KV head of the load side's current item
  int d_rec = 4 * i_first + 1, d_pg0 = 0, d_pg1 = 0;   // unit 0: the first item's first query unit
  auto dma_issue = [&](int m) {
    char* buf = s_ring + (m % kSkBuf) * kSkUnit;
    if (d_rec & 1) {
      const SkItem it = sk_item(a, s_seq, d_rec >> 2, maxblk);
      const int h0 = 64 * ((d_rec >> 1) & 1);
      d_g = it.g;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = 16 * t + 4 * u + (lane >> 4);
        const int pr = min(it.pr0 + h0 + r, it.pr_last);
        const bf16* row = qp + ((size_t)(it.r0 + pr / a.G) * a.Hq + it.g * a.G + pr % a.G) * D;
        dma16(row + 8 * ((lane & 15) ^ (r & 7)), buf + 1024 * (4 * t + u));
      }
    } else {
      const size_t b0 = (size_t)(d_pg0 * a.Hkv + d_g) * PS * D;
      const size_t b1 = (size_t)(d_pg1 * a.Hkv + d_g) * PS * D;
      dma16(kc + b0 + k_src, buf + 1024 * t);
      dma16(vc + b0 + v_src, buf + 1024 * (8 + t));
      dma16(kc + b1 + k_src, buf + 1024 * (4 + t));
      dma16(vc + b1 + v_src, buf + 1024 * (12 + t));
    }
  };
  auto dma_next = [&](int m) {
    d_rec = uni(s_uq[min(m + 1, n_units - 1)]);
    if (!(d_rec & 1)) {
      d_pg0 = uni(s_pg[(d_rec >> 2) * 2]);
      d_pg1 = uni(s_pg[(d_rec >> 2) * 2 + 1]);
    }
  };
  auto dma_unit = [&](int m) {
    dma_issue(m);
    dma_next(m);
  };
  // The first query unit needs no table: it is issued now, so that its load
  // overlaps the page-table reads and the window append below.
  dma_issue(0);

  // Unit records: query unit h (rows 64 h .. 64 h + 63 of the item) holds
  // 4 item + 2 h + 1; a key/value unit holds 4 x + 2 (last block of the
  // item's piece) with x the block's offset in the share.  Block x of item i is
  // unit (x - lo) + QT (non-empty items from i_first through i); the QT units
  // before an item's first block are its queries.  The page ids of a
  // thread's first block stay in registers until the window append below has
  // issued its own loads, so that both sets of loads are in flight together;
  // those of further blocks (shares above 256 blocks) are written at once.
  int pg_x = -1, pg_a = 0, pg_b = 0;
  for (int x = lo + tid; x < hi; x += 256) {
    const int i = item_of(x, i_first, i_last);
    const int u = (x - lo) + QT * (s_ne[i + 1] - s_ne[i_first]);
    const int last = (x + 1 == s_start[i + 1] || x + 1 == hi) ? 2 : 0;
    s_uq[u] = 4 * (x - lo) + last;
    if (x == max(lo, s_start[i]))
      for (int h = 0; h < QT; ++h) s_uq[u - QT + h] = 4 * i + 2 * h + 1;
    const SkItem m = sk_item(a, s_seq, i, maxblk);
    const int* pt_row = a.page_table + (size_t)m.b * a.max_pages;
    const int pl = 2 * (x - s_start[i]);
    const int ga = pt_row[min(pl, a.max_pages - 1)], gb = pt_row[min(pl + 1, a.max_pages - 1)];
    if (pg_x < 0) {
      pg_x = x;
      pg_a = ga;
      pg_b = gb;
    } else {
      s_pg[2 * (x - lo)] = clampi(ga, 0, a.num_pages - 1);
      s_pg[2 * (x - lo) + 1] = clampi(gb, 0, a.num_pages - 1);
    }
  }

  // Window append: the window's keys and values at positions L .. L+k-1 go
  // to the pages, for the positions inside this share's blocks (every window
  // position lies in some item's blocks; positions in two shares are written
  // twice, with the same values).  Each workgroup writes the positions it
  // reads, and waits for the writes before it loads any key/value unit.
  {
    bf16* kw = reinterpret_cast<bf16*>(a.k_cache);
    bf16* vw = reinterpret_cast<bf16*>(a.v_cache);
    const bf16* kn = reinterpret_cast<const bf16*>(a.k_new);
    const bf16* vn = reinterpret_cast<const bf16*>(a.v_new);
    for (int i = i_first; i <= i_last; ++i) {
      const SkItem m = sk_item(a, s_seq, i, maxblk);
      if (m.nb == 0) continue;
      const int kb = s_seq[4 * m.slot + 3];
      const int xb = max(lo, s_start[i]) - s_start[i], xe = min(hi, s_start[i + 1]) - s_start[i];
      const int p_lo = max(m.L, kBlk * xb), p_hi = min(m.L + kb, kBlk * xe);
      const int* pt_row = a.page_table + (size_t)m.b * a.max_pages;
      for (int e = tid; e < (p_hi - p_lo) * (D / 8); e += 256) {
        const int pos = p_lo + e / (D / 8), d0 = 8 * (e % (D / 8));
        const int page = clampi(pt_row[clampi(pos >> 4, 0, a.max_pages - 1)], 0, a.num_pages - 1);
        const int sl = pos & (PS - 1);
        const size_t src = ((size_t)(m.r0 + pos - m.L) * a.Hkv + m.g) * D + d0;
        const bf16x8 kv = *reinterpret_cast<const bf16x8*>(kn + src);
        const bf16x8 vv = *reinterpret_cast<const bf16x8*>(vn + src);
        const size_t pb = (size_t)(page * a.Hkv + m.g) * PS * D;
        *reinterpret_cast<bf16x8*>(kw + pb + (d0 / 32) * (PS * 32) + sl * 32 + (d0 & 31)) = kv;
#pragma unroll
        for (int c = 0; c < 8; ++c) vw[pb + (size_t)(d0 + c) * PS + sl] = vv[c];
      }
    }
  }
  if (pg_x >= 0) {
    s_pg[2 * (pg_x - lo)] = clampi(pg_a, 0, a.num_pages - 1);
    s_pg[2 * (pg_x - lo) + 1] = clampi(pg_b, 0, a.num_pages - 1);
  }

  // The window's stores and the page-table reads are done and the tables are
  // visible before the first key/value unit is issued.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  dma_next(0);
  for (int m = 1; m < kSkBuf - 1; ++m) dma_unit(m);

  // Per-lane LDS offsets of the MFMA operands within a unit.  Channel
  // 16 dt + c16 lies in value piece dt / 2 at unit 2 (16 (dt % 2) + c16) + h',
  // and h' does not depend on dt, so the value offsets step by 512 bytes.
  int k_off[2];
#pragma unroll
  for (int st = 0; st < 2; ++st) {
    const int kk = 8 * (c16 >> 2) + 4 * st + (c16 & 3);
    k_off[st] = 4096 * (kk >> 4) + 16 * kpiece_unit(kk & 15, j);
  }
  const int v_off0 = 8192 + 4096 * (j >> 1) + 16 * vpiece_unit(c16, j & 1);

  // Compute side.  The units come as items: QT query units, then the item's
  // key/value units up to the one that ends its piece.  Tile tt of this wave
  // holds the item's rows 64 tt + 16 t .. 64 tt + 16 t + 15.
  int c_rec = uni(s_uq[0]);
  int n = 0;
  // Unit n of this wave's loads has landed (the next one may still be in
  // flight) and every LDS read this wave issued has returned (the query
  // fragments are read into registers one unit or more before their first
  // use, so the compiler would not wait for them here); after the barrier
  // every wave's pieces of unit n are visible, and every wave is done with
  // unit n - 1, whose buffer the next issue refills.
  auto next_unit = [&](int& rec) -> const char* {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(4 * (kSkBuf - 2)) : "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    dma_unit(n + kSkBuf - 1);
    rec = c_rec;
    c_rec = uni(s_uq[min(n + 1, n_units - 1)]);
    const char* buf = s_ring + (n % kSkBuf) * kSkUnit;
    ++n;
    return buf;
  };
  while (n < n_units) {
    int rec;
    const int i = uni(c_rec >> 2);
    SkItem it = sk_item(a, s_seq, i, maxblk);
    it.g = uni(it.g);
    it.L = uni(it.L);
    it.r0 = uni(it.r0);
    it.pr0 = uni(it.pr0);
    it.pr_last = uni(it.pr_last);
    it.n_keys = uni(it.n_keys);
    const int x0 = uni(s_start[i] - lo);   // offset in the share of the item's block 0 (may be negative)
    const bool full = uni(s_start[i] >= lo && s_start[i + 1] <= hi);   // the whole item lies in this share
    RegQT<D, QT> qf;
    int qlimit[QT], prq[QT];
    bool has_rows[QT];
#pragma unroll
    for (int tt = 0; tt < QT; ++tt) {
      const char* buf = next_unit(rec);
      prq[tt] = it.pr0 + 64 * tt + 16 * t + c16;
      qlimit[tt] = it.L + min(prq[tt], it.pr_last) / a.G + 1;
      has_rows[tt] = uni(it.pr0 + 64 * tt + 16 * t <= it.pr_last);
      const int r = 16 * t + c16;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        qf.q[tt][ks] = *reinterpret_cast<const bf16x8*>(buf + 256 * r + 16 * ((j + 4 * ks) ^ (r & 7)));
        if (prq[tt] > it.pr_last) qf.q[tt][ks] = bf16x8{};
      }
    }
    floatx4 acc[QT][D / 16];
    float m_run[QT], l_run[QT];
#pragma unroll
    for (int tt = 0; tt < QT; ++tt) {
      m_run[tt] = -INFINITY;
      l_run[tt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[tt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    // Blocks that end at or before main_end hold no key past any row's
    // limit and no stand-in key: they take the unmasked block, in a loop of
    // their own; the item's last blocks (the window's) follow, masked.  All
    // QT tiles run, also where the last has no rows (its query fragments are
    // zero and its results are never written).
    const int main_end = min(it.n_keys, it.L & ~(kBlk - 1));
    bool ended = false;
    while (n < n_units) {
      const int t0 = kBlk * ((c_rec >> 2) - x0);   // the next unit: a key/value unit of this item
      if (t0 + kBlk > main_end) break;
      const char* buf = next_unit(rec);
      if (has_rows[0]) {
        const LdsFrags<false> f{buf, k_off[0], k_off[1], v_off0, 0, 0};
        attend_block<bf16, D, QT, false>(a, f, qf, qlimit, t0, acc, m_run, l_run);
      }
      if (rec & 2) { ended = true; break; }
    }
    while (!ended && n < n_units) {
      const char* buf = next_unit(rec);
      const int t0 = kBlk * ((rec >> 2) - x0);
      if (has_rows[0]) {
        const LdsFrags<true> f{buf, k_off[0], k_off[1], v_off0, t0 + 8 * j, it.n_keys};
        attend_block<bf16, D, QT, true>(a, f, qf, qlimit, t0, acc, m_run, l_run);
      }
      ended = rec & 2;
    }
    // The item's piece ends here.  A whole item is written out; a piece
    // leaves a partial at slot item + workgroup.
#pragma unroll
    for (int tt = 0; tt < QT; ++tt) {
      float l_tot = l_run[tt] + lane_xor16(l_run[tt]);
      l_tot += lane_xor32(l_tot);
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      if (!has_rows[tt] || prq[tt] > it.pr_last) continue;
      if (full) {
        const int ri = prq[tt] / a.G, hl = prq[tt] % a.G;
        bf16* orow = reinterpret_cast<bf16*>(a.out) + ((size_t)(it.r0 + ri) * a.Hq + it.g * a.G + hl) * D;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(acc[tt][dt][e] * inv);
          *reinterpret_cast<bf16x4*>(orow + 16 * dt + 4 * j) = v;
        }
      } else {
        const size_t ps = (size_t)i + w;
        const int row = 64 * tt + 16 * t + c16;
        float* po = a.part_o + (ps * kRowsI + row) * D;
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt)
          *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * j) = acc[tt][dt] * inv;
        if (j == 0)
          a.part_lse[ps * kRowsI + row] = l_tot > 0.f ? m_run[tt] + fast_log2(l_tot) : -INFINITY;
      }
    }
    // The loop's count-based waits ("all but the newest unit's loads") count
    // on the memory operations in flight completing in issue order, which is
    // not promised once stores are mixed in: the piece's stores (and the
    // units in flight) are waited for here.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // reloads past the end
}

// Merge the pieces of every item that the stream-K kernel split between
// workgroups: piece w of item it sits at slot it + w, for the workgroups w
// whose share of blocks meets the item.
__global__ __launch_bounds__(256) void attn_combine_sk_kernel(AttnParams a) {
  // Grid x = item_rows / 16 parts per item: 16 packed rows per workgroup,
  // 16 threads per row, 8 channels per thread.
  constexpr int D = 128;
  const int R = a.item_rows;
  const int qg = blockIdx.x / (R / 16), rq = blockIdx.x % (R / 16);
  const int slot = blockIdx.y / a.Hkv, g = blockIdx.y % a.Hkv;
  const int it = (slot * a.Hkv + g) * a.n_qg + qg;
  const int n_it = a.n_seq * a.Hkv * a.n_qg;
  // the item's block range and the sequence's rows, loaded side by side
  const int B_tot = a.sk_start[n_it];
  const int s0 = a.sk_start[it], s1 = a.sk_start[it + 1];
  const int b = a.seq_ids ? a.seq_ids[slot] : slot;
  const int r0 = a.cu_q[b];
  const int kb = a.cu_q[b + 1] - r0;
  if (s1 <= s0) return;
  const int NE = a.sk_ne[n_it], ne = a.sk_ne[it];
  const int W = min(a.sk_grid, B_tot);
  // Workgroup whose share holds block x: the last w whose span starts, at
  // C S(w) / S(W), at or below the block's cost start 4 x + c4 (ne + 1) (the
  // attention kernel's split; S the weighted span prefix).
  const int c4 = sk_item_cost(R / 64);
  const long C = 4L * B_tot + (long)c4 * NE;
  const SkSpan sp = sk_spans(B_tot, W, a.sk_first);
  const long SW = sk_span_prefix(W, sp);
  auto wg_of = [&](int x) {
    const long cx = 4L * x + (long)c4 * (ne + 1);
    return sk_span_owner(((cx + 1) * SW + C - 1) / C - 1, W, sp);   // the largest S(w) allowed
  };
  const int w0 = wg_of(s0), w1 = wg_of(s1 - 1);
  if (w0 == w1) return;   // written whole by one workgroup
  const int G = a.G;
  const int r = 16 * rq + threadIdx.x / 16;           // packed row within the group
  const int dq = (threadIdx.x % 16) * (D / 16);
  const int pr = qg * R + r;
  if (pr >= min(kb * G, (qg + 1) * R)) return;
  // One pass over the pieces with a running maximum: each piece's weight and
  // partial are loaded together.
  float M = -INFINITY, wsum = 0.f;
  floatx4 o0 = {0.f, 0.f, 0.f, 0.f}, o1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int w = w0; w <= w1; ++w) {
    const float lse = a.part_lse[((size_t)it + w) * R + r];
    const float* po = a.part_o + (((size_t)it + w) * R + r) * D + dq;
    const floatx4 p0 = ld16<floatx4>(po), p1 = ld16<floatx4>(po + 4);
    const float Mn = fmaxf(M, lse);
    const float Mu = (Mn == -INFINITY) ? 0.f : Mn;
    const float sc = fast_exp2(M - Mu);                 // 0 while M is -inf
    const float wgt = fast_exp2(lse - Mu);
    wsum = wsum * sc + wgt;
    o0 = o0 * sc + wgt * p0;
    o1 = o1 * sc + wgt * p1;
    M = Mn;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const int i = pr / G, hl = pr % G;
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = static_cast<bf16>(o0[e] * inv);
    v[4 + e] = static_cast<bf16>(o1[e] * inv);
  }
  *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(a.out) + ((size_t)(r0 + i) * a.Hq + g * G + hl) * D + dq) = v;
}

// Merge the chunk partials of every (sequence, KV head, row group) that spans
// more than one chunk: out = sum_c 2^(lse_c - M) o_c / sum_c 2^(lse_c - M).
template <typename DT, int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams a) {
  const int qg = blockIdx.x;
  const int slot = blockIdx.y / a.Hkv, g = blockIdx.y % a.Hkv;
  const int b = a.seq_ids ? a.seq_ids[slot] : slot;
  const int L = max(a.ctx_lens[b], 0);
  const int r0 = a.cu_q[b];
  const int kb = a.cu_q[b + 1] - r0;
  const int G = a.G;
  const int pr0 = qg * kRows;
  if (pr0 >= kb * G) return;
  const int pr_last = min(kb * G, pr0 + kRows) - 1;
  const int n_keys = L + pr_last / G + 1;
  const int n_chunks = min((n_keys + a.chunk - 1) / a.chunk, a.max_chunks);
  if (n_chunks <= 1) return;
  const int r = threadIdx.x / 4;            // packed row within the group
  const int dq = (threadIdx.x % 4) * (D / 4);
  const int pr = pr0 + r;
  if (pr > pr_last) return;
  const size_t base = (((size_t)slot * a.Hkv + g) * a.n_qg + qg) * a.max_chunks;
  float M = -INFINITY;
  for (int cc = 0; cc < n_chunks; ++cc) M = fmaxf(M, a.part_lse[(base + cc) * kRows + r]);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float o[D / 4];
#pragma unroll
  for (int e = 0; e < D / 4; ++e) o[e] = 0.f;
  float wsum = 0.f;
  for (int cc = 0; cc < n_chunks; ++cc) {
    const float wgt = fast_exp2(a.part_lse[(base + cc) * kRows + r] - Mu);
    wsum += wgt;
    const float* po = a.part_o + ((base + cc) * kRows + r) * D + dq;
#pragma unroll
    for (int e = 0; e < D / 4; e += 4) {
      floatx4 v = ld16<floatx4>(po + e);
      o[e] += wgt * v[0];
      o[e + 1] += wgt * v[1];
      o[e + 2] += wgt * v[2];
      o[e + 3] += wgt * v[3];
    }
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const int i = pr / G, hl = pr % G;
  DT* orow = reinterpret_cast<DT*>(a.out) + ((size_t)(r0 + i) * a.Hq + g * G + hl) * D + dq;
#pragma unroll
  for (int e = 0; e < D / 4; ++e) orow[e] = from_f32<DT>(o[e] * inv);
}

template <typename DT, int D, int QT>
hipError_t launch_t(const AttnParams& p, dim3 grid, dim3 cgrid, hipStream_t st) {
  trace_begin(st);
  hipLaunchKernelGGL((append_window_kernel<DT, D>), dim3(cgrid.y), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_mark(st);
  hipLaunchKernelGGL((verify_attn_kernel<DT, D, QT>), grid, dim3(256), 0, st, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_mark(st);
  hipLaunchKernelGGL((attn_combine_kernel<DT, D>), cgrid, dim3(256), 0, st, p);
  e = hipGetLastError();
  trace_mark(st);
  return e;
}

hipError_t launch_sk(const AttnParams& p, dim3 cgrid, hipStream_t st) {
  // The window append happens inside the attention kernel (an empty
  // interval in the trace where the other path has its append kernel).
  trace_begin(st);
  trace_mark(st);
  hipError_t e;
  if (p.item_rows == 128)
    hipLaunchKernelGGL(verify_attn_sk_kernel<2>, dim3(p.sk_grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(verify_attn_sk_kernel<1>, dim3(p.sk_grid), dim3(256), 0, st, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  trace_mark(st);
  hipLaunchKernelGGL(attn_combine_sk_kernel, dim3(cgrid.x * (p.item_rows / 16), cgrid.y), dim3(256), 0, st, p);
  e = hipGetLastError();
  trace_mark(st);
  return e;
}

template <typename DT, int D>
hipError_t launch_d(const AttnParams& p, int qt, dim3 grid, dim3 cgrid, hipStream_t st) {
  switch (qt) {
    case 1: return launch_t<DT, D, 1>(p, grid, cgrid, st);
    case 2: return launch_t<DT, D, 2>(p, grid, cgrid, st);
    case 3: return launch_t<DT, D, 3>(p, grid, cgrid, st);
    default: return launch_t<DT, D, 4>(p, grid, cgrid, st);
  }
}

}  // namespace

AttnPlan attn_plan(int n_seq, int Hq, int Hkv, int D, int max_q, int max_pages, int page_size) {
  AttnPlan pl{};
  const int G = Hq / Hkv;
  const long rows = (long)max_q * G;
  pl.n_qg = (int)((rows + kRows - 1) / kRows);
  pl.qt = rows >= kRows ? 4 : (int)((rows + 15) / 16);
  // Keys per wave: the largest split that still yields enough workgroups
  // (>= 4 per CU, by the host-side upper bound of the key count) for the
  // hardware to balance ragged lengths.
  {
    const long max_keys_ub = (long)max_pages * page_size;
    pl.sub = 128;
    for (int s = 1024; s >= 256; s /= 2) {
      const long items = (long)n_seq * Hkv * pl.n_qg * ((max_keys_ub + 4L * s - 1) / (4L * s));
      if (items >= 4L * 256) { pl.sub = s; break; }
    }
  }
  // A wave's keys must span at most 64 pages (one page id per lane).
  while (pl.sub > 32 && pl.sub > 63 * page_size) pl.sub /= 2;
  pl.chunk = kWaves * pl.sub;
  const long max_keys = (long)max_pages * page_size;
  int mc = (int)((max_keys + pl.chunk - 1) / pl.chunk);
  pl.max_chunks = mc;
  const size_t slots = (size_t)n_seq * Hkv * pl.n_qg * pl.max_chunks;
  pl.part_o_bytes = slots * kRows * D * sizeof(float);
  pl.part_lse_bytes = slots * kRows * sizeof(float);
  pl.workspace_bytes = pl.part_o_bytes + pl.part_lse_bytes + 256;
  // D = 128 heads in 16-slot pages take the persistent stream-K kernel (bf16;
  // the launch checks the type) when its LDS tables fit: item starts and
  // non-empty counts, sequence data, and per workgroup two page ids per
  // block and one record per unit (its units add sk_qt per item).
  // More than 64 rows per (sequence, KV head) take 128-row items, two 16-row
  // tiles per wave, so that each key is read once per 128 rows.
  pl.sk_qt = rows > kRows ? 2 : 1;
  pl.sk_n_qg = (int)((rows + 64L * pl.sk_qt - 1) / (64L * pl.sk_qt));
  const long n_it = (long)n_seq * Hkv * pl.sk_n_qg;
  const long maxblk = (max_keys + kBlk - 1) / kBlk;
  // A share spans at most C wmax / S(W) + 1 quarter blocks of cost (C = 4
  // blocks + c4 per non-empty item; with the span weights W is the full grid
  // and S(W) >= W wmin), so it holds at most that / 4 + 1 blocks; costs stay
  // below 2^31.
  const long c4 = sk_item_cost(pl.sk_qt);
  const long wmax = std::max(std::max(kSkSpan[0], kSkSpan[1]), std::max(kSkSpan[2], kSkSpan[3]));
  const long wmin = std::min(std::min(kSkSpan[0], kSkSpan[1]), std::min(kSkSpan[2], kSkSpan[3]));
  const long wden = 4L * kSkGrid * wmin;
  const long share = std::max((n_it * (4 * maxblk + c4) * wmax + wden - 1) / wden, (c4 + 3) / 4 + 1) + 2;
  pl.sk = D == 128 && page_size == 16 && n_it * (4 * maxblk + c4) < (1L << 31) &&
          2 * (n_it + 1) + 4L * n_seq + 3 * share + pl.sk_qt * n_it <= kSkMeta;
  if (pl.sk) {
    const size_t sk_slots = (size_t)n_it + kSkGrid;
    const size_t sk_rows = 64 * (size_t)pl.sk_qt;
    pl.sk_o_bytes = std::max(pl.part_o_bytes, sk_slots * sk_rows * D * sizeof(float));
    pl.sk_lse_bytes = std::max(pl.part_lse_bytes, sk_slots * sk_rows * sizeof(float));
    pl.workspace_bytes = pl.sk_o_bytes + pl.sk_lse_bytes + 2 * (n_it + 1) * sizeof(int32_t) + 256;
  }
  return pl;
}

// Split-KV scratch of the allocation-free entry point (verify_attn_paged_noalloc):
// every partial and item start a call reads is written earlier in the same
// call, so nothing in it needs clearing.  Each GPU the library runs on holds
// its own copy until the process ends; calls that overlap on one GPU share it
// and race.
static __device__ __align__(256) char scratch[IPDV_NOALLOC_SCRATCH_BYTES_DEV];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch`, per device

// The current device's address of `scratch`, looked up once per device with
// that device current.  In host code the array's name is not a device address.
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

hipError_t launch_verify_attn_noalloc(const AttnLaunch& L, const AttnPlan& pl, hipStream_t st) {
  if (pl.workspace_bytes > IPDV_NOALLOC_SCRATCH_BYTES_DEV) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return e;
  AttnLaunch l2 = L;
  l2.workspace = ws;
  return launch_verify_attn(l2, pl, st);
}

hipError_t launch_verify_attn(const AttnLaunch& L, const AttnPlan& pl, hipStream_t st) {
  AttnParams p{};
  p.q = L.q;
  p.k_new = L.k_new;
  p.v_new = L.v_new;
  p.k_cache = L.k_cache;
  p.v_cache = L.v_cache;
  p.page_table = L.page_table;
  p.ctx_lens = L.ctx_lens;
  p.cu_q = L.cu_q;
  p.seq_ids = L.seq_ids;
  p.out = L.out;
  p.part_o = reinterpret_cast<float*>(L.workspace);
  p.part_lse = reinterpret_cast<float*>(reinterpret_cast<char*>(L.workspace) + pl.part_o_bytes);
  p.max_pages = L.max_pages;
  p.Hq = L.Hq;
  p.Hkv = L.Hkv;
  p.G = L.Hq / L.Hkv;
  p.page_size = L.page_size;
  p.log2ps = __builtin_ctz(L.page_size);
  p.num_pages = L.num_pages;
  p.chunk = pl.chunk;
  p.sub = pl.sub;
  p.max_chunks = pl.max_chunks;
  p.n_qg = pl.n_qg;
  p.n_seq = L.n_seq;
  p.scale_log2 = L.scale * 1.4426950408889634f;
  dim3 grid((L.n_seq * L.Hkv + 7) / 8 * 8, pl.n_qg, pl.max_chunks);
  dim3 cgrid(pl.n_qg, L.n_seq * L.Hkv);
  if (pl.sk && L.dtype_bf16 && L.D == 128 && L.page_size == 16) {
    p.part_lse = reinterpret_cast<float*>(reinterpret_cast<char*>(L.workspace) + pl.sk_o_bytes);
    p.sk_start = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(L.workspace) + pl.sk_o_bytes + pl.sk_lse_bytes);
    p.sk_ne = p.sk_start + ((size_t)L.n_seq * L.Hkv * pl.sk_n_qg + 1);
    p.sk_grid = kSkGrid;
    p.sk_first = device_cus();
    p.n_qg = pl.sk_n_qg;
    p.item_rows = 64 * pl.sk_qt;
    return launch_sk(p, dim3(pl.sk_n_qg, L.n_seq * L.Hkv), st);
  }
  if (L.dtype_bf16) {
    return L.D == 64 ? launch_d<bf16, 64>(p, pl.qt, grid, cgrid, st)
                     : launch_d<bf16, 128>(p, pl.qt, grid, cgrid, st);
  }
  return launch_d<float, 64>(p, pl.qt, grid, cgrid, st);   // fp32: D = 64 only
}

}  // namespace ipdv
